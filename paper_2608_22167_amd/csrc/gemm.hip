// Weight-streaming grouped GEMM on gfx950: the general fallback (fp32 layers,
// shapes the weight-slab and tiled kernels do not take).
//
// At decode every projection of the layer is skinny: a few to a few hundred
// token rows against a weight matrix that is read exactly once, so the kernels
// are bound by streaming the weights from HBM. A workgroup owns a slab of
// 16 * WN * NB consecutive weight rows of one group (one expert, or the single
// dense matrix) and all token rows of that group. Its WN x WK wavefronts split
// the slab along N (WN) and the reduction dimension along K (WK); each
// wavefront keeps an NB x MB grid of 16x16 accumulators, so every token
// fragment it loads feeds NB matrix-core products and every weight fragment
// feeds MB. Partial tiles of the WK wavefronts are summed into LDS in a fixed
// order, and a fused epilogue finishes the slab:
//   EPI_QKV      + bias, rotary embedding of q and k, q to the q buffer and
//                k / v straight into their KV-cache pages (the append)
//   EPI_RESIDUAL + bias + residual (fp32), e.g. h1 = x + o W_o^T + b_o
//   EPI_SWIGLU   + bias, gate/up pairs (rows 2j, 2j+1) -> clamped SwiGLU
//   EPI_BIAS     + bias (fp32)
// Token rows may be gathered through row_src (the expert-sorted order), so the
// permuted activations are never materialised.
#include "device.h"
#include "gemm_epilogue.h"
#include "kernels.h"

namespace mcpu {

// ---------------------------------------------------------------------------
// weight sources: where a lane's 8 weights of a 32-wide chunk come from
// ---------------------------------------------------------------------------

// Dense weights in the layer dtype.
template <typename T, int WF> struct WSrc {
  using Raw = Frag<T>;
  const T* p;
  __device__ __forceinline__ void init(const Gemm& P, int grp, int row, int kg) {
    p = reinterpret_cast<const T*>(P.w) + grp * P.w_group_stride + (int64_t)row * P.k + 8 * kg;
  }
  __device__ __forceinline__ void fetch(Raw& r, int c) const { r.load(p + c * 32); }
  __device__ __forceinline__ Frag<T> frag(const Raw& r, bool&) const { return r; }
};

// One E2M1 element (4-bit code: sign, 2 exponent bits, 1 mantissa bit) times the
// block scale, as bfloat16 bits. dexp = (scale - 127) << 7 adds the E8M0 power of
// two to the bfloat16 exponent field; E2M1 magnitudes 0, .5, 1, 1.5, 2, 3, 4, 6
// are 0 and bfloat16 0x3F00, 0x3F80 + 0x40 (m - 2) for m >= 2.
__device__ __forceinline__ uint32_t e2m1_to_bf16(uint32_t nib, int32_t dexp) {
  const uint32_t m = nib & 7u;
  uint32_t b = m >= 2u ? 0x3F80u + (m - 2u) * 0x40u : (m == 1u ? 0x3F00u : 0u);
  b = b ? (uint32_t)((int32_t)b + dexp) : 0u;
  return b | ((nib & 8u) << 12);
}

// MXFP4 experts (OCP MX): per row, K/2 bytes of E2M1 codes (low nibble = even
// column) and K/32 E8M0 scales; one 32-wide chunk is exactly one scale block.
// Scales outside [2, 252] (results that are not normal bfloat16) raise
// MCPU_DEVERR_MXFP4 and contribute zero.
template <> struct WSrc<bf16, 1> {
  struct Raw {
    uint32_t codes, scale;
  };
  const uint32_t* cp;
  const uint8_t* sp;
  __device__ __forceinline__ void init(const Gemm& P, int grp, int row, int kg) {
    cp = reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint8_t*>(P.w) + grp * P.w_group_stride +
                                           (int64_t)row * (P.k / 2)) + kg;
    sp = P.w_scales + grp * (P.w_group_stride / 16) + (int64_t)row * (P.k / 32);
  }
  __device__ __forceinline__ void fetch(Raw& r, int c) const {
    r.codes = cp[c * 4];
    r.scale = sp[c];
  }
  __device__ __forceinline__ Frag<bf16> frag(const Raw& r, bool& bad) const {
    const bool ok = r.scale >= 2u && r.scale <= 252u;
    bad = bad || !ok;
    const uint32_t codes = ok ? r.codes : 0u;
    const int32_t dexp = ((int32_t)r.scale - 127) * 128;
    Frag<bf16> f;
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = e2m1_to_bf16((codes >> (8 * i)) & 0xFu, dexp) | (e2m1_to_bf16((codes >> (8 * i + 4)) & 0xFu, dexp) << 16);
    f.v = make_uint4(w[0], w[1], w[2], w[3]);
    return f;
  }
};

// Pipeline depth: chunks whose fragments are in flight per wavefront, sized so
// the fragment ring stays within about 64 registers.
template <typename T, int NB, int MB>
struct Depth {
  static constexpr int frag_regs = sizeof(Frag<T>) / 4;
  static constexpr int v = (64 / ((NB + MB) * frag_regs)) < 2 ? 2 : (64 / ((NB + MB) * frag_regs)) > 8 ? 8
                                                                   : (64 / ((NB + MB) * frag_regs));
};

template <typename T, int WN, int WK, int NB, int MB, int EPI, int U = Depth<T, NB, MB>::v, int WF = 0>
__global__ __launch_bounds__(64 * WN * WK) void gemm_kernel(Gemm P) {
  constexpr int NT = 16 * WN * NB;  // weight rows per workgroup
  constexpr int LD = NT + 1;
  __shared__ float cr[MB * 16 * LD];
  const int lane = lane_id(), wave = uniform(threadIdx.x >> 6);
  const int wn = wave % WN, wk = wave / WN;
  const int n_tiles = P.n / NT;
  const int tile = blockIdx.x % n_tiles, grp = blockIdx.x / n_tiles;
  int r0 = 0, r1 = P.n_rows;
  if (P.group_off) {
    r0 = P.group_off[grp];
    r1 = P.group_off[grp + 1];
  }
  r0 = uniform(r0);
  r1 = uniform(r1);
  if (r1 <= r0) return;

  const int nl = lane & 15, kg = lane >> 4;
  using Src = WSrc<T, WF>;
  Src ws[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) ws[nb].init(P, grp, block_row<EPI>(P, (tile * WN + wn) * NB + nb, nl), kg);
  bool bad_scale = false;
  const int nC = P.k >> 5;
  const int c0 = wk * nC / WK, c1 = (wk + 1) * nC / WK;

  for (int m0 = r0; m0 < r1; m0 += MB * 16) {
    const int mrows = min(MB * 16, r1 - m0);
    const int amb = (mrows + 15) >> 4;
    const T* xp[MB];
    bool xv[MB];
    const int src0 = P.row_src ? P.row_src[r0] : r0;  // a valid row for lanes past the group
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int row = m0 + mb * 16 + nl;
      xv[mb] = row < r1;
      const int src = xv[mb] ? (P.row_src ? P.row_src[row] : row) : src0;
      xp[mb] = reinterpret_cast<const T*>(P.x) + (int64_t)src * P.k + 8 * kg;
    }
    f32x4 acc[NB][MB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) acc[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // U-deep ring of fragments: while chunk c is multiplied, chunks c+1 ..
    // c+U-1 are in flight and chunk c+U is issued into its slot. The steady
    // state has no branches (chunk indices are clamped, rows past the group
    // are zeroed by a select) so the loads stay in flight across iterations.
    const int nck = c1 - c0;
    auto kloop = [&](auto amb_c) {
      constexpr int AMB = decltype(amb_c)::value;
      typename Src::Raw wa[U][NB];
      Frag<T> xb[U][AMB];
      auto fetch = [&](int slot, int i) {
        const int c = c0 + min(i, nck - 1);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) ws[nb].fetch(wa[slot][nb], c);
#pragma unroll
        for (int mb = 0; mb < AMB; ++mb) {
          xb[slot][mb].load(xp[mb] + c * 32);
          xb[slot][mb].keep_if(xv[mb]);
        }
      };
      auto compute = [&](int slot) {
        Frag<T> a[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) a[nb] = ws[nb].frag(wa[slot][nb], bad_scale);
#pragma unroll
        for (int mb = 0; mb < AMB; ++mb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) acc[nb][mb] = mma32(a[nb], xb[slot][mb], acc[nb][mb]);
      };
#pragma unroll
      for (int u = 0; u < U; ++u) fetch(u, u);
      int i = 0;
      for (; i + U <= nck; i += U) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          compute(u);
          fetch(u, i + u + U);
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (i + u < nck) compute(u);
    };
    if (c1 > c0) {
      if constexpr (MB >= 1) if (amb == 1) kloop(std::integral_constant<int, 1>{});
      if constexpr (MB >= 2) if (amb == 2) kloop(std::integral_constant<int, 2 <= MB ? 2 : 1>{});
      if constexpr (MB >= 3) if (amb == 3) kloop(std::integral_constant<int, 3 <= MB ? 3 : 1>{});
      if constexpr (MB >= 4) if (amb == 4) kloop(std::integral_constant<int, 4 <= MB ? 4 : 1>{});
      if constexpr (MB > 4) if (amb > 4) kloop(std::integral_constant<int, MB>{});
    }

    if (bad_scale) set_error(P.err, 16);

    // sum the WK partial tiles into LDS in wavefront order (deterministic)
    for (int k = 0; k < WK; ++k) {
      if (wk == k) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int n = (wn * NB + nb) * 16 + 4 * kg + r, m = mb * 16 + nl;
              if (k == 0) cr[m * LD + n] = acc[nb][mb][r];
              else cr[m * LD + n] += acc[nb][mb][r];
            }
      }
      __syncthreads();
    }
    epilogue<T, EPI>(P, cr, LD, m0, mrows, tile * WN * NB, WN * NB, grp);
    __syncthreads();
  }
}

template <typename T, int WN, int WK, int NB, int MB, int U = Depth<T, NB, MB>::v, int WF = 0>
hipError_t gemm_launch_cfg(const Gemm& g, hipStream_t s) {
  constexpr int NT = 16 * WN * NB;
  if (g.n % NT) return hipErrorInvalidValue;
  dim3 grid((g.n / NT) * g.n_groups), block(64 * WN * WK);
  switch (g.epi) {
    case EPI_QKV: hipLaunchKernelGGL((gemm_kernel<T, WN, WK, NB, MB, EPI_QKV, U, WF>), grid, block, 0, s, g); break;
    case EPI_RESIDUAL: hipLaunchKernelGGL((gemm_kernel<T, WN, WK, NB, MB, EPI_RESIDUAL, U, WF>), grid, block, 0, s, g); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_kernel<T, WN, WK, NB, MB, EPI_SWIGLU, U, WF>), grid, block, 0, s, g); break;
    default: hipLaunchKernelGGL((gemm_kernel<T, WN, WK, NB, MB, EPI_BIAS, U, WF>), grid, block, 0, s, g); break;
  }
  return hipGetLastError();
}

// Tiling choice (this kernel serves the shapes the weight-slab and tiled
// kernels do not take: fp32 layers, 65-127-row dense projections, reductions
// that are not a multiple of 64). Grouped (expert) GEMMs have many slabs, so
// each wavefront streams whole rows (WK = 1); dense projections have few, so
// four wavefronts split the reduction to keep loads in flight. Deeper rings
// measured no faster for the 16-64-row dense shapes.
template <typename T>
static hipError_t gemm_dispatch(const Gemm& g, hipStream_t s) {
  const int mb = (g.max_rows_per_group + 15) / 16;
  if (g.n_groups > 1) {
    if (mb <= 4) return gemm_launch_cfg<T, 2, 1, 2, 4, 2>(g, s);
    return gemm_launch_cfg<T, 2, 2, 2, 8, 2>(g, s);
  }
  if (mb <= 4) return gemm_launch_cfg<T, 1, 4, 2, 4, 1>(g, s);
  return gemm_launch_cfg<T, 1, 4, 2, 8, 1>(g, s);
}

// MXFP4 expert weights (bf16 activations): the fragment ring holds raw codes
// (2 registers per chunk), decoded to bfloat16 right before each product.
static hipError_t gemm_dispatch_mxfp4(const Gemm& g, hipStream_t s) {
  const int mb = (g.max_rows_per_group + 15) / 16;
  if (g.k % 32 || !g.w_scales) return hipErrorInvalidValue;
  if (mb <= 4) return gemm_launch_cfg<bf16, 2, 1, 2, 4, 4, 1>(g, s);
  return gemm_launch_cfg<bf16, 2, 2, 2, 8, 2, 1>(g, s);
}

hipError_t launch_gemm(int dtype, int expert_fmt, const Gemm& g, hipStream_t s) {
  if (g.n_groups == 0 || g.n == 0) return hipSuccess;
  if (expert_fmt == 2) return dtype == 1 ? launch_gemm_mx(g, s) : hipErrorNotSupported;  // MXFP8 x MXFP4
  if (g.epi == EPI_LOGITS) {  // the slab, tiled and pipelined kernels carry the logits epilogue
    if (slab_gemm_applies(dtype, expert_fmt, g)) return launch_gemm_slab(expert_fmt, g, s);
    if (tiled_gemm_applies(dtype, g)) return launch_gemm_tiled(expert_fmt, g, s);
    return hipErrorNotSupported;
  }
  if (slab_gemm_applies(dtype, expert_fmt, g)) return launch_gemm_slab(expert_fmt, g, s);
  if (tiled_gemm_applies(dtype, g)) return launch_gemm_tiled(expert_fmt, g, s);
  if (expert_fmt != 0) return dtype == 1 ? gemm_dispatch_mxfp4(g, s) : hipErrorNotSupported;
  return dtype == 0 ? gemm_dispatch<float>(g, s) : gemm_dispatch<bf16>(g, s);
}

}  // namespace mcpu
