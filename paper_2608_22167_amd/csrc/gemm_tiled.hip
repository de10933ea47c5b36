// LDS-tiled grouped GEMM for many token rows per weight matrix (gfx950, bf16).
//
// Once a weight matrix meets tens of token rows or more, streaming it through
// every wavefront (gemm.hip) re-reads the activations from L2 once per weight
// slab and runs out of matrix-core work per byte. Here a workgroup of four
// wavefronts owns one BM x BN output tile: token rows m0 .. m0 + BM - 1 of one
// group against weight rows n0 .. n0 + BN - 1 of that group's matrix. Per
// 64-wide slice of the reduction the workgroup stages the BM activation rows
// (gathered through row_src) and the BN weight rows in LDS, double buffered,
// and each wavefront multiplies a (BM/2) x (BN/2) quadrant out of LDS with the
// 16x16x32 bf16 matrix-core product while the next R slices are in flight
// in a ring of R register sets (deep rings for weight-streaming shapes, whose
// time goes into HBM latency). MXFP4 weights are decoded once, while they are staged, with the
// packed e2m1 -> bf16 conversion that applies the block scale (exact: every
// product of an e2m1 value and a scale in [2^-125, 2^125] is a normal
// bfloat16).
//
// Work items are (m-tile, n-tile) pairs over all groups; the per-group m-tile
// counts come from group_off on the device, so the host only bounds the grid.
// Within a group the items go in bands of GM m-tiles: a band walks the
// n-tiles, and each n-tile visits the band's m-tiles back to back, so a weight
// tile is fetched once per band and the band's activation tiles stay in L2.
// The item sequence is cut into eight contiguous ranges, one per XCD
// (workgroups are dealt to the XCDs round robin), so that reuse happens within
// one XCD's L2. The finished fp32 tile goes through LDS to the fused epilogue.
#include <type_traits>

#include "device.h"
#include "gemm_epilogue.h"
#include "kernels.h"

namespace mcpu {

// 16-byte staging registers as a native vector type: copies of HIP's uint4
// struct become memcpy calls that keep the register sets in scratch memory.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

// LDS plan of a BM x BN tile with BK-wide reduction slices. Rows are padded by
// 16 B (BK = 64: 144 B apart; BK = 32: 80 B apart), which spreads the eight
// 16-byte fragment reads a cycle serves over all banks. The fp32 output tile
// reuses the operand buffers, EP rows at a time.
template <int BM, int BN, int BK, int NTH>
struct TiledSmem {
  static constexpr int ldk = BK + 8;              // LDS row stride in bf16
  static constexpr int stage = (BM + BN) * ldk;   // bf16 elements per stage
  static constexpr int ab_bytes = 2 * stage * 2;
  static constexpr int c_ld = BN + 4;             // fp32 tile row stride
  static constexpr int EP = BM * c_ld * 4 <= ab_bytes ? BM : 64;  // output rows per epilogue pass
  static_assert(EP * c_ld * 4 <= ab_bytes, "an epilogue pass must fit the operand buffers");
  static constexpr int bytes = ab_bytes;
  static constexpr int cpr = BK / 8;              // 16-byte chunks per staged row
  static constexpr int rpp = NTH / cpr;           // rows one pass of the workgroup stages
};

// Staged weight rows: dense bf16 (16-byte chunks, BK / 8 per row and slice) ...
template <int BN, int BK, int WF, int NTH>
struct TiledW {
  static constexpr int cpr = BK / 8, rpp = NTH / cpr;
  static constexpr int J = BN / rpp;
  struct Regs {
    u32x4 r[J];
  };
  const bf16* src[J];
  static __device__ __forceinline__ int row(int tid, int j) { return tid / cpr + rpp * j; }
  __device__ __forceinline__ void init(const Gemm& P, int grp, const int* wrow, int tid) {
#pragma unroll
    for (int j = 0; j < J; ++j)
      src[j] = reinterpret_cast<const bf16*>(P.w) + grp * P.w_group_stride + (int64_t)wrow[j] * P.k +
               (tid % cpr) * 8;
  }
  template <bool NTL>
  __device__ __forceinline__ void fetch(Regs& g, int ks) const {
#pragma unroll
    for (int j = 0; j < J; ++j) g.r[j] = NTL ? ld_stream16(src[j] + ks * BK) : ld16(src[j] + ks * BK);
  }
  static __device__ __forceinline__ void store(const Regs& g, bf16* ws, int tid, bool&) {
#pragma unroll
    for (int j = 0; j < J; ++j) st16(ws + row(tid, j) * (BK + 8) + (tid % cpr) * 8, g.r[j]);
  }
};

// ... or MXFP4: per row and slice BK / 2 code bytes (BK / 32 scale blocks)
// and BK / 32 E8M0 scales; a thread stages one block of 32 weights per chunk.
template <int BN, int BK, int NTH>
struct TiledW<BN, BK, 1, NTH> {
  static constexpr int bpr = BK / 32;  // scale blocks per row and slice
  static constexpr int J = BN * bpr / NTH;
  static_assert(J >= 1 && BN * bpr % NTH == 0, "whole scale blocks per thread");
  struct Regs {
    u32x4 r[J];
    uint32_t s[J];
  };
  const uint8_t* csrc[J];
  const uint8_t* ssrc[J];
  static __device__ __forceinline__ int row(int tid, int j) { return (tid + NTH * j) / bpr; }
  static __device__ __forceinline__ int blk(int tid, int j) { return (tid + NTH * j) % bpr; }
  __device__ __forceinline__ void init(const Gemm& P, int grp, const int* wrow, int tid) {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      csrc[j] = reinterpret_cast<const uint8_t*>(P.w) + grp * P.w_group_stride + (int64_t)wrow[j] * (P.k / 2) +
                16 * blk(tid, j);
      ssrc[j] = P.w_scales + grp * (P.w_group_stride / 16) + (int64_t)wrow[j] * (P.k / 32) + blk(tid, j);
    }
  }
  template <bool NTL>
  __device__ __forceinline__ void fetch(Regs& g, int ks) const {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      g.r[j] = NTL ? ld_stream16(csrc[j] + ks * (BK / 2)) : ld16(csrc[j] + ks * (BK / 2));
      g.s[j] = ssrc[j][ks * bpr];
    }
  }
  static __device__ __forceinline__ void store(const Regs& g, bf16* ws, int tid, bool& bad) {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const bool ok = g.s[j] >= 2u && g.s[j] <= 252u;
      bad = bad || !ok;
      const float scale = __uint_as_float(ok ? g.s[j] << 23 : 127u << 23);
      const uint32_t w4[4] = {ok ? g.r[j][0] : 0u, ok ? g.r[j][1] : 0u, ok ? g.r[j][2] : 0u, ok ? g.r[j][3] : 0u};
      uint32_t o[16];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // byte b of word i holds weights 8i + 2b (low nibble) and 8i + 2b + 1
        o[4 * i + 0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w4[i], scale, 0));
        o[4 * i + 1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w4[i], scale, 1));
        o[4 * i + 2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w4[i], scale, 2));
        o[4 * i + 3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w4[i], scale, 3));
      }
      bf16* d = ws + row(tid, j) * (BK + 8) + 32 * blk(tid, j);
#pragma unroll
      for (int q = 0; q < 4; ++q) st16(d + 8 * q, u32x4{o[4 * q], o[4 * q + 1], o[4 * q + 2], o[4 * q + 3]});
    }
  }
};

template <int BM, int BN, int BK, int R, int NW, int EPI, int WF>
__global__ __launch_bounds__(NW * 64) void gemm_tiled_kernel(Gemm P) {
  static_assert(R == 1 || R % 2 == 0, "the unrolled ring must cover both LDS buffers");
  constexpr int UN = R == 1 ? 2 : R;  // loop unroll: a multiple of the ring and of the two buffers
  constexpr int NTH = NW * 64;
  using S = TiledSmem<BM, BN, BK, NTH>;
  constexpr int LDK = S::ldk;
  constexpr int GM = BM == 64 ? 8 : BM == 128 ? 4 : 2;  // m-tiles per band: 2-3 MB of activations
  __shared__ __align__(16) unsigned char smem_raw[S::bytes];
  __shared__ int mt_start[TILE_MAXG + 1];
  bf16* smem = reinterpret_cast<bf16*>(smem_raw);
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  int grp, mt, tn;
  if (!tile_of_block<BM, BN, GM>(P, mt_start, grp, mt, tn)) return;
  const int gr0 = P.group_off ? P.group_off[grp] : 0;
  const int gr1 = P.group_off ? P.group_off[grp + 1] : P.n_rows;
  const int m0 = uniform(gr0 + mt * BM);
  const int mrows = min(BM, gr1 - m0);
  const int n0 = uniform(tn * BN), nrows = min(BN, P.n - n0);

  // activation rows this thread stages: tid / cpr + rpp j, chunk tid % cpr;
  // rows past the tile's end repeat its last row (their results are dropped)
  constexpr int XJ = BM / S::rpp;
  const bf16* xsrc[XJ];
#pragma unroll
  for (int j = 0; j < XJ; ++j) {
    const int row = m0 + min(tid / S::cpr + S::rpp * j, mrows - 1);
    const int src = P.row_src ? P.row_src[row] : row;
    xsrc[j] = reinterpret_cast<const bf16*>(P.x) + (int64_t)src * P.k + (tid % S::cpr) * 8;
  }
  using WL = TiledW<BN, BK, WF, NTH>;
  WL wl;
  {
    int wrow[WL::J];
#pragma unroll
    for (int j = 0; j < WL::J; ++j) {
      const int rr = min(WL::row(tid, j), nrows - 1);
      wrow[j] = block_row<EPI>(P, (n0 + rr) >> 4, rr & 15);
    }
    wl.init(P, grp, wrow, tid);
  }
  struct Regs {
    u32x4 x[XJ];
    typename WL::Regs w;
  };
  const int nk = P.k / BK;
  // slices past the end re-read the last one (branch-free; never staged for use)
  auto fetch = [&](Regs& g, int ks, auto NTL_) __attribute__((always_inline)) {
    ks = min(ks, nk - 1);
#pragma unroll
    for (int j = 0; j < XJ; ++j) g.x[j] = ld16(xsrc[j] + ks * BK);
    wl.template fetch<decltype(NTL_)::value>(g.w, ks);
  };
  bool bad_scale = false;
  auto stage = [&](const Regs& g, int buf) __attribute__((always_inline)) {
    bf16* xs = smem + buf * S::stage;
#pragma unroll
    for (int j = 0; j < XJ; ++j)
      st16(xs + (tid / S::cpr + S::rpp * j) * LDK + (tid % S::cpr) * 8, g.x[j]);
    WL::store(g.w, xs + BM * LDK, tid, bad_scale);
  };

  // wavefronts in 2 x NW/2: each owns BM/2 token rows and BN/(NW/2) weight rows
  constexpr int WN = BN / (NW / 2);
  const int wm = wave & 1, wn = wave >> 1;
  constexpr int MT = BM / 32, NT = WN / 16;  // 16-row tiles per wavefront
  f32x4 acc[NT][MT];
#pragma unroll
  for (int nb = 0; nb < NT; ++nb)
#pragma unroll
    for (int mb = 0; mb < MT; ++mb) acc[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int fr = lane & 15, fk = 8 * (lane >> 4);
  auto compute = [&](int buf) __attribute__((always_inline)) {
    const bf16* xs = smem + buf * S::stage + (wm * (BM / 2) + fr) * LDK + fk;
    const bf16* ws = smem + buf * S::stage + (BM + wn * WN + fr) * LDK + fk;
#pragma unroll
    for (int c = 0; c < BK / 32; ++c) {
      Frag<bf16> a[NT], b[MT];
#pragma unroll
      for (int nb = 0; nb < NT; ++nb) a[nb].load(ws + nb * 16 * LDK + 32 * c);
#pragma unroll
      for (int mb = 0; mb < MT; ++mb) b[mb].load(xs + mb * 16 * LDK + 32 * c);
#pragma unroll
      for (int nb = 0; nb < NT; ++nb)
#pragma unroll
        for (int mb = 0; mb < MT; ++mb) acc[nb][mb] = mma32(a[nb], b[mb], acc[nb][mb]);
    }
  };

  // Slice j is loaded into register set j % R and staged into LDS buffer j & 1.
  // While slice ks is multiplied out of LDS, slices ks + 1 .. ks + R are in
  // flight; afterwards slice ks + 1 is staged and its set refilled with slice
  // ks + 1 + R. The loop is unrolled R times so every set index is a
  // constant, and only the products are conditional (past the last slice the
  // loads are clamped and the staged copies never read), so the wait counts
  // at the loop head see one load order on every path. The scheduling
  // barriers keep the loads ahead of the products and the LDS writes, which
  // wait for their loads, behind them.
  // Expert launches: weight tiles of a group with one m-tile are read by this
  // workgroup alone, so they take streaming loads (see ld_stream16); a group
  // with more m-tiles shares them through L2, which streaming loads do not
  // fill, so those keep plain loads. The pipeline is instantiated for both,
  // so every load count is static (C3 gate/up 199 -> 191 us). One-matrix
  // launches keep one plain pipeline: the second costs registers (64 x 64
  // tiles: 124 -> 154 VGPRs, a wavefront per SIMD).
  auto pipeline = [&](auto NTL_) __attribute__((always_inline)) {
    Regs rs[R];
#pragma unroll
    for (int u = 0; u < R; ++u) {
      fetch(rs[u], u, NTL_);
      __builtin_amdgcn_sched_barrier(0);
    }
    stage(rs[0], 0);
    fetch(rs[0], R, NTL_);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    for (int ks = 0; ks < nk; ks += UN) {
#pragma unroll
      for (int u = 0; u < UN; ++u) {
        if (ks + u < nk) compute(u & 1);
        __builtin_amdgcn_sched_barrier(0);
        stage(rs[(u + 1) % R], (u + 1) & 1);
        fetch(rs[(u + 1) % R], ks + u + 1 + R, NTL_);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
      }
    }
  };
  constexpr bool EXPERT = EPI == EPI_SWIGLU || EPI == EPI_BIAS;
  if constexpr (EXPERT) {
    if (uniform(mt_start[grp + 1] - mt_start[grp]) == 1)
      pipeline(std::true_type{});
    else
      pipeline(std::false_type{});
  } else {
    pipeline(std::false_type{});
  }
  if constexpr (EPI == EPI_LOGITS && WN == LOGIT_SLOT) {
    // Vocabulary logits with one 64-column sampling slot per wavefront: each
    // lane holds, per 16-row tile mb, columns 16 nb + 4 (lane / 16) + r (nb, r
    // < 4) of row 16 mb + lane % 16, so a slot's record folds 16 values per
    // lane and then the four lanes of a row (two cross-lane steps), straight
    // from the product registers. Same record, draws and tie rule (lowest
    // column on equal values) as the LDS epilogue.
    LogitSlot* out = reinterpret_cast<LogitSlot*>(P.out);
    const int n_slots = (P.n + LOGIT_SLOT - 1) / LOGIT_SLOT;
    const int cb = n0 + wn * WN, c_end = n0 + nrows, gq = lane >> 4;
    const bool draw = !P.greedy;
    const float NEG = -__builtin_inff();
    int pos[MT], seq[MT], tgt[MT];
#pragma unroll
    for (int mb = 0; mb < MT; ++mb) {
      const int r = m0 + min(wm * (BM / 2) + 16 * mb + fr, mrows - 1);
      pos[mb] = draw ? P.row_pos[r] : 0;
      seq[mb] = draw ? P.row_seq[r] : 0;
      tgt[mb] = P.target ? P.target[r] : -1;
    }
#pragma unroll
    for (int mb = 0; mb < MT; ++mb) {
      float sv[NT][4];
      float mx = NEG, pert = NEG, sb = NEG, st = NEG;
      int bi = 0x7FFFFFFF;
#pragma unroll
      for (int nb = 0; nb < NT; ++nb) {
        const int c0 = cb + 16 * nb + 4 * gq;
        float gn[4] = {0.f, 0.f, 0.f, 0.f};
        if (draw && c0 < c_end) {
          const U32x4 rr = philox4x32_10(U32x4{(uint32_t)(c0 >> 2), (uint32_t)pos[mb], (uint32_t)seq[mb], LOGIT_RNG_TAG},
                                         (uint32_t)P.seed, (uint32_t)(P.seed >> 32));
          gn[0] = gumbel_of(rr.x); gn[1] = gumbel_of(rr.y); gn[2] = gumbel_of(rr.z); gn[3] = gumbel_of(rr.w);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {  // increasing columns: the first of equal values is the lowest
          const bool ok = c0 + r < c_end;
          sv[nb][r] = ok ? acc[nb][mb][r] * P.inv_temp : NEG;
          mx = fmaxf(mx, sv[nb][r]);
          const float pv = sv[nb][r] + gn[r];
          if (ok && pv > pert) { pert = pv; sb = sv[nb][r]; bi = c0 + r; }
          if (ok && c0 + r == tgt[mb]) st = sv[nb][r];
        }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      float sum = 0.f;
#pragma unroll
      for (int nb = 0; nb < NT; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          sum += cb + 16 * nb + 4 * gq + r < c_end ? __builtin_amdgcn_exp2f((sv[nb][r] - mx) * 1.44269504088896341f) : 0.f;
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        sum += __shfl_xor(sum, o, 64);
        const float p2 = __shfl_xor(pert, o, 64), s2 = __shfl_xor(sb, o, 64);
        const int i2 = __shfl_xor(bi, o, 64);
        if (p2 > pert || (p2 == pert && i2 < bi)) { pert = p2; sb = s2; bi = i2; }
        st = fmaxf(st, __shfl_xor(st, o, 64));
      }
      const int m = wm * (BM / 2) + 16 * mb + fr;
      if (gq == 0 && m < mrows && cb < c_end) {
        LogitSlot rec;
        rec.m = mx; rec.l = sum; rec.pert = pert; rec.s_best = sb; rec.idx = bi; rec.s_tgt = st;
        rec.pad[0] = rec.pad[1] = 0.f;
        out[(int64_t)(m0 + m) * n_slots + cb / LOGIT_SLOT] = rec;
      }
    }
    return;
  }
  __syncthreads();  // the fp32 tile below reuses the operand buffers
  if (bad_scale) set_error(P.err, 16);

  // acc[nb][mb][r] = C[m = wm*BM/2 + 16 mb + fr][n = wn*BN/2 + 16 nb + 4 (lane/16) + r];
  // the fp32 tile goes through LDS EP rows at a time
  float* cr = reinterpret_cast<float*>(smem_raw);
  const EpiBias eb = epilogue_bias<EPI>(P, n0 >> 4, nrows >> 4, grp);
#pragma unroll
  for (int e0 = 0; e0 < BM; e0 += S::EP) {
    if (e0 >= mrows) break;  // uniform
#pragma unroll
    for (int nb = 0; nb < NT; ++nb)
#pragma unroll
      for (int mb = 0; mb < MT; ++mb) {
        const int m = wm * (BM / 2) + mb * 16 + fr, n = wn * WN + nb * 16 + 4 * (lane >> 4);
        if (m >= e0 && m < e0 + S::EP)  // the same for all lanes of a 16-row tile
          *reinterpret_cast<float4*>(cr + (m - e0) * S::c_ld + n) =
              make_float4(acc[nb][mb][0], acc[nb][mb][1], acc[nb][mb][2], acc[nb][mb][3]);
      }
    __syncthreads();
    epilogue<bf16, EPI>(P, cr, S::c_ld, m0 + e0, min(S::EP, mrows - e0), n0 >> 4, nrows >> 4, grp, &eb);
    __syncthreads();
  }
}

template <int BM, int BN, int BK, int R, int NW, int WF>
static hipError_t tiled_launch(const Gemm& g, hipStream_t s) {
  const int64_t grid = tile_grid(g, BM, BN);
  if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
  dim3 gd((unsigned)grid), bd(NW * 64);
  switch (g.epi) {
    case EPI_QKV: hipLaunchKernelGGL((gemm_tiled_kernel<BM, BN, BK, R, NW, EPI_QKV, WF>), gd, bd, 0, s, g); break;
    case EPI_RESIDUAL: hipLaunchKernelGGL((gemm_tiled_kernel<BM, BN, BK, R, NW, EPI_RESIDUAL, WF>), gd, bd, 0, s, g); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_tiled_kernel<BM, BN, BK, R, NW, EPI_SWIGLU, WF>), gd, bd, 0, s, g); break;
    case EPI_LOGITS:  // vocabulary logits: bf16 weights
      if constexpr (WF == 0) {
        hipLaunchKernelGGL((gemm_tiled_kernel<BM, BN, BK, R, NW, EPI_LOGITS, WF>), gd, bd, 0, s, g);
        break;
      } else {
        return hipErrorNotSupported;
      }
    default: hipLaunchKernelGGL((gemm_tiled_kernel<BM, BN, BK, R, NW, EPI_BIAS, WF>), gd, bd, 0, s, g); break;
  }
  return hipGetLastError();
}

bool tiled_gemm_applies(int dtype, const Gemm& g) {
  if (dtype != 1 || g.k <= 0 || g.k % 64 || g.n % 16 || g.n_groups > TILE_MAXG || g.n_rows < TILED_MIN_TOTAL_ROWS) return false;
  return (int64_t)g.n_rows >= (int64_t)TILED_MIN_ROWS * g.n_groups;
}

// Tile choice by rows per group and the number of tiles a launch has: the
// pipelined 256 x 256 kernel (gemm_pipe.hip) once groups average 256 rows
// with two tiles per compute unit; else 128 x 128 tiles once they average 128
// rows with a few tiles per compute unit; 64-row tiles otherwise (less
// padding per group), 64 x 64 for a single dense matrix that would not fill
// the chip. The 64-row tiles of decode batches stage two slices ahead (four
// measured slower at batch 256).
hipError_t launch_gemm_tiled(int expert_fmt, const Gemm& g, hipStream_t s) {
  if (expert_fmt != 0 && !g.w_scales) return hipErrorInvalidValue;
  if (pipe_gemm_applies(1, g)) return launch_gemm_pipe(expert_fmt, g, s);
  const int64_t groups = g.group_off ? g.n_groups : 1;
  auto tiles = [&](int bm, int bn) { return ((int64_t)g.n_rows / bm + groups) * ((g.n + bn - 1) / bn); };
  const bool big = (int64_t)g.n_rows >= 128LL * g.n_groups && tiles(128, 128) >= 1024;
  if (expert_fmt != 0)
    return big ? tiled_launch<128, 128, 64, 2, 4, 1>(g, s) : tiled_launch<64, 128, 64, 4, 4, 1>(g, s);
  if (big) return tiled_launch<128, 128, 64, 2, 4, 0>(g, s);
  if (tiles(64, 128) < 512) return tiled_launch<64, 64, 64, 4, 4, 0>(g, s);
  // 128-wide n-tiles, or 160-wide where those divide n and 128-wide ones
  // do not (2880 = 18 x 160: the expert down projection, whose last 128-wide
  // tile would be half empty; 114 -> 109 us at batch 256). The 128-wide
  // tiles run eight wavefronts (2 x 4, 32 weight rows each): more loads in
  // flight per CU than four (gate/up 201 -> 199 us at batch 256); 160 rows do
  // not split four ways into 16-row MFMA tiles.
  if (g.n % 128 && g.n % 160 == 0) return tiled_launch<64, 160, 64, 2, 4, 0>(g, s);
  return tiled_launch<64, 128, 64, 2, 8, 0>(g, s);
}

}  // namespace mcpu
