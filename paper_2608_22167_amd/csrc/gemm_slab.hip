// Weight-streaming slabs for grouped GEMMs with up to about a hundred token
// rows per weight matrix (gfx950, bf16 activations, bf16 or MXFP4 weights):
// the expert projections of decode batches of up to a few thousand tokens.
//
// There each weight byte meets only a few dozen token rows, so the bound is
// HBM, and the kernel's job is to keep enough weight bytes in flight. A
// workgroup of four wavefronts owns one work item: up to SMT token rows of one
// group (64; 128 for MXFP4 groups of over 32 rows on average, so that a group
// just past 64 rows decodes its weights once) against NS weight rows. Each
// wavefront streams its NS / 4 weight rows straight from global memory into
// registers, already in matrix-core operand order, through a ring of RC
// reduction chunks (128 indices each), so weights never pass through LDS; the
// group's token rows, shared by the four wavefronts (and by all the group's
// slabs, so they come from L2), are staged per chunk through double-buffered
// LDS from one register set.
//
// MXFP4 weights are loaded 16 code bytes (32 weights) per lane: lane group g
// of a 16-row fragment holds indices 32 g .. 32 g + 31 of the chunk, and
// product s of the chunk takes indices 32 g + 8 s .. + 7 from every group,
// the token-row fragments reading the same indices. A chunk's 32-weight blocks
// then coincide with the lane groups, one E8M0 scale per lane, decoded in
// registers with the packed e2m1 -> bf16 conversion (exact, as in the LDS
// kernels). bf16 weights use the plain fragment order.
//
// Token rows sit in LDS as [half chunk][SMT rows][128 B] with 16-byte chunk c
// of row r in slot c ^ (r & 7): the fragment reads of 16 rows and the 8-lane
// staging writes of one row both cover all bank groups. Reductions that end
// in half a chunk (k % 128 == 64) skip the missing half: bf16 products are
// not issued, MXFP4 weights of the missing half are zero.
#include <algorithm>
#include <type_traits>

#include "device.h"
#include "gemm_epilogue.h"
#include "kernels.h"

namespace mcpu {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int BUF_D3 = 0x00020000;  // raw buffer descriptor word 3 (gfx9 family)
constexpr int AUX_NT = 2;           // buffer-load cache policy: the non-temporal bit

constexpr int SM = 64;              // token rows per item (split projections; experts: 64 or 128)
constexpr int SKC = 128;            // reduction indices per chunk
constexpr int SPLIT_MAX_K = 16;     // most reduction splits of one tile

__device__ __forceinline__ f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                  0, 0, 0);
}

// Weight side of one wavefront: NF 16-row fragments.
template <int NF, int WF>
struct SlabW;

// bf16: per chunk and fragment four 16-byte loads (products 0..3 of the
// chunk), from row-major weights (each load: 16 rows x 64 bytes) or from the
// streaming-order copy (each load: one contiguous KiB, whole cache lines)
template <int NF>
struct SlabW<NF, 0> {
  struct Regs {
    u32x4 f[NF][4];
  };
  __amdgpu_buffer_rsrc_t rs;
  uint32_t vo[NF];
  int kstep, tstep;  // bytes between chunks and between products of a row
  __device__ __forceinline__ void init(const Gemm& P, int grp, const int* wrow, int g) {
    const uint8_t* base;
    if (P.w_packed) {
      const int nkc = (P.k + SKC - 1) / SKC;
      base = reinterpret_cast<const uint8_t*>(P.w_packed) + (int64_t)grp * (P.n / 16) * nkc * 4096;
#pragma unroll
      for (int nb = 0; nb < NF; ++nb)
        vo[nb] = (uint32_t)(wrow[nb] >> 4) * (uint32_t)(nkc * 4096) + 16 * (wrow[nb] & 15) + 256 * g;
      kstep = 4096;
      tstep = 1024;
    } else {
      base = reinterpret_cast<const uint8_t*>(P.w) + (int64_t)grp * P.w_group_stride * 2;
#pragma unroll
      for (int nb = 0; nb < NF; ++nb) vo[nb] = (uint32_t)wrow[nb] * (uint32_t)(P.k * 2) + 16 * g;
      kstep = SKC * 2;
      tstep = 64;
    }
    rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(base), 0, 0x7FFFFFFF, BUF_D3);
  }
  template <int AUX>
  __device__ __forceinline__ void fetch(Regs& r, int kc, int nsteps) const {
#pragma unroll
    for (int nb = 0; nb < NF; ++nb)
#pragma unroll
      for (int t = 0; t < 4; ++t)
        r.f[nb][t] = __builtin_amdgcn_raw_buffer_load_b128(rs, vo[nb], uniform(kc * kstep + tstep * min(t, nsteps - 1)), AUX);
  }
  struct Dec {};
  __device__ __forceinline__ void prepare(const Regs&, Dec&, uint32_t&, uint32_t) const {}
  // fragment of product t
  __device__ __forceinline__ u32x4 frag(const Regs& r, const Dec&, int nb, int t) const { return r.f[nb][t]; }
};

// MXFP4: per chunk and fragment one 16-byte code load and one scale byte
template <int NF>
struct SlabW<NF, 1> {
  struct Regs {
    u32x4 c[NF];
    uint32_t s[NF];
  };
  __amdgpu_buffer_rsrc_t rc, rsc;
  uint32_t vo[NF], so[NF];
  int g;
  __device__ __forceinline__ void init(const Gemm& P, int grp, const int* wrow, int g_) {
    g = g_;
    const uint8_t* cb = reinterpret_cast<const uint8_t*>(P.w) + (int64_t)grp * P.w_group_stride;
    const uint8_t* sb = P.w_scales + (int64_t)grp * (P.w_group_stride / 16);
    rc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(cb), 0, 0x7FFFFFFF, BUF_D3);
    rsc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(sb), 0, 0x7FFFFFFF, BUF_D3);
#pragma unroll
    for (int nb = 0; nb < NF; ++nb) {
      vo[nb] = (uint32_t)wrow[nb] * (uint32_t)(P.k / 2) + 16 * g;
      so[nb] = (uint32_t)wrow[nb] * (uint32_t)(P.k / 32) + g;
    }
  }
  template <int AUX>
  __device__ __forceinline__ void fetch(Regs& r, int kc, int nsteps) const {
    // in a half chunk, lane groups 2 and 3 read the first half again (their
    // weights are zeroed when decoded)
    const int off = nsteps == 4 ? 0 : -2 * (g >> 1);
#pragma unroll
    for (int nb = 0; nb < NF; ++nb) {
      r.c[nb] = __builtin_amdgcn_raw_buffer_load_b128(rc, vo[nb] + 16 * off, uniform(kc * (SKC / 2)), AUX);
      r.s[nb] = __builtin_amdgcn_raw_buffer_load_b8(rsc, so[nb] + off, uniform(kc * (SKC / 32)), 0);
    }
  }
  // per chunk and fragment: the scale as a float and a mask that zeroes the
  // codes of a rejected scale or of a missing half chunk (keep)
  struct Dec {
    float scale[NF];
    uint32_t mask[NF];
  };
  __device__ __forceinline__ void prepare(const Regs& r, Dec& d, uint32_t& bad, uint32_t keep) const {
#pragma unroll
    for (int nb = 0; nb < NF; ++nb) {
      const uint32_t sc = r.s[nb];
      const bool ok = sc >= 2u && sc <= 252u;
      bad |= ok ? 0u : 1u;
      d.scale[nb] = __uint_as_float(ok ? sc << 23 : 127u << 23);
      d.mask[nb] = ok ? keep : 0u;
    }
  }
  __device__ __forceinline__ u32x4 frag(const Regs& r, const Dec& d, int nb, int s) const {
    const uint32_t w = r.c[nb][s] & d.mask[nb];
    const float scale = d.scale[nb];
    return u32x4{__builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, scale, 0)),
                 __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, scale, 1)),
                 __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, scale, 2)),
                 __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, scale, 3))};
  }
};

template <int NS, int WF, int RC, int EPI, bool SPLIT, int SMT, int NX, bool NTW>
__global__ __launch_bounds__(256, 2) void gemm_slab_kernel(Gemm P) {
  static_assert(SMT == 64 || SMT == 128, "items of 64 or 128 token rows");
  static_assert(!SPLIT || SMT == SM, "split tiles have 64 token rows");
  constexpr int NF = NS / 64;        // weight fragments per wavefront
  constexpr int MB = SMT / 16;       // token-row fragments per item
  constexpr int XR = SMT / 32;       // token rows each thread stages
  constexpr int CLD = NS + 4;        // fp32 tile row stride
  constexpr int SXHALF = SMT * 128;  // bytes of a staged half chunk (SMT rows x 64 indices)
  constexpr int SXSTAGE = 2 * SXHALF;
  constexpr int SMEM = 2 * SXSTAGE > SMT * CLD * 4 ? 2 * SXSTAGE : SMT * CLD * 4;
  __shared__ __align__(16) unsigned char smem[SMEM];
  __shared__ int mt_start[TILE_MAXG + 1];
  __shared__ int row_start[TILE_MAXG + 1];
  __shared__ int last_split;
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  const int fr = lane & 15, g = lane >> 4;

  // SPLIT: one matrix; block = tile * k_splits + split, tiles m-major
  int grp = 0, mt, tn, tile = 0, ks = 0;
  if constexpr (SPLIT) {
    const int ntn = (P.n + NS - 1) / NS;
    tile = uniform((int)blockIdx.x / P.k_splits);
    ks = uniform((int)blockIdx.x % P.k_splits);
    mt = tile / ntn;
    tn = tile % ntn;
  } else if (!tile_of_block<SMT, NS, 1>(P, mt_start, grp, mt, tn, row_start)) {
    return;
  }
  const int n0 = uniform(tn * NS), nrows = min(NS, P.n - n0);
  const int nk = (P.k + SKC - 1) / SKC;
  const int tail_steps = (P.k % SKC) ? (P.k % SKC) / 32 : 4;
  // this workgroup's chunks: kb .. kb + nkl - 1
  const int kb = SPLIT ? uniform(ks * nk / P.k_splits) : 0;
  const int nkl = SPLIT ? uniform((ks + 1) * nk / P.k_splits) - kb : nk;

  // weight rows of this wavefront: n0 + NS/4 * wave + 16 nb + fr (clamped; dropped)
  SlabW<NF, WF> wl;
  {
    int wrow[NF];
#pragma unroll
    for (int nb = 0; nb < NF; ++nb) {
      const int rr = min((NS / 4) * wave + 16 * nb + fr, nrows - 1);
      const int blk = (n0 + rr) >> 4, nl = rr & 15;
      wrow[nb] = EPI == EPI_QKV ? block_row<EPI_QKV>(P, blk, nl) : blk * 16 + nl;
    }
    wl.init(P, grp, wrow, g);
  }
  // The group's rows come from LDS; the source row of this thread's staged
  // token row is requested first and waited for only after the first RC
  // chunks of weights have been requested (loads complete in order), so that
  // its latency overlaps the start of the weight stream.
  const int gr0 = P.group_off ? row_start[grp] : 0;
  const int gr1 = P.group_off ? row_start[grp + 1] : P.n_rows;
  const int m0 = uniform(gr0 + mt * SMT);
  const int mrows = min(SMT, gr1 - m0);
  const int mbs = uniform((mrows + 15) >> 4);  // token-row fragments holding rows
  const int xr = tid >> 3, xc = tid & 7;
  int src[XR];
#pragma unroll
  for (int j = 0; j < XR; ++j) {
    const int xrow = m0 + min(xr + 32 * j, mrows - 1);
    src[j] = P.row_src ? P.row_src[xrow] : xrow;
  }
  typename SlabW<NF, WF>::Regs wr[RC];
  // weights of this workgroup's chunk i (clamped to its last)
  auto wfetch = [&](typename SlabW<NF, WF>::Regs& r, int i) __attribute__((always_inline)) {
    const int kc = kb + min(i, nkl - 1);
    wl.template fetch<NTW ? AUX_NT : 0>(r, kc, kc == nk - 1 ? tail_steps : 4);
  };
  if constexpr (NX == 1) {
#pragma unroll
    for (int u = 0; u < RC; ++u) {
      wfetch(wr[u], u);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // token-row staging: thread t stages rows t / 8 + 32 j (j < SMT / 32),
  // 16-byte chunk t % 8 of both half chunks, so that eight lanes read one
  // whole 128-byte line per load (2-3% faster on the projections than pieces
  // strided over two loads); rows past the end repeat the last row (dropped)
  uint32_t xvo[XR];
#pragma unroll
  for (int j = 0; j < XR; ++j) xvo[j] = (uint32_t)src[j] * (uint32_t)(P.k * 2) + 16 * xc;
  const uint8_t* xbase = reinterpret_cast<const uint8_t*>(P.x);
  const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(xbase), 0, 0x7FFFFFFF, BUF_D3);
  struct XRegs {
    u32x4 v[XR][2];  // [row][half]
  };
  auto xfetch = [&](XRegs& r, int i) __attribute__((always_inline)) {
    const int kc = kb + min(i, nkl - 1);
    // a half chunk past k re-reads the first half (never multiplied)
    const int h1 = (kc == nk - 1 && tail_steps < 4) ? 0 : 128;
#pragma unroll
    for (int j = 0; j < XR; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        r.v[j][h] = __builtin_amdgcn_raw_buffer_load_b128(xrs, xvo[j] + (h ? h1 : 0), uniform(kc * SKC * 2), 0);
  };
  auto xstore = [&](const XRegs& r, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < XR; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        *reinterpret_cast<u32x4*>(smem + buf * SXSTAGE + h * SXHALF + (xr + 32 * j) * 128 + 16 * (xc ^ (xr & 7))) =
            r.v[j][h];
  };
  XRegs xs[NX];
  // Weights of chunk i sit in register set i % RC, token rows in set i % NX.
  // With one token-row set (the grouped launches: their first token rows wait
  // for the gathered row index, after RC chunks of weights are requested),
  // chunk i's token rows are requested two chunks ahead. With NX = RC (the
  // one-matrix launches, whose token rows need no index) they are requested
  // with the weights, RC chunks ahead and before them (2-4% faster there;
  // rings deeper than two chunks were slower).
  if constexpr (NX > 1) {
#pragma unroll
    for (int u = 0; u < RC; ++u) {
      wfetch(wr[u], u);
      xfetch(xs[u], u);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // token-row fragment mb of product t (bf16 order) or s (MXFP4 order)
  auto xfrag = [&](int buf, int mb, int t) __attribute__((always_inline)) {
    int h, c8;
    if (WF == 0) {
      h = t >> 1;
      c8 = 4 * (t & 1) + g;
    } else {
      h = g >> 1;
      c8 = 4 * (g & 1) + t;
    }
    return *reinterpret_cast<const u32x4*>(smem + buf * SXSTAGE + h * SXHALF + (16 * mb + fr) * 128 +
                                           16 * (c8 ^ (fr & 7)));
  };

  f32x4 acc[NF][MB];
#pragma unroll
  for (int nb = 0; nb < NF; ++nb)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint32_t bad_scale = 0;

  // Chunk kc: weights from register set kc % RC, token rows from LDS buffer
  // kc & 1; afterwards chunk kc + 1's token rows are staged from their
  // registers, which then take chunk kc + 1 + NX's, ahead of the weights of
  // chunk kc + RC. Unrolled over RC (even, a multiple of NX) so the set
  // indices are constants; only the products are conditional. The loop is
  // instantiated per count of token-row fragments holding rows (MBS).
  static_assert(RC % 2 == 0, "the unrolled ring must cover both LDS buffers");
  static_assert(NX == 1 || NX == RC, "one token-row set, or one per weight set");
  if constexpr (NX == 1) xfetch(xs[0], 0);
  xstore(xs[0], 0);
  xfetch(xs[0], NX);
  __syncthreads();
  // MXFP4 in a half chunk: lane groups 2 and 3 hold no indices
  const uint32_t keep_tail = (WF == 1 && tail_steps < 4 && g >= 2) ? 0u : ~0u;
  auto run = [&](auto MBS_) __attribute__((always_inline)) {
    constexpr int MBS = decltype(MBS_)::value;
    for (int kc0 = 0; kc0 < nkl; kc0 += RC) {
#pragma unroll
      for (int u = 0; u < RC; ++u) {
        const int kc = kc0 + u;
        const int buf = u & 1;
        if (kc < nkl) {
          const bool tail = kb + kc == nk - 1;
          const int nsteps = tail ? tail_steps : 4;
          typename SlabW<NF, WF>::Dec dec;
          wl.prepare(wr[u], dec, bad_scale, tail ? keep_tail : ~0u);
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            if (WF == 0 && t >= nsteps) break;  // bf16: missing half chunk
            u32x4 xf[MBS];
#pragma unroll
            for (int mb = 0; mb < MBS; ++mb) xf[mb] = xfrag(buf, mb, t);
#pragma unroll
            for (int nb = 0; nb < NF; ++nb) {
              const u32x4 wf = wl.frag(wr[u], dec, nb, t);
#pragma unroll
              for (int mb = 0; mb < MBS; ++mb) acc[nb][mb] = mfma_bf16(wf, xf[mb], acc[nb][mb]);
            }
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        xstore(xs[(u + 1) % NX], buf ^ 1);
        xfetch(xs[(u + 1) % NX], kc + 1 + NX);
        wfetch(wr[u], kc + RC);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
      }
    }
  };
  switch (mbs) {
    case 1: run(std::integral_constant<int, 1>{}); break;
    case 2: run(std::integral_constant<int, 2>{}); break;
    case 3: run(std::integral_constant<int, 3>{}); break;
    case 4: run(std::integral_constant<int, 4>{}); break;
    default:
      if constexpr (MB > 4) {
        switch (mbs) {
          case 5: run(std::integral_constant<int, 5>{}); break;
          case 6: run(std::integral_constant<int, 6>{}); break;
          case 7: run(std::integral_constant<int, 7>{}); break;
          default: run(std::integral_constant<int, MB>{}); break;
        }
      }
      break;
  }
  if (bad_scale) set_error(P.err, 16);

  if constexpr (SPLIT) {
    if (P.k_splits > 1) {
      // This split's partial tile, in thread order ([nb][mb][thread], 16
      // bytes each); the last split of the tile to arrive sums all of them in
      // split order, so the result does not depend on the arrival order.
      // Partials are stored and loaded at device scope (SC1: coherent across
      // the XCDs' L2 caches without a cache-wide write-back or invalidate);
      // the stores are complete (vmcnt 0) before the arrival is counted.
      constexpr int PT = NF * MB * 256 * 16;  // bytes per partial tile
      constexpr int SC1 = 16;
      const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(
          reinterpret_cast<uint8_t*>(P.part) + (int64_t)tile * P.k_splits * PT, 0, 0x7FFFFFFF, BUF_D3);
#pragma unroll
      for (int nb = 0; nb < NF; ++nb)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          if (mb < mbs)
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[nb][mb]), prs,
                                                   ((nb * 4 + mb) * 256 + tid) * 16, ks * PT, SC1);
      __builtin_amdgcn_s_waitcnt(0xF70);  // vmcnt(0)
      __syncthreads();
      if (tid == 0)
        last_split = __hip_atomic_fetch_add(P.part_cnt + tile, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                     P.k_splits - 1;
      __syncthreads();
      if (!last_split) return;
      // all partials of a fragment in flight at once, then added in order
#pragma unroll
      for (int nb = 0; nb < NF; ++nb)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          if (mb < mbs) {
            const uint32_t vo = ((nb * 4 + mb) * 256 + tid) * 16;
            u32x4 v[SPLIT_MAX_K];
#pragma unroll
            for (int j = 0; j < SPLIT_MAX_K; ++j)
              if (j < P.k_splits) v[j] = __builtin_amdgcn_raw_buffer_load_b128(prs, vo, j * PT, SC1);
            f32x4 sum = __builtin_bit_cast(f32x4, v[0]);
#pragma unroll
            for (int j = 1; j < SPLIT_MAX_K; ++j)
              if (j < P.k_splits) sum += __builtin_bit_cast(f32x4, v[j]);
            acc[nb][mb] = sum;
          }
      if (tid == 0) __hip_atomic_store(P.part_cnt + tile, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }

  // acc[nb][mb][r] = C[m = 16 mb + fr][n = NS/4 * wave + 16 nb + 4 g + r]
  float* cr = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int nb = 0; nb < NF; ++nb)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int n = (NS / 4) * wave + 16 * nb + 4 * g;
      *reinterpret_cast<float4*>(cr + (16 * mb + fr) * CLD + n) =
          make_float4(acc[nb][mb][0], acc[nb][mb][1], acc[nb][mb][2], acc[nb][mb][3]);
    }
  __syncthreads();
  epilogue<bf16, EPI>(P, cr, CLD, m0, mrows, n0 >> 4, nrows >> 4, grp);
}

template <int NS, int WF, int RC, bool SPLIT, int SMT = SM, int NX = 1, bool NTW = false>
hipError_t slab_launch(const Gemm& g, hipStream_t s, int64_t grid) {
  if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
  dim3 gd((unsigned)grid), bd(256);
  switch (g.epi) {
    case EPI_QKV: hipLaunchKernelGGL((gemm_slab_kernel<NS, WF, RC, EPI_QKV, SPLIT, SMT, NX, NTW>), gd, bd, 0, s, g); break;
    case EPI_RESIDUAL: hipLaunchKernelGGL((gemm_slab_kernel<NS, WF, RC, EPI_RESIDUAL, SPLIT, SMT, NX, NTW>), gd, bd, 0, s, g); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_slab_kernel<NS, WF, RC, EPI_SWIGLU, SPLIT, SMT, NX, NTW>), gd, bd, 0, s, g); break;
    case EPI_LOGITS:  // vocabulary logits: bf16 weights, one reduction pass
      if constexpr (WF == 0 && !SPLIT) {
        hipLaunchKernelGGL((gemm_slab_kernel<NS, WF, RC, EPI_LOGITS, SPLIT, SMT, NX, NTW>), gd, bd, 0, s, g);
        break;
      } else {
        return hipErrorNotSupported;
      }
    default: hipLaunchKernelGGL((gemm_slab_kernel<NS, WF, RC, EPI_BIAS, SPLIT, SMT, NX, NTW>), gd, bd, 0, s, g); break;
  }
  return hipGetLastError();
}

// Split plan of one matrix: 64-wide slabs, the reduction in up to four parts
// (at least two chunks each), as many as bring the launch near SPLIT_WG
// workgroups (none past 64 rows, where the tiles alone make hundreds). Measured on MI355X for 16-64 rows against the gpt-oss-20b
// projections (weights from HBM): 2880 x 4096 (45 slabs) in 14 us with four
// parts against 17 with two and 22 unsplit; 5120 x 2880 (80 slabs) in 18.5 us
// with two against 20.7 with four and 23 unsplit. Finer splits, 128-wide
// slabs or a split of 256-512-row tiles were slower (more partial traffic,
// shorter pipelines).
constexpr int NSPLIT = 64;
constexpr int SPLIT_K = 4;
constexpr int SPLIT_WG = 192;
struct SplitPlan {
  int tiles = 0, k_splits = 0;
};
SplitPlan split_plan(int n, int k, int n_rows) {
  SplitPlan p;
  if (n <= 0 || k <= 0 || n % 16 || k % 64 || n_rows <= 0 || n_rows > SLAB_WIDE_MAX_ROWS) return p;
  if ((int64_t)n * k * 2 >= (1LL << 31) || (int64_t)n_rows * k * 2 >= (1LL << 31)) return p;
  const int tiles = ((n_rows + SM - 1) / SM) * ((n + NSPLIT - 1) / NSPLIT);
  if (tiles > SPLIT_MAX_TILES) return p;
  const int nk = (k + SKC - 1) / SKC;
  p.tiles = tiles;
  const int want = (SPLIT_WG + tiles / 2) / tiles;  // SPLIT_WG / tiles, rounded
  p.k_splits = std::max(1, std::min({want, SPLIT_K, nk / 2, SPLIT_MAX_K}));
  if (n_rows > SPLIT_MAX_ROWS) p.k_splits = 1;  // no partial tiles are provided past 64 rows
  return p;
}

}  // namespace

size_t slab_split_part_floats(int n, int k, int n_rows) {
  const SplitPlan p = split_plan(n, k, n_rows);
  return (size_t)p.tiles * p.k_splits * SM * NSPLIT;
}

bool slab_gemm_applies(int dtype, int expert_fmt, const Gemm& g) {
  if (dtype != 1 || g.k <= 0 || g.k % 64 || g.n % 16 || g.n_groups > TILE_MAXG) return false;
  if (!g.group_off) {  // one matrix: a split reduction, or wide with its streaming-order copy
    if (expert_fmt != 0 || g.n_groups != 1 || !g.part || !g.part_cnt) return false;
    if (g.n_rows > SPLIT_MAX_ROWS && !(g.w_packed && g.n >= SLAB_WIDE_MIN_N)) return false;
    return split_plan(g.n, g.k, g.n_rows).tiles > 0;
  }
  // 32-bit buffer offsets: token rows from x itself, weights within one group
  const int64_t xr = g.x_rows > 0 ? g.x_rows : g.n_rows;
  if (xr * g.k * 2 >= (1LL << 31) || (int64_t)g.n * g.k * 2 >= (1LL << 31)) return false;
  if (g.w_packed && (expert_fmt != 0 || (int64_t)g.n * ((g.k + SKC - 1) / SKC) * 256 >= (1LL << 31))) return false;
  if (expert_fmt != 0) return (int64_t)g.n_rows <= (int64_t)SLAB_MAX_ROWS_FP4 * g.n_groups;
  return !tiled_gemm_applies(dtype, g);
}

// One thread per 16-byte piece of the streaming-order copy: piece i of block
// (group, row block, chunk) = i / 256 holds row 16 rb + lane % 16, columns
// 128 c + 32 t + 8 (lane / 16) .. + 7, with t = i / 64 % 4 and lane = i % 64.
__global__ __launch_bounds__(256) void pack_weights_kernel(const bf16* __restrict__ src, uint8_t* __restrict__ dst,
                                                            int rows, int cols, int64_t pieces) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= pieces) return;
  const int nkc = (cols + SKC - 1) / SKC, rbs = rows / 16;
  const int lane = (int)(i & 63), t = (int)((i >> 6) & 3);
  const int64_t blk = i >> 8;
  const int c = (int)(blk % nkc);
  const int64_t grb = blk / nkc;
  const int rb = (int)(grb % rbs);
  const int64_t grp = grb / rbs;
  const int col = SKC * c + 32 * t + 8 * (lane >> 4);  // a multiple of 8; cols a multiple of 64
  uint4 v = make_uint4(0u, 0u, 0u, 0u);
  if (col < cols) v = *reinterpret_cast<const uint4*>(src + (grp * rows + 16 * rb + (lane & 15)) * cols + col);
  *reinterpret_cast<uint4*>(dst + i * 16) = v;
}

hipError_t launch_gemm_slab(int expert_fmt, const Gemm& g, hipStream_t s) {
  if (!g.group_off) {
    const SplitPlan p = split_plan(g.n, g.k, g.n_rows);
    if (expert_fmt != 0 || p.tiles == 0 || !g.part || !g.part_cnt) return hipErrorInvalidValue;
    Gemm gs = g;
    gs.k_splits = p.k_splits;
    // up to 64 rows every weight slab is read by one workgroup: the streaming
    // policy (the wide form's four or more m-tiles re-read each slab from L2,
    // which streaming loads do not keep: QKV at 256 rows 28 -> 38 us)
    if (g.n_rows <= SPLIT_MAX_ROWS)
      return slab_launch<NSPLIT, 0, 2, true, SM, 2, true>(gs, s, (int64_t)p.tiles * p.k_splits);
    return slab_launch<NSPLIT, 0, 2, true, SM, 2, false>(gs, s, (int64_t)p.tiles * p.k_splits);
  }
  if (expert_fmt != 0) {
    if (!g.w_scales) return hipErrorInvalidValue;
    // groups of over 32 rows on average: 128-row items, so that a group just
    // past 64 rows is one item (its weights decoded once) instead of two
    if ((int64_t)g.n_rows > 32LL * g.n_groups)
      return slab_launch<128, 1, 2, false, 128>(g, s, tile_grid(g, 128, 128));
    return slab_launch<128, 1, 2, false>(g, s, tile_grid(g, SM, 128));
  }
  // groups of up to 32 rows on average mostly fit one 64-row item, whose
  // weights no other workgroup reads: the streaming policy (C2 experts 8% faster)
  if ((int64_t)g.n_rows <= 32LL * g.n_groups) return slab_launch<128, 0, 2, false, SM, 1, true>(g, s, tile_grid(g, SM, 128));
  return slab_launch<128, 0, 2, false>(g, s, tile_grid(g, SM, 128));
}

hipError_t launch_pack_weights(const void* src, void* dst, int groups, int rows, int cols, hipStream_t s) {
  const int64_t pieces = (int64_t)groups * (rows / 16) * ((cols + SKC - 1) / SKC) * 256;
  if (pieces <= 0) return hipSuccess;
  const int64_t blocks = (pieces + 255) / 256;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pack_weights_kernel, dim3((unsigned)blocks), dim3(256), 0, s, reinterpret_cast<const bf16*>(src),
                     reinterpret_cast<uint8_t*>(dst), rows, cols, pieces);
  return hipGetLastError();
}

}  // namespace mcpu
