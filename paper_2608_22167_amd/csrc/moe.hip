// Router, token permutation and expert combine for gfx950.
//
//  router       RMSNorm of the residual stream in fp32, fp32 router logits
//               (bf16 router weights widened exactly), top-k (ties to the
//               lower expert id), softmax over the selected logits: one
//               workgroup per token for small batches, 16 tokens per
//               workgroup with fp32 matrix-core products for large ones
//  permute      per-expert histogram, exclusive scan, and a stable placement
//               of every (token, slot) assignment into expert-sorted rows
//               using wavefront ballots; no atomics on the placement, so the
//               order is deterministic. One workgroup up to 4096 assignments;
//               beyond, per-chunk histograms, one scan over the chunks and a
//               per-chunk placement
//  moe_combine  one workgroup per token: out = h + sum_k w_k y_k in slot order
#include "device.h"
#include "kernels.h"

namespace mcpu {

__device__ __forceinline__ float block_sum_256(float v, float* scratch) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if (lane_id() == 0) scratch[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) t += scratch[i];
  __syncthreads();
  return t;
}

// Thread i of 256 loads float4 number i + 256 j (j < NV) of a row of length H
// and of its gain vector, all loads in flight at once (rows past H read
// element 0 and are masked); returns the thread's sum of squares.
template <int NV>
__device__ __forceinline__ float load_row(const float* x, const float* g, int H, float4* xv, float4* gv) {
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = (threadIdx.x + 256 * j) * 4;
    const int ii = i < H ? i : 0;
    xv[j] = *reinterpret_cast<const float4*>(x + ii);
    gv[j] = *reinterpret_cast<const float4*>(g + ii);
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const bool v = (threadIdx.x + 256 * j) * 4 < H;
    ss += v ? xv[j].x * xv[j].x + xv[j].y * xv[j].y + xv[j].z * xv[j].z + xv[j].w * xv[j].w : 0.f;
  }
  return ss;
}

// ---------------------------------------------------------------------------
// router
// ---------------------------------------------------------------------------

constexpr int ROUTER_MAX_H = 8192;
constexpr int ROUTER_MAX_E = 64;

// 8 consecutive router weights, loaded raw and widened to fp32 (exact)
template <typename T> struct Raw8;
template <> struct Raw8<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = reinterpret_cast<const float4*>(p)[0];
    b = reinterpret_cast<const float4*>(p)[1];
  }
  __device__ __forceinline__ void widen(float w[8]) const {
    w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w; w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
  }
};
template <> struct Raw8<bf16> {
  uint4 v;
  __device__ __forceinline__ void load(const bf16* p) { v = *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ void widen(float w[8]) const {
    const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      w[2 * i] = __uint_as_float(u[i] << 16);
      w[2 * i + 1] = __uint_as_float(u[i] & 0xFFFF0000u);
    }
  }
};

// Step of the router's reduce-scatter: N partial sums per lane, partner at
// lane distance O. The upper lane of each pair keeps the upper half of the
// sums (adding its partner's copy), the lower lane the lower half; with one
// sum left, partners just add. Templated so every index is a constant (a
// runtime half-width would put the array in scratch memory).
template <int N, int O, int E>
__device__ __forceinline__ void reduce_scatter(float (&acc)[E], int lane) {
  if constexpr (O >= 1) {
    if constexpr (N > 1) {
      constexpr int half = N / 2;
      const bool upper = (lane & O) != 0;
#pragma unroll
      for (int j = 0; j < half; ++j) {
        const float send = upper ? acc[j] : acc[j + half];
        const float keep = upper ? acc[j + half] : acc[j];
        acc[j] = keep + __shfl_xor(send, O, 64);
      }
      reduce_scatter<half, O / 2, E>(acc, lane);
    } else {
      acc[0] += __shfl_xor(acc[0], O, 64);
      reduce_scatter<1, O / 2, E>(acc, lane);
    }
  }
}

// Top-k experts of token t and their softmax weights (wavefront 0 of the
// workgroup; logits in LDS): lane s < k keeps the s-th selection in registers
// (the selection count is a runtime value, so an array indexed by it would
// live in scratch memory); ties go to the lower expert id; forced selections
// replace the arg-max when given.
__device__ __forceinline__ void router_topk(const Router& P, const float* logits, int t, int lane) {
  const int NE = P.n_experts, K = P.top_k;
  float v = lane < NE ? logits[lane] : -INFINITY;
  int my_e = 0;
  float my_v = -INFINITY;
  for (int s = 0; s < K; ++s) {
    int e;
    if (P.force_idx) {
      e = P.force_idx[(int64_t)t * K + s];
      if (e < 0 || e >= NE) {
        if (lane == 0) set_error(P.err, 4);
        e = 0;
      }
    } else {
      // arg-max over lanes, ties to the lower expert id
      float bv = v;
      int bi = lane;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const float ov = __shfl_xor(bv, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (ov > bv || (ov == bv && oi < bi)) {
          bv = ov;
          bi = oi;
        }
      }
      e = bi;
      if (lane == e) v = -INFINITY;
    }
    if (lane == s) {
      my_e = e;
      my_v = logits[e];
    }
  }
  // softmax over the selections, maximum and sum taken in selection order
  float mx = __shfl(my_v, 0, 64);
  for (int s = 1; s < K; ++s) mx = fmaxf(mx, __shfl(my_v, s, 64));
  const float ex = expf(my_v - mx);
  float den = 0.f;
  for (int s = 0; s < K; ++s) den += __shfl(ex, s, 64);
  if (lane < K) {
    P.idx_out[(int64_t)t * K + lane] = my_e;
    P.w_out[(int64_t)t * K + lane] = ex / den;
  }
}

// One workgroup per token. Thread i owns the 8-wide reduction chunks i, i+256,
// ... and accumulates all E logits over them; partial logits are then summed
// across lanes (wavefront butterflies) and across the 4 wavefronts (LDS).
template <typename T, int E, int NV>
__global__ __launch_bounds__(256) void router_kernel(Router P) {
  __shared__ float hn[ROUTER_MAX_H];
  __shared__ float part[4][E];
  __shared__ float logits[E];
  __shared__ float scratch[8];
  const int t = blockIdx.x, H = P.hidden;
  float4 hv[NV], gv[NV];
  const float ss = load_row<NV>(P.h + (int64_t)t * H, P.g2, H, hv, gv);
  const float inv = 1.0f / sqrtf(block_sum_256(ss, scratch) / (float)H + P.eps);
  T* hq = reinterpret_cast<T*>(P.hn_out) + (int64_t)t * H;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = (threadIdx.x + 256 * j) * 4;
    if (i < H) {
      const float4 v = make_float4(hv[j].x * inv * gv[j].x, hv[j].y * inv * gv[j].y,
                                   hv[j].z * inv * gv[j].z, hv[j].w * inv * gv[j].w);
      *reinterpret_cast<float4*>(hn + i) = v;
      store4(hq + i, v);
    }
  }
  __syncthreads();

  const int wave = threadIdx.x >> 6, lane = lane_id();
  const T* wr = reinterpret_cast<const T*>(P.w_r);
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  const int nchunk = H / 8;
  for (int c0 = 0; c0 < nchunk; c0 += blockDim.x) {
    // branch-free: out-of-range chunks and experts read a valid address and
    // contribute zero
    const int c = c0 + threadIdx.x;
    const bool cv = c < nchunk;
    const int cc = cv ? c : nchunk - 1;
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = cv ? hn[8 * cc + j] : 0.f;
    // the raw chunks of up to 32 experts are loaded together, then widened
    constexpr int G = E < 32 ? E : 32;
#pragma unroll
    for (int e0 = 0; e0 < E; e0 += G) {
      Raw8<T> raw[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int e = e0 + g, ee = e < P.n_experts ? e : 0;
        raw[g].load(wr + (int64_t)ee * H + 8 * cc);
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float w[8];
        raw[g].widen(w);
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[e0 + g] += x[j] * w[j];
      }
    }
  }
  // reduce-scatter across the 64 lanes: each halving step trades half of the
  // partial sums with the partner lane, so lane l ends with expert l / (64 / E)
  reduce_scatter<E, 32>(acc, lane);
  if (lane % (64 / E) == 0) part[wave][lane / (64 / E)] = acc[0];
  __syncthreads();
  if (threadIdx.x < P.n_experts) {
    const int e = threadIdx.x;
    logits[e] = part[0][e] + part[1][e] + part[2][e] + part[3][e] + P.b_r[e];
    if (P.logits_out) P.logits_out[(int64_t)t * P.n_experts + e] = logits[e];
  }
  __syncthreads();

  if (wave == 0) router_topk(P, logits, t, lane);
}

// Router for one token per workgroup of 1024 threads: 1024 / E threads per
// expert, thread l of expert e taking the 8-wide reduction chunks l, l + TPE,
// ... of its router row. All of a thread's router-weight loads are issued at
// the start, together with the residual row's, so the whole kernel waits for
// memory once; the normalised row then goes through LDS, each expert's
// partial sums meet in a butterfly over its threads (across two wavefronts
// through LDS when E = 8), and wavefront 0 takes the top k as above.
constexpr int RW_THREADS = 1024;

template <typename T, int E, int NV, int CPT>
__global__ __launch_bounds__(RW_THREADS) void router_wide_kernel(Router P) {
  constexpr int TPE = RW_THREADS / E;  // threads per expert
  constexpr int TW = TPE < 64 ? TPE : 64;
  __shared__ float hn[ROUTER_MAX_H];
  __shared__ float logits[E];
  __shared__ float half_sum[E];
  __shared__ float scratch[RW_THREADS / 64];
  const int t = blockIdx.x, H = P.hidden, tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
  const int e = tid / TPE, l = tid % TPE;
  const int nchunk = H / 8;

  // router-weight chunks of this thread (rows past n_experts and chunks past
  // the row read valid addresses and are not used)
  const T* wr = reinterpret_cast<const T*>(P.w_r) + (int64_t)(e < P.n_experts ? e : 0) * H;
  Raw8<T> raw[CPT];
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int c = l + TPE * i;
    raw[i].load(wr + 8 * (c < nchunk ? c : 0));
  }
  // residual row and gain: float4 j of thread t is features 4 (t + 1024 j) ..
  float4 hv[NV], gv[NV];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = (tid + RW_THREADS * j) * 4;
    const int ii = i < H ? i : 0;
    hv[j] = *reinterpret_cast<const float4*>(P.h + (int64_t)t * H + ii);
    gv[j] = *reinterpret_cast<const float4*>(P.g2 + ii);
  }
#pragma unroll
  for (int j = 0; j < NV; ++j)
    if ((tid + RW_THREADS * j) * 4 < H)
      ss += hv[j].x * hv[j].x + hv[j].y * hv[j].y + hv[j].z * hv[j].z + hv[j].w * hv[j].w;
  // sum of squares over the workgroup
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o, 64);
  if (lane == 0) scratch[wave] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < RW_THREADS / 64; ++w) tot += scratch[w];
  const float inv = 1.0f / sqrtf(tot / (float)H + P.eps);
  T* hq = reinterpret_cast<T*>(P.hn_out) + (int64_t)t * H;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = (tid + RW_THREADS * j) * 4;
    if (i < H) {
      const float4 v = make_float4(hv[j].x * inv * gv[j].x, hv[j].y * inv * gv[j].y, hv[j].z * inv * gv[j].z,
                                   hv[j].w * inv * gv[j].w);
      *reinterpret_cast<float4*>(hn + i) = v;
      store4(hq + i, v);
    }
  }
  __syncthreads();

  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int c = l + TPE * i;
    if (c < nchunk) {
      float w[8];
      raw[i].widen(w);
      const float4 x0 = *reinterpret_cast<const float4*>(hn + 8 * c);
      const float4 x1 = *reinterpret_cast<const float4*>(hn + 8 * c + 4);
      acc += x0.x * w[0] + x0.y * w[1] + x0.z * w[2] + x0.w * w[3] + x1.x * w[4] + x1.y * w[5] + x1.z * w[6] +
             x1.w * w[7];
    }
  }
  // over the expert's threads: a butterfly within the wavefront, then (TPE =
  // 128) the two wavefronts' halves through LDS
#pragma unroll
  for (int o = TW / 2; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
  if constexpr (TPE > 64) {
    if (l == 64) half_sum[e] = acc;
    __syncthreads();
    if (l == 0) acc += half_sum[e];
  }
  if (l == 0 && e < P.n_experts) {
    const float v = acc + P.b_r[e];
    logits[e] = v;
    if (P.logits_out) P.logits_out[(int64_t)t * P.n_experts + e] = v;
  }
  __syncthreads();
  if (wave == 0) router_topk(P, logits, t, lane);
}

// Router for many tokens: a workgroup owns 16 tokens, so the router weights
// are read once per 16 tokens instead of once per token, and its four
// wavefronts split the reduction into quarters. Pass 1 sums the squares of
// each token's residual row; pass 2 normalises it (hn is written in the layer
// dtype) and feeds the fp32 matrix-core product logits^T = W_r hn^T in
// 16 x 16 x 4 tiles (16 experts x 16 tokens). A lane loads four consecutive
// reduction indices of its expert row and token row and spends one per
// product, so both operands see the same index order; RU independent
// accumulator chains keep loads of later indices in flight. The quarters'
// logits meet in LDS, and lanes 0-15 of wavefront 0 take one token each for
// the top-k (ties to the lower expert id) and the softmax.
constexpr int RT_TOK = 16;
constexpr int ROUTER_TILED_MIN_TOKENS = 1024;

template <typename T> struct Raw4;
template <> struct Raw4<float> {
  __device__ __forceinline__ static float4 load(const float* p) { return *reinterpret_cast<const float4*>(p); }
};
template <> struct Raw4<bf16> {
  __device__ __forceinline__ static float4 load(const bf16* p) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u), __uint_as_float(u.y << 16),
                       __uint_as_float(u.y & 0xFFFF0000u));
  }
};

template <typename T, int EB>
__global__ __launch_bounds__(256) void router_tiled_kernel(Router P) {
  constexpr int EMAX = 16 * EB, RU = 4;
  __shared__ float lg[4][RT_TOK][EMAX + 1];
  __shared__ float ssq[4][RT_TOK];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tok0 = blockIdx.x * RT_TOK;
  const int H = P.hidden, E = P.n_experts, HQ = H / 4;
  const int c = lane & 15, grp = lane >> 4;
  const bool live = tok0 + c < P.n_tokens;
  const int t = live ? tok0 + c : P.n_tokens - 1;  // rows past the end repeat the last (dropped)
  const int k_begin = wave * HQ + 4 * grp, k_end = (wave + 1) * HQ;
  const float* hrow = P.h + (int64_t)t * H;

  float ssu[RU] = {};  // RU loads in flight
  int k = k_begin;
  for (; k + 16 * (RU - 1) < k_end; k += 16 * RU) {
#pragma unroll
    for (int u = 0; u < RU; ++u) {
      const float4 v = *reinterpret_cast<const float4*>(hrow + k + 16 * u);
      ssu[u] += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    }
  }
  for (; k < k_end; k += 16) {
    const float4 v = *reinterpret_cast<const float4*>(hrow + k);
    ssu[0] += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < RU; ++u) ss += ssu[u];
  ss += __shfl_xor(ss, 16, 64);
  ss += __shfl_xor(ss, 32, 64);
  if (grp == 0) ssq[wave][c] = ss;
  __syncthreads();
  const float inv = 1.0f / sqrtf((ssq[0][c] + ssq[1][c] + ssq[2][c] + ssq[3][c]) / (float)H + P.eps);

  const T* wr = reinterpret_cast<const T*>(P.w_r);
  const T* wrow[EB];
#pragma unroll
  for (int b = 0; b < EB; ++b) wrow[b] = wr + (int64_t)min(16 * b + c, E - 1) * H;  // rows past E: dropped
  T* hq = reinterpret_cast<T*>(P.hn_out) + (int64_t)t * H;
  f32x4 acc[RU][EB];
#pragma unroll
  for (int u = 0; u < RU; ++u)
#pragma unroll
    for (int b = 0; b < EB; ++b) acc[u][b] = f32x4{0.f, 0.f, 0.f, 0.f};
  // per group of RU indices: every load, then the products, then the hn
  // stores (a store between loads would serialise them)
  auto group = [&](int k0, int n) __attribute__((always_inline)) {
    float4 v[RU], g[RU], w[RU][EB];
#pragma unroll
    for (int u = 0; u < RU; ++u) {
      if (u < n) {
        v[u] = *reinterpret_cast<const float4*>(hrow + k0 + 16 * u);
        g[u] = *reinterpret_cast<const float4*>(P.g2 + k0 + 16 * u);
#pragma unroll
        for (int b = 0; b < EB; ++b) w[u][b] = Raw4<T>::load(wrow[b] + k0 + 16 * u);
      }
    }
    float4 hn[RU];
#pragma unroll
    for (int u = 0; u < RU; ++u) {
      if (u < n) {
        hn[u] = make_float4(v[u].x * inv * g[u].x, v[u].y * inv * g[u].y, v[u].z * inv * g[u].z,
                            v[u].w * inv * g[u].w);
#pragma unroll
        for (int b = 0; b < EB; ++b) {
          acc[u][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(w[u][b].x, hn[u].x, acc[u][b], 0, 0, 0);
          acc[u][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(w[u][b].y, hn[u].y, acc[u][b], 0, 0, 0);
          acc[u][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(w[u][b].z, hn[u].z, acc[u][b], 0, 0, 0);
          acc[u][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(w[u][b].w, hn[u].w, acc[u][b], 0, 0, 0);
        }
      }
    }
    // rows past the end rewrite the last row's identical values
#pragma unroll
    for (int u = 0; u < RU; ++u)
      if (u < n) store4(hq + k0 + 16 * u, hn[u]);
  };
  k = k_begin;
  for (; k + 16 * (RU - 1) < k_end; k += 16 * RU) group(k, RU);
  for (; k < k_end; k += 16) group(k, 1);
  // acc[.][b][r] = partial logit of expert 16 b + 4 grp + r for token c
#pragma unroll
  for (int b = 0; b < EB; ++b)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v = 0.f;
#pragma unroll
      for (int u = 0; u < RU; ++u) v += acc[u][b][r];
      lg[wave][c][16 * b + 4 * grp + r] = v;
    }
  __syncthreads();
  if (wave == 0 && lane < RT_TOK && tok0 + lane < P.n_tokens) {
    const int tk = tok0 + lane, K = P.top_k;
    float* L = lg[0][lane];
    for (int e = 0; e < E; ++e) {
      const float v = L[e] + lg[1][lane][e] + lg[2][lane][e] + lg[3][lane][e] + P.b_r[e];
      L[e] = v;
      if (P.logits_out) P.logits_out[(int64_t)tk * E + e] = v;
    }
    int sel_e[8];
    float sel_v[8];
    uint64_t taken = 0;
    for (int s = 0; s < K; ++s) {
      int e = 0;
      if (P.force_idx) {
        e = P.force_idx[(int64_t)tk * K + s];
        if (e < 0 || e >= E) {
          set_error(P.err, 4);
          e = 0;
        }
      } else {
        float bv = -INFINITY;
        e = -1;
        for (int x = 0; x < E; ++x)  // first maximum among the rest: ties to the lower id
          if (!((taken >> x) & 1) && (e < 0 || L[x] > bv)) {
            bv = L[x];
            e = x;
          }
        taken |= 1ull << e;
      }
      sel_e[s] = e;
      sel_v[s] = L[e];
    }
    float mx = sel_v[0];
    for (int s = 1; s < K; ++s) mx = fmaxf(mx, sel_v[s]);
    float den = 0.f, wv[8];
    for (int s = 0; s < K; ++s) {
      wv[s] = expf(sel_v[s] - mx);
      den += wv[s];
    }
    for (int s = 0; s < K; ++s) {
      P.idx_out[(int64_t)tk * K + s] = sel_e[s];
      P.w_out[(int64_t)tk * K + s] = wv[s] / den;
    }
  }
}

template <typename T, int E>
static void router_nv(const Router& p, hipStream_t s) {
  const int nv = (p.hidden + 1023) / 1024;
  dim3 g(p.n_tokens), b(256);
  if (nv <= 1) hipLaunchKernelGGL((router_kernel<T, E, 1>), g, b, 0, s, p);
  else if (nv <= 2) hipLaunchKernelGGL((router_kernel<T, E, 2>), g, b, 0, s, p);
  else if (nv <= 3) hipLaunchKernelGGL((router_kernel<T, E, 3>), g, b, 0, s, p);
  else if (nv <= 4) hipLaunchKernelGGL((router_kernel<T, E, 4>), g, b, 0, s, p);
  else hipLaunchKernelGGL((router_kernel<T, E, 8>), g, b, 0, s, p);
}

// The wide router when each thread's share of its expert row is at most 16
// chunks (8 for fp32 weights) with 1024 / E threads per expert, else one
// workgroup of 256 threads per token.
template <typename T, int E>
static void router_pick(const Router& p, hipStream_t s) {
  constexpr int TPE = RW_THREADS / E;
  const int cpt = (p.hidden / 8 + TPE - 1) / TPE;
  const int nv = (p.hidden + 4 * RW_THREADS - 1) / (4 * RW_THREADS);
  dim3 g(p.n_tokens), b(RW_THREADS);
#define RW(NV, CPT) hipLaunchKernelGGL((router_wide_kernel<T, E, NV, CPT>), g, b, 0, s, p)
  if constexpr (sizeof(T) == 4) {  // fp32 weights: 8 registers a chunk, at most 8 chunks
    if (nv == 1 && cpt <= 4) RW(1, 4);
    else if (nv == 1 && cpt <= 8) RW(1, 8);
    else router_nv<T, E>(p, s);
  } else {
    if (nv == 1 && cpt <= 4) RW(1, 4);
    else if (nv == 1 && cpt <= 8) RW(1, 8);
    else if (nv == 1 && cpt <= 12) RW(1, 12);
    else if (nv == 1 && cpt <= 16) RW(1, 16);
    else if (nv == 2 && cpt <= 16) RW(2, 16);
    else router_nv<T, E>(p, s);
  }
#undef RW
}

// Up to one wide workgroup per compute unit; more tokens than that run
// faster on the 256-thread workgroups (several resident per compute unit).
constexpr int ROUTER_WIDE_MAX_TOKENS = 256;

template <typename T>
static void router_e(const Router& p, hipStream_t s) {
  if (p.n_tokens > ROUTER_WIDE_MAX_TOKENS) {
    if (p.n_experts <= 8) router_nv<T, 8>(p, s);
    else if (p.n_experts <= 16) router_nv<T, 16>(p, s);
    else if (p.n_experts <= 32) router_nv<T, 32>(p, s);
    else router_nv<T, 64>(p, s);
    return;
  }
  if (p.n_experts <= 8) router_pick<T, 8>(p, s);
  else if (p.n_experts <= 16) router_pick<T, 16>(p, s);
  else if (p.n_experts <= 32) router_pick<T, 32>(p, s);
  else router_pick<T, 64>(p, s);
}

template <typename T>
static void router_tiled(const Router& p, hipStream_t s) {
  dim3 g((p.n_tokens + RT_TOK - 1) / RT_TOK), b(256);
  if (p.n_experts <= 16) hipLaunchKernelGGL((router_tiled_kernel<T, 1>), g, b, 0, s, p);
  else if (p.n_experts <= 32) hipLaunchKernelGGL((router_tiled_kernel<T, 2>), g, b, 0, s, p);
  else hipLaunchKernelGGL((router_tiled_kernel<T, 4>), g, b, 0, s, p);
}

hipError_t launch_router(int dtype, const Router& p, hipStream_t s) {
  if (p.n_tokens == 0) return hipSuccess;
  if (p.hidden > ROUTER_MAX_H || p.hidden % 8 || p.n_experts > ROUTER_MAX_E || p.top_k > 8)
    return hipErrorInvalidValue;
  if (p.n_tokens >= ROUTER_TILED_MIN_TOKENS && p.hidden % 64 == 0) {
    if (dtype == 0) router_tiled<float>(p, s);
    else router_tiled<bf16>(p, s);
    return hipGetLastError();
  }
  if (dtype == 0) router_e<float>(p, s);
  else router_e<bf16>(p, s);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// permute: expert-sorted rows, stable in (token, slot) order
// ---------------------------------------------------------------------------

constexpr int PERM_SUB = PERM_CHUNK / 64;  // 64-assignment sub-chunks per workgroup

// rank of this lane among the valid lanes of its wavefront holding the same
// expert and a lower lane id: the lanes that agree with this one on every bit
// of the expert id (one ballot per bit, nbits = ceil(log2 E)), counted below it
__device__ __forceinline__ int rank_in_chunk(int e, bool valid, int nbits) {
  const int lane = lane_id();
  const uint64_t lt = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  uint64_t same = __ballot(valid);
  for (int b = 0; b < nbits; ++b) {  // uniform trip count
    const bool bit = (e >> b) & 1;
    const uint64_t ones = __ballot(bit);
    same &= bit ? ones : ~ones;
  }
  return __popcll(same & lt);
}

__device__ __forceinline__ int checked_expert(const Permute& P, int a) {
  const int e = P.idx[a];
  if (e < 0 || e >= P.n_experts) {
    set_error(P.err, 4);
    return 0;
  }
  return e;
}

// Ranks the assignments a0 .. a0 + nloc - 1 (at most PERM_CHUNK) stably by
// expert and scatters them. base (per expert, the chunk's first row) comes
// from the multi-chunk scan; without it the workgroup holds the whole batch
// and writes group_off itself. A wavefront owns sub-chunks w, w + 4, ...; all
// of its expert ids are loaded up front, so the ids cost one memory round
// trip rather than one per sub-chunk and pass.
__device__ void permute_chunk(const Permute& P, int a0, int nloc, const int32_t* base) {
  __shared__ int cnt[PERM_SUB][64];
  constexpr int PW = PERM_SUB / 4;  // sub-chunks per wavefront
  const int E = P.n_experts;
  const int nch = (nloc + 63) / 64;
  const int nbits = 32 - __clz(max(E - 1, 1));  // bits of the largest expert id
  const int wave = threadIdx.x >> 6, lane = lane_id();
  int ex[PW];
#pragma unroll
  for (int i = 0; i < PW; ++i) {
    const int a = (wave + 4 * i) * 64 + lane;
    ex[i] = a < nloc ? P.idx[a0 + a] : 0;
  }
  for (int i = threadIdx.x; i < PERM_SUB * 64; i += blockDim.x) (&cnt[0][0])[i] = 0;
  // an id outside [0, E) sets the error bit and counts as expert 0
  bool bad = false;
#pragma unroll
  for (int i = 0; i < PW; ++i) {
    const bool valid = (wave + 4 * i) * 64 + lane < nloc;
    if (valid && (ex[i] < 0 || ex[i] >= E)) {
      bad = true;
      ex[i] = 0;
    }
  }
  if (bad) set_error(P.err, 4);
  __syncthreads();
  // per-sub-chunk histograms (integer counts; order-independent)
#pragma unroll
  for (int i = 0; i < PW; ++i) {
    const int c = wave + 4 * i;
    if (c * 64 + lane < nloc) atomicAdd(&cnt[c][ex[i]], 1);
  }
  __syncthreads();
  // lane e of wave 0: running first row of expert e in each sub-chunk
  if (wave == 0) {
    int run = 0;
    if (base) {
      run = lane < E ? base[lane] : 0;
    } else {
      int tot = 0;
      if (lane < E)
        for (int c = 0; c < nch; ++c) tot += cnt[c][lane];
      const int incl = wave_incl_scan(tot);
      run = incl - tot;
      if (lane < E) P.group_off[lane] = run;
      if (lane == E - 1) P.group_off[E] = incl;
    }
    if (lane < E)
      for (int c = 0; c < nch; ++c) {
        const int k = cnt[c][lane];
        cnt[c][lane] = run;
        run += k;
      }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < PW; ++i) {
    const int c = wave + 4 * i;
    if (c >= nch) break;  // uniform
    const int a = c * 64 + lane;
    const bool valid = a < nloc;
    const int r = rank_in_chunk(ex[i], valid, nbits);
    if (valid) {
      const int pos = cnt[c][ex[i]] + r;
      P.pos_of[a0 + a] = pos;
      P.src_tok[pos] = (a0 + a) / P.top_k;
    }
  }
}

__global__ __launch_bounds__(256) void permute_kernel(Permute P) {
  permute_chunk(P, 0, P.n_tokens * P.top_k, nullptr);
}

// Larger batches: per-chunk histograms, one scan over chunks, per-chunk scatter.
__global__ __launch_bounds__(256) void perm_count_kernel(Permute P) {
  __shared__ int cnt[64];
  const int n = P.n_tokens * P.top_k, E = P.n_experts;
  if (threadIdx.x < 64) cnt[threadIdx.x] = 0;
  __syncthreads();
  const int a0 = blockIdx.x * PERM_CHUNK, a1 = min(n, a0 + PERM_CHUNK);
  for (int a = a0 + (int)threadIdx.x; a < a1; a += blockDim.x) atomicAdd(&cnt[checked_expert(P, a)], 1);
  __syncthreads();
  if ((int)threadIdx.x < E) P.chunk_cnt[(int64_t)blockIdx.x * E + threadIdx.x] = cnt[threadIdx.x];
}

// One wavefront, lane e = expert: totals -> group_off, and each chunk's count
// replaced by the chunk's first row for that expert (stable in assignment order).
__global__ __launch_bounds__(64) void perm_scan_kernel(Permute P, int n_chunks) {
  const int lane = lane_id(), E = P.n_experts;
  int tot = 0;
  if (lane < E)
    for (int c = 0; c < n_chunks; ++c) tot += P.chunk_cnt[(int64_t)c * E + lane];
  const int incl = wave_incl_scan(tot);
  int run = incl - tot;
  if (lane < E) P.group_off[lane] = run;
  if (lane == E - 1) P.group_off[E] = incl;
  if (lane < E)
    for (int c = 0; c < n_chunks; ++c) {
      const int k = P.chunk_cnt[(int64_t)c * E + lane];
      P.chunk_cnt[(int64_t)c * E + lane] = run;
      run += k;
    }
}

__global__ __launch_bounds__(256) void perm_scatter_kernel(Permute P) {
  const int n = P.n_tokens * P.top_k;
  const int a0 = blockIdx.x * PERM_CHUNK;
  permute_chunk(P, a0, min(PERM_CHUNK, n - a0), P.chunk_cnt + (int64_t)blockIdx.x * P.n_experts);
}

hipError_t launch_permute(const Permute& p, hipStream_t s) {
  if (p.n_experts > 64) return hipErrorInvalidValue;
  const int n = p.n_tokens * p.top_k;
  if (n <= PERM_CHUNK) {
    hipLaunchKernelGGL(permute_kernel, dim3(1), dim3(256), 0, s, p);
    return hipGetLastError();
  }
  if (!p.chunk_cnt) return hipErrorInvalidValue;
  const int chunks = (n + PERM_CHUNK - 1) / PERM_CHUNK;
  hipLaunchKernelGGL(perm_count_kernel, dim3(chunks), dim3(256), 0, s, p);
  hipLaunchKernelGGL(perm_scan_kernel, dim3(1), dim3(64), 0, s, p, chunks);
  hipLaunchKernelGGL(perm_scatter_kernel, dim3(chunks), dim3(256), 0, s, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// combine: out[t] = h[t] + sum_{s < k} w[t][s] * y[pos_of[t k + s]]
// ---------------------------------------------------------------------------

// grid (tokens, H / 1024): each thread combines 4 consecutive features
__global__ __launch_bounds__(256) void moe_combine_kernel(MoeCombine P) {
  const int t = blockIdx.x, H = P.hidden, K = P.top_k;
  const int i = (blockIdx.y * 256 + threadIdx.x) * 4;
  if (i >= H) return;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s = 0; s < K; ++s) {
    const int row = P.pos_of[(int64_t)t * K + s];
    const float w = P.w[(int64_t)t * K + s];
    const float4 y = *reinterpret_cast<const float4*>(P.y + (int64_t)row * H + i);
    acc.x += w * y.x; acc.y += w * y.y; acc.z += w * y.z; acc.w += w * y.w;
  }
  const float4 h = *reinterpret_cast<const float4*>(P.h + (int64_t)t * H + i);
  *reinterpret_cast<float4*>(P.out + (int64_t)t * H + i) =
      make_float4(h.x + acc.x, h.y + acc.y, h.z + acc.z, h.w + acc.w);
}

hipError_t launch_moe_combine(const MoeCombine& p, hipStream_t s) {
  if (p.n_tokens == 0) return hipSuccess;
  if (p.hidden % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(moe_combine_kernel, dim3(p.n_tokens, (p.hidden + 1023) / 1024), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace mcpu
