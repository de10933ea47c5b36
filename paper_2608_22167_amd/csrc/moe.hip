// Normalisation, router, token permutation and expert combine for gfx950.
//
//  rmsnorm      one workgroup per token: y = x / sqrt(mean(x^2) + eps) * g
//  router       one workgroup per token: RMSNorm of the residual stream in
//               fp32, fp32 router logits (bf16 router weights widened
//               exactly), top-k by wavefront arg-max reductions (ties to the
//               lower expert id), softmax over the selected logits
//  permute      one workgroup: per-expert histogram, exclusive scan, and a
//               stable placement of every (token, slot) assignment into
//               expert-sorted rows using wavefront ballots; no atomics on the
//               placement, so the order is deterministic
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

template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_kernel(RmsNorm P) {
  __shared__ float scratch[8];
  const int t = blockIdx.x;
  const float* x = P.x + (int64_t)t * P.hidden;
  float ss = 0.f;
  for (int i = threadIdx.x; i < P.hidden; i += blockDim.x) ss += x[i] * x[i];
  ss = block_sum_256(ss, scratch);
  const float inv = 1.0f / sqrtf(ss / (float)P.hidden + P.eps);
  T* out = reinterpret_cast<T*>(P.out) + (int64_t)t * P.hidden;
  for (int i = threadIdx.x; i < P.hidden; i += blockDim.x) Elem<T>::store(out, i, x[i] * inv * P.g[i]);
}

hipError_t launch_rmsnorm(int dtype, const RmsNorm& p, hipStream_t s) {
  if (p.n_tokens == 0) return hipSuccess;
  if (dtype == 0) hipLaunchKernelGGL((rmsnorm_kernel<float>), dim3(p.n_tokens), dim3(256), 0, s, p);
  else hipLaunchKernelGGL((rmsnorm_kernel<bf16>), dim3(p.n_tokens), dim3(256), 0, s, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// router
// ---------------------------------------------------------------------------

constexpr int ROUTER_MAX_H = 8192;

template <typename T>
__global__ __launch_bounds__(256) void router_kernel(Router P) {
  __shared__ float hn[ROUTER_MAX_H];
  __shared__ float logits[64];
  __shared__ float scratch[8];
  const int t = blockIdx.x, H = P.hidden;
  const float* h = P.h + (int64_t)t * H;
  float ss = 0.f;
  for (int i = threadIdx.x; i < H; i += blockDim.x) ss += h[i] * h[i];
  ss = block_sum_256(ss, scratch);
  const float inv = 1.0f / sqrtf(ss / (float)H + P.eps);
  T* hq = reinterpret_cast<T*>(P.hn_out) + (int64_t)t * H;
  for (int i = threadIdx.x; i < H; i += blockDim.x) {
    const float v = h[i] * inv * P.g2[i];
    hn[i] = v;
    Elem<T>::store(hq, i, v);
  }
  __syncthreads();

  const int wave = threadIdx.x >> 6, lane = lane_id(), nw = blockDim.x >> 6;
  const T* wr = reinterpret_cast<const T*>(P.w_r);
  for (int e = wave; e < P.n_experts; e += nw) {
    float acc = 0.f;
    for (int i = lane; i < H; i += 64) acc += hn[i] * Elem<T>::load(wr, (int64_t)e * H + i);
    acc = wave_sum(acc);
    if (lane == 0) logits[e] = acc + P.b_r[e];
  }
  __syncthreads();

  if (wave == 0) {
    const int E = P.n_experts, K = P.top_k;
    float v = lane < E ? logits[lane] : -INFINITY;
    int sel_e[8];
    float sel_v[8];
    for (int s = 0; s < K; ++s) {
      int e;
      if (P.force_idx) {
        e = P.force_idx[(int64_t)t * K + s];
        if (e < 0 || e >= E) {
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
      sel_e[s] = e;
      sel_v[s] = logits[e];
    }
    float mx = sel_v[0];
    for (int s = 1; s < K; ++s) mx = fmaxf(mx, sel_v[s]);
    float den = 0.f, wv[8];
    for (int s = 0; s < K; ++s) {
      wv[s] = expf(sel_v[s] - mx);
      den += wv[s];
    }
    if (lane < K) {
      float mine = 0.f;
      int me = 0;
      for (int s = 0; s < K; ++s)
        if (s == lane) {
          mine = wv[s] / den;
          me = sel_e[s];
        }
      P.idx_out[(int64_t)t * K + lane] = me;
      P.w_out[(int64_t)t * K + lane] = mine;
    }
  }
}

hipError_t launch_router(int dtype, const Router& p, hipStream_t s) {
  if (p.n_tokens == 0) return hipSuccess;
  if (p.hidden > ROUTER_MAX_H || p.n_experts > 64 || p.top_k > 8) return hipErrorInvalidValue;
  if (dtype == 0) hipLaunchKernelGGL((router_kernel<float>), dim3(p.n_tokens), dim3(256), 0, s, p);
  else hipLaunchKernelGGL((router_kernel<bf16>), dim3(p.n_tokens), dim3(256), 0, s, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// permute: expert-sorted rows, stable in (token, slot) order
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void permute_kernel(Permute P) {
  __shared__ int cnt[64];
  const int n = P.n_tokens * P.top_k, E = P.n_experts;
  if (threadIdx.x < 64) cnt[threadIdx.x] = 0;
  __syncthreads();
  for (int a = threadIdx.x; a < n; a += blockDim.x) {
    int e = P.idx[a];
    if (e < 0 || e >= E) {
      set_error(P.err, 4);
      e = 0;
    }
    atomicAdd(&cnt[e], 1);  // integer counts: order-independent
  }
  __syncthreads();
  if (threadIdx.x >= 64) return;
  const int lane = threadIdx.x;
  const int c = lane < E ? cnt[lane] : 0;
  const int incl = wave_incl_scan(c);
  int base = incl - c;  // lane e holds the next free row of expert e
  if (lane < E) P.group_off[lane] = base;
  if (lane == E - 1) P.group_off[E] = incl;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int a0 = 0; a0 < n; a0 += 64) {
    const int a = a0 + lane;
    int e = a < n ? P.idx[a] : -1;
    if (a < n && (e < 0 || e >= E)) e = 0;
    bool todo = a < n;
    int pos = -1;
    uint64_t pending = __ballot(todo);
    while (pending) {
      const int first = __ffsll((unsigned long long)pending) - 1;
      const int e0 = __shfl(e, first, 64);
      const uint64_t m = __ballot(todo && e == e0);
      const int b0 = __shfl(base, e0, 64);
      if (todo && e == e0) {
        pos = b0 + __popcll(m & lt_mask);
        todo = false;
      }
      if (lane == e0) base += __popcll(m);
      pending = __ballot(todo);
    }
    if (a < n) {
      P.pos_of[a] = pos;
      P.src_tok[pos] = a / P.top_k;
    }
  }
}

hipError_t launch_permute(const Permute& p, hipStream_t s) {
  if (p.n_experts > 64) return hipErrorInvalidValue;
  hipLaunchKernelGGL(permute_kernel, dim3(1), dim3(256), 0, s, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// combine: out[t] = h[t] + sum_{s < k} w[t][s] * y[pos_of[t k + s]]
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void moe_combine_kernel(MoeCombine P) {
  const int t = blockIdx.x, H = P.hidden, K = P.top_k;
  int rows[8];
  float ws[8];
  for (int s = 0; s < K; ++s) {
    rows[s] = P.pos_of[(int64_t)t * K + s];
    ws[s] = P.w[(int64_t)t * K + s];
  }
  for (int i = threadIdx.x; i < H; i += blockDim.x) {
    float acc = 0.f;
    for (int s = 0; s < K; ++s) acc += ws[s] * P.y[(int64_t)rows[s] * H + i];
    P.out[(int64_t)t * H + i] = P.h[(int64_t)t * H + i] + acc;
  }
}

hipError_t launch_moe_combine(const MoeCombine& p, hipStream_t s) {
  if (p.n_tokens == 0) return hipSuccess;
  hipLaunchKernelGGL(moe_combine_kernel, dim3(p.n_tokens), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace mcpu
