// Token embedding, the final RMSNorm in front of the vocabulary projection,
// and the reduction that turns the projection's per-slot summaries
// (EPI_LOGITS, gemm_epilogue.h) into one sampled token and its
// log-probabilities per row.
#include "device.h"
#include "kernels_lm.h"

namespace mcpu {

// x[t] = E[tokens[t]] widened to fp32; an id outside [0, vocab) writes zeros
// and sets error bit 32. One workgroup per token, 8 bf16 per thread per pass.
__global__ __launch_bounds__(256) void embed_kernel(EmbedArgs P) {
  const int t = blockIdx.x;
  const int id = P.tokens[t];
  const bool ok = id >= 0 && id < P.vocab;
  if (!ok && threadIdx.x == 0) set_error(P.err, 32);
  const bf16* e = reinterpret_cast<const bf16*>(P.table) + (int64_t)(ok ? id : 0) * P.hidden;
  float* x = P.x + (int64_t)t * P.hidden;
  for (int c = 8 * threadIdx.x; c < P.hidden; c += 8 * blockDim.x) {
    const uint4 v = *reinterpret_cast<const uint4*>(e + c);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    float f[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = ok ? __uint_as_float(w[i] << 16) : 0.f;
      f[2 * i + 1] = ok ? __uint_as_float(w[i] & 0xFFFF0000u) : 0.f;
    }
    reinterpret_cast<float4*>(x + c)[0] = make_float4(f[0], f[1], f[2], f[3]);
    reinterpret_cast<float4*>(x + c)[1] = make_float4(f[4], f[5], f[6], f[7]);
  }
}

// xn[t] = x[t] / sqrt(mean(x[t]^2) + eps) * g, stored as bf16 (the
// projection's operand); workgroup 0 also writes the one-group row range
// {0, n_tokens} the grouped GEMM kernels read.
__global__ __launch_bounds__(256) void final_norm_kernel(FinalNorm P) {
  __shared__ float part[4];
  const int t = blockIdx.x, tid = threadIdx.x;
  if (t == 0 && tid == 0) {
    P.group_off[0] = 0;
    P.group_off[1] = P.n_tokens;
  }
  const float* x = P.x + (int64_t)(P.rows ? P.rows[t] : t) * P.hidden;
  float ss = 0.f;
  for (int c = 4 * tid; c < P.hidden; c += 4 * blockDim.x) {
    const float4 v = *reinterpret_cast<const float4*>(x + c);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = wave_sum(ss);
  if (lane_id() == 0) part[tid >> 6] = ss;
  __syncthreads();
  const float r = rsqrtf((part[0] + part[1] + part[2] + part[3]) / (float)P.hidden + P.eps);
  bf16* out = reinterpret_cast<bf16*>(P.out) + (int64_t)t * P.hidden;
  for (int c = 4 * tid; c < P.hidden; c += 4 * blockDim.x) {
    const float4 v = *reinterpret_cast<const float4*>(x + c);
    const float4 g = *reinterpret_cast<const float4*>(P.g + c);
    *reinterpret_cast<uint2*>(out + c) = make_uint2(pack_bf16(v.x * r * g.x, v.y * r * g.y),
                                                     pack_bf16(v.z * r * g.z, v.w * r * g.w));
  }
}

// One workgroup per row merges the row's slot summaries: log-sum-exp of s by
// a running maximum, the largest s + g (lowest column on equal values), and
// the target's s.
__global__ __launch_bounds__(256) void lm_sample_reduce_kernel(LmReduce P) {
  __shared__ float sm[4], sl[4], sp[4], ss[4], st[4];
  __shared__ int si[4];
  const int row = blockIdx.x, tid = threadIdx.x, lane = lane_id(), w = tid >> 6;
  const LogitSlot* rec = P.slots + (int64_t)row * P.n_slots;
  const float NEG = -__builtin_inff();
  float m = NEG, l = 0.f, pert = NEG, sb = NEG, stg = NEG;
  int bi = 0x7FFFFFFF;
  for (int j = tid; j < P.n_slots; j += blockDim.x) {
    const LogitSlot r = rec[j];
    const float mn = fmaxf(m, r.m);
    l = l * expf(m - mn) + r.l * expf(r.m - mn);
    m = mn;
    if (r.pert > pert || (r.pert == pert && r.idx < bi)) { pert = r.pert; sb = r.s_best; bi = r.idx; }
    stg = fmaxf(stg, r.s_tgt);
  }
  // across the wavefront, then across the four wavefronts
  for (int o = 32; o; o >>= 1) {
    const float m2 = __shfl_xor(m, o, 64), l2 = __shfl_xor(l, o, 64);
    const float mn = fmaxf(m, m2);
    l = (m == NEG ? 0.f : l * expf(m - mn)) + (m2 == NEG ? 0.f : l2 * expf(m2 - mn));
    m = mn;
    const float p2 = __shfl_xor(pert, o, 64), s2 = __shfl_xor(sb, o, 64);
    const int i2 = __shfl_xor(bi, o, 64);
    if (p2 > pert || (p2 == pert && i2 < bi)) { pert = p2; sb = s2; bi = i2; }
    stg = fmaxf(stg, __shfl_xor(stg, o, 64));
  }
  if (lane == 0) { sm[w] = m; sl[w] = l; sp[w] = pert; ss[w] = sb; si[w] = bi; st[w] = stg; }
  __syncthreads();
  if (tid == 0) {
    for (int k = 1; k < 4; ++k) {
      const float mn = fmaxf(m, sm[k]);
      l = (m == NEG ? 0.f : l * expf(m - mn)) + (sm[k] == NEG ? 0.f : sl[k] * expf(sm[k] - mn));
      m = mn;
      if (sp[k] > pert || (sp[k] == pert && si[k] < bi)) { pert = sp[k]; sb = ss[k]; bi = si[k]; }
      stg = fmaxf(stg, st[k]);
    }
    const float lse = m + logf(l);
    if (P.tokens) P.tokens[row] = bi;
    if (P.logprob) P.logprob[row] = sb - lse;
    if (P.lse) P.lse[row] = lse;
    if (P.target_logprob) P.target_logprob[row] = stg - lse;
  }
}

hipError_t launch_embed(const EmbedArgs& p, hipStream_t s) {
  if (p.n_tokens == 0) return hipSuccess;
  hipLaunchKernelGGL(embed_kernel, dim3(p.n_tokens), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_final_norm(const FinalNorm& p, hipStream_t s) {
  if (p.n_tokens == 0) return hipSuccess;
  hipLaunchKernelGGL(final_norm_kernel, dim3(p.n_tokens), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_lm_reduce(const LmReduce& p, hipStream_t s) {
  if (p.n_rows == 0) return hipSuccess;
  hipLaunchKernelGGL(lm_sample_reduce_kernel, dim3(p.n_rows), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace mcpu
