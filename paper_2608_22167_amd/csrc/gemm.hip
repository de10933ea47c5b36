// Weight-streaming grouped GEMM for the decode step on gfx950.
//
// At decode every projection of the layer is skinny: a few to a few hundred
// token rows against a weight matrix that is read exactly once, so the kernels
// are bound by streaming the weights from HBM. One workgroup owns a 16-row
// slab of one group's weight matrix (one expert, or the single dense matrix)
// and all token rows of that group; its KW wavefronts split the reduction
// dimension, each streaming a contiguous K range with one 16x16x32 matrix-core
// product per 32-wide chunk and token block, then the partial tiles are summed
// through LDS in a fixed order and a fused epilogue finishes the slab:
//   EPI_QKV      + bias, rotary embedding of q and k, q to the q buffer and
//                k / v straight into their KV-cache pages (the append)
//   EPI_RESIDUAL + bias + residual (fp32), e.g. h1 = x + o W_o^T + b_o
//   EPI_SWIGLU   + bias, gate/up pairs (rows 2j, 2j+1) -> clamped SwiGLU
//   EPI_BIAS     + bias (fp32)
// Token rows may be gathered through row_src (the expert-sorted order), so the
// permuted activations are never materialised.
#include "device.h"
#include "kernels.h"

namespace mcpu {

// W row (output feature) that lane-row nl of slab `tile` multiplies. For the
// QKV projection a slab holds dims 8t..8t+7 and d/2+8t..d/2+8t+7 of one head,
// so both members of every rotary pair land in the same workgroup.
template <int EPI>
__device__ __forceinline__ int slab_row(const Gemm& P, int tile, int nl) {
  if (EPI == EPI_QKV) {
    const int D = P.head_dim, tph = D / 16;
    const int head = tile / tph, ti = tile - head * tph;
    return head * D + (nl < 8 ? 8 * ti + nl : D / 2 + 8 * ti + nl - 8);
  }
  return tile * 16 + nl;
}

__device__ __forceinline__ float swiglu(float gate, float up, float alpha, float limit, float beta) {
  gate = fminf(gate, limit);
  up = fminf(fmaxf(up, -limit), limit);
  return gate / (1.0f + expf(-alpha * gate)) * (up + beta);
}

template <typename T, int EPI>
__device__ void epilogue(const Gemm& P, const float* cr, int m0, int mrows, int tile, int grp) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const float* bias = P.bias + (int64_t)grp * P.bias_group_stride;
  if constexpr (EPI == EPI_QKV) {
    const int D = P.head_dim, tph = D / 16, half = D / 2;
    const int head = tile / tph, ti = tile - head * tph;
    for (int idx = tid; idx < mrows * 8; idx += nt) {
      const int m = idx >> 3, i = idx & 7, t = m0 + m;
      const int j = 8 * ti + i;  // dim within the head, < D/2
      const int f_lo = head * D + j, f_hi = f_lo + half;
      float lo = cr[m * 17 + i] + bias[f_lo];
      float hi = cr[m * 17 + 8 + i] + bias[f_hi];
      const int pos = P.tok_pos[t];
      if (head < P.hq + P.hkv) {  // q or k: rotate the pair (j, j + d/2)
        if (pos < 0 || pos >= P.rope_max_pos) {
          set_error(P.err, 2);
          continue;
        }
        const float c = P.rope_cos[(int64_t)pos * half + j], s = P.rope_sin[(int64_t)pos * half + j];
        const float a = lo, b = hi;
        lo = a * c - b * s;
        hi = a * s + b * c;
      }
      if (head < P.hq) {
        T* q = reinterpret_cast<T*>(P.q_out) + ((int64_t)t * P.hq + head) * D;
        Elem<T>::store(q, j, lo);
        Elem<T>::store(q, j + half, hi);
        continue;
      }
      const int lp = pos >> 4;
      const int seq = P.tok_seq[t];
      const int page = (pos >= 0 && lp < P.max_pages) ? P.page_table[(int64_t)seq * P.max_pages + lp] : -1;
      if (page < 0 || page >= P.n_pages) {
        set_error(P.err, 1);
        continue;
      }
      const int slot = pos & 15;
      if (head < P.hq + P.hkv) {
        const int g = head - P.hq;
        T* kp = reinterpret_cast<T*>(P.k_pool) + ((int64_t)page * P.hkv + g) * PAGE * D;
        Elem<T>::store(kp, k_off(slot, j), lo);
        Elem<T>::store(kp, k_off(slot, j + half), hi);
      } else {
        const int g = head - P.hq - P.hkv;
        T* vp = reinterpret_cast<T*>(P.v_pool) + ((int64_t)page * P.hkv + g) * PAGE * D;
        Elem<T>::store(vp, v_off(slot, j), lo);
        Elem<T>::store(vp, v_off(slot, j + half), hi);
      }
    }
  } else if constexpr (EPI == EPI_RESIDUAL) {
    float* out = reinterpret_cast<float*>(P.out);
    for (int idx = tid; idx < mrows * 16; idx += nt) {
      const int m = idx >> 4, n = idx & 15;
      const int64_t o = (int64_t)(m0 + m) * P.n + tile * 16 + n;
      out[o] = cr[m * 17 + n] + bias[tile * 16 + n] + P.residual[o];
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    T* out = reinterpret_cast<T*>(P.out);
    const int half_n = P.n / 2;
    for (int idx = tid; idx < mrows * 8; idx += nt) {
      const int m = idx >> 3, j = idx & 7;
      const float gate = cr[m * 17 + 2 * j] + bias[tile * 16 + 2 * j];
      const float up = cr[m * 17 + 2 * j + 1] + bias[tile * 16 + 2 * j + 1];
      Elem<T>::store(out, (int64_t)(m0 + m) * half_n + tile * 8 + j,
                     swiglu(gate, up, P.swiglu_alpha, P.swiglu_limit, P.swiglu_beta));
    }
  } else {  // EPI_BIAS
    float* out = reinterpret_cast<float*>(P.out);
    for (int idx = tid; idx < mrows * 16; idx += nt) {
      const int m = idx >> 4, n = idx & 15;
      out[(int64_t)(m0 + m) * P.n + tile * 16 + n] = cr[m * 17 + n] + bias[tile * 16 + n];
    }
  }
}

template <typename T, int MB, int KW, int EPI>
__global__ __launch_bounds__(64 * KW) void gemm_ws_kernel(Gemm P) {
  __shared__ float red[KW * MB * 256];
  const int lane = lane_id(), wave = uniform(threadIdx.x >> 6);
  const int n_tiles = P.n >> 4;
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
  const T* wp = reinterpret_cast<const T*>(P.w) + grp * P.w_group_stride +
                (int64_t)slab_row<EPI>(P, tile, nl) * P.k + 8 * kg;
  const int nC = P.k >> 5;
  const int c0 = wave * nC / KW, c1 = (wave + 1) * nC / KW;

  for (int m0 = r0; m0 < r1; m0 += MB * 16) {
    const int mrows = min(MB * 16, r1 - m0);
    const int amb = (mrows + 15) >> 4;
    const T* xp[MB];
    bool xv[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int row = m0 + mb * 16 + nl;
      xv[mb] = row < r1;
      const int src = xv[mb] ? (P.row_src ? P.row_src[row] : row) : 0;
      xp[mb] = reinterpret_cast<const T*>(P.x) + (int64_t)src * P.k + 8 * kg;
    }
    f32x4 acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll 4
    for (int c = c0; c < c1; ++c) {
      Frag<T> a;
      a.load(wp + c * 32);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        if (mb < amb) {
          Frag<T> bx;
          if (xv[mb]) bx.load(xp[mb] + c * 32); else bx.zero();
          acc[mb] = mma32(a, bx, acc[mb]);
        }
      }
    }

    // fixed-order reduction of the KW partial tiles
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[((wave * MB + mb) * 4 + r) * 64 + lane] = acc[mb][r];
    __syncthreads();
    constexpr int PER = (MB * 256 + 64 * KW - 1) / (64 * KW);
    float sum[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int e = threadIdx.x + q * 64 * KW;
      float v = 0.f;
      if (e < MB * 256) {
#pragma unroll
        for (int w = 0; w < KW; ++w) v += red[w * MB * 256 + e];
      }
      sum[q] = v;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int e = threadIdx.x + q * 64 * KW;
      if (e < MB * 256) {
        const int mb = e >> 8, r = (e >> 6) & 3, ln = e & 63;
        const int n = 4 * (ln >> 4) + r, m = mb * 16 + (ln & 15);
        red[m * 17 + n] = sum[q];
      }
    }
    __syncthreads();
    epilogue<T, EPI>(P, red, m0, mrows, tile, grp);
    __syncthreads();
  }
}

template <typename T, int MB, int KW>
static hipError_t gemm_epi(const Gemm& g, hipStream_t s) {
  dim3 grid((g.n / 16) * g.n_groups), block(64 * KW);
  switch (g.epi) {
    case EPI_QKV: hipLaunchKernelGGL((gemm_ws_kernel<T, MB, KW, EPI_QKV>), grid, block, 0, s, g); break;
    case EPI_RESIDUAL: hipLaunchKernelGGL((gemm_ws_kernel<T, MB, KW, EPI_RESIDUAL>), grid, block, 0, s, g); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_ws_kernel<T, MB, KW, EPI_SWIGLU>), grid, block, 0, s, g); break;
    default: hipLaunchKernelGGL((gemm_ws_kernel<T, MB, KW, EPI_BIAS>), grid, block, 0, s, g); break;
  }
  return hipGetLastError();
}

template <typename T>
static hipError_t gemm_dispatch(const Gemm& g, hipStream_t s) {
  const int mb = (g.max_rows_per_group + 15) / 16;
  if (mb <= 1) return gemm_epi<T, 1, 8>(g, s);
  if (mb <= 2) return gemm_epi<T, 2, 8>(g, s);
  if (mb <= 4) return gemm_epi<T, 4, 8>(g, s);
  if (mb <= 8) return gemm_epi<T, 8, 4>(g, s);
  return gemm_epi<T, 16, 4>(g, s);
}

hipError_t launch_gemm(int dtype, int expert_fmt, const Gemm& g, hipStream_t s) {
  if (expert_fmt != 0) return hipErrorNotSupported;
  if (g.n_groups == 0 || g.n == 0) return hipSuccess;
  return dtype == 0 ? gemm_dispatch<float>(g, s) : gemm_dispatch<bf16>(g, s);
}

}  // namespace mcpu
