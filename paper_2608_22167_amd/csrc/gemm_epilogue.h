// Shared pieces of the GEMM kernels: the weight-row order of a 16-row block,
// the work-item order of the LDS-tiled kernels and the fused epilogues that
// finish an fp32 output tile held in LDS.
//   EPI_QKV      + bias, rotary embedding of q and k, q to the q buffer and
//                k / v straight into their KV-cache pages (the append)
//   EPI_RESIDUAL + bias + residual (fp32), e.g. h1 = x + o W_o^T + b_o
//   EPI_SWIGLU   + bias, gate/up pairs (rows 2j, 2j+1) -> clamped SwiGLU
//   EPI_BIAS     + bias (fp32)
//   EPI_LOGITS   vocabulary logits -> per-row, per-64-column sampling summaries
#pragma once
#include "device.h"
#include "kernels.h"

namespace mcpu {

// W row (output feature) that lane-row nl of 16-row block `blk` multiplies. For
// the QKV projection a block holds dims 8t..8t+7 and d/2+8t..d/2+8t+7 of one
// head, so both members of every rotary pair land in the same block.
template <int EPI>
__device__ __forceinline__ int block_row(const Gemm& P, int blk, int nl) {
  if (EPI == EPI_QKV) {
    const int D = P.head_dim, tph = D / 16;
    const int head = blk / tph, ti = blk - head * tph;
    return head * D + (nl < 8 ? 8 * ti + nl : D / 2 + 8 * ti + nl - 8);
  }
  return blk * 16 + nl;
}

constexpr int TILE_MAXG = 256;  // groups (experts) one tiled launch supports

// Position of local item L of a group with mt_g m-tiles and n_tn n-tiles, in
// bands of GM m-tiles (the last band may be shorter).
template <int GM>
__device__ __forceinline__ void band_order(int L, int mt_g, int n_tn, int& mt, int& tn) {
  const int full = mt_g / GM;
  if (L < full * GM * n_tn) {
    const int b = L / (GM * n_tn), r = L - b * (GM * n_tn);
    tn = r / GM;
    mt = b * GM + (r - tn * GM);
  } else {
    const int rem = mt_g - full * GM, r = L - full * GM * n_tn;
    tn = r / rem;
    mt = full * GM + (r - tn * rem);
  }
}

// Work item of this workgroup in a tiled launch: (group, m-tile, n-tile) of a
// BM x BN tiling of every group's rows against the n weight rows. mt_start
// (LDS, TILE_MAXG + 1 ints) receives the exclusive prefix of m-tiles per group,
// computed from group_off on the device so the host only bounds the grid.
// Items are cut into eight contiguous ranges, one per XCD (workgroups are
// dealt to the XCDs round robin), so that a band's reuse stays in one L2.
// Returns false for a workgroup past the last item. Contains a barrier: every
// thread of the workgroup calls it. row_start (LDS, TILE_MAXG + 1 ints), if
// given, receives each group's first row and, last, the end of the last group.
template <int BM, int BN, int GM>
__device__ bool tile_of_block(const Gemm& P, int* mt_start, int& grp, int& mt, int& tn, int* row_start = nullptr) {
  const int lane = threadIdx.x & 63, wave = uniform((int)threadIdx.x >> 6);
  const int G = P.n_groups;
  if (wave == 0) {  // one wavefront, 64 groups per pass
    int carry = 0;
    for (int g0 = 0; g0 < G; g0 += 64) {
      const int g = g0 + lane;
      int cnt = 0;
      if (g < G) {
        const int r0 = P.group_off ? P.group_off[g] : 0;
        const int r1 = P.group_off ? P.group_off[g + 1] : P.n_rows;
        cnt = (max(r1 - r0, 0) + BM - 1) / BM;
        if (row_start) {  // the group's rows, r0 .. r1 - 1
          row_start[g] = r0;
          if (g == G - 1) row_start[G] = r1;
        }
      }
      const int incl = wave_incl_scan(cnt);
      if (g < G) mt_start[g] = carry + incl - cnt;
      carry += __shfl(incl, 63, 64);
    }
    if (lane == 0) mt_start[G] = carry;
  }
  __syncthreads();
  const int n_tn = (P.n + BN - 1) / BN;
  const int total = mt_start[G] * n_tn;
  const int chunk = (total + 7) >> 3;
  const int local = blockIdx.x >> 3;
  const int item = (blockIdx.x & 7) * chunk + local;
  if (local >= chunk || item >= total) return false;
  // group of the item: last g with mt_start[g] * n_tn <= item (each group owns mt_g * n_tn items)
  int lo = 0, hi = G - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (mt_start[mid] * n_tn <= item) lo = mid; else hi = mid - 1;
  }
  grp = uniform(lo);
  band_order<GM>(item - mt_start[grp] * n_tn, mt_start[grp + 1] - mt_start[grp], n_tn, mt, tn);
  return true;
}

// Grid bound of a tiled launch: sum_g ceil(rows_g / BM) <= rows / BM + groups
// m-tiles, rounded up to whole rounds of the eight XCDs.
inline int64_t tile_grid(const Gemm& g, int bm, int bn) {
  const int64_t mt_bound = g.group_off ? (int64_t)g.n_rows / bm + g.n_groups : ((int64_t)g.n_rows + bm - 1) / bm;
  const int64_t items = mt_bound * ((g.n + bn - 1) / bn);
  return (items + 7) / 8 * 8;
}

__device__ __forceinline__ float swiglu(float gate, float up, float alpha, float limit, float beta) {
  gate = fminf(gate, limit);
  up = fminf(fmaxf(up, -limit), limit);
  return gate / (1.0f + expf(-alpha * gate)) * (up + beta);
}

// 8 consecutive elements from fp32 (16 or 32 bytes; p 16-byte aligned)
__device__ __forceinline__ void store8(float* p, const float v[8]) {
  reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ __forceinline__ void store8(bf16* p, const float v[8]) {
  *reinterpret_cast<uint4*>(p) =
      make_uint4(pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3]), pack_bf16(v[4], v[5]), pack_bf16(v[6], v[7]));
}

// cr[m * ld + n]: the finished fp32 tile for token rows m0 .. m0 + mrows - 1 and
// the nblk 16-row weight blocks starting at blk0.
// A thread's bias values in the SwiGLU and bias/residual epilogues: the same
// columns in every pass over a tile's rows, so a kernel that writes a tile in
// several passes loads them once (epilogue_bias) and hands them to each pass.
struct EpiBias {
  float4 v;
};
template <int EPI>
__device__ __forceinline__ EpiBias epilogue_bias(const Gemm& P, int blk0, int nblk, int grp) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const float* bias = P.bias + (int64_t)grp * P.bias_group_stride;
  EpiBias e{make_float4(0.f, 0.f, 0.f, 0.f)};
  if constexpr (EPI == EPI_SWIGLU) {
    const int cols = nblk * 8;
    if (cols <= nt && tid < (nt / cols) * cols) {
      const int c = tid % cols, col = (blk0 + (c >> 3)) * 16 + 2 * (c & 7);
      e.v.x = bias[col];
      e.v.y = bias[col + 1];
    }
  } else if constexpr (EPI == EPI_RESIDUAL || EPI == EPI_BIAS) {
    const int nq = nblk * 4;
    if (nq <= nt && tid < (nt / nq) * nq) {
      const int n = blk0 * 16 + 4 * (tid % nq);
      e.v = make_float4(bias[n], bias[n + 1], bias[n + 2], bias[n + 3]);
    }
  }
  return e;
}

template <typename T, int EPI>
__device__ void epilogue(const Gemm& P, const float* cr, int ld, int m0, int mrows, int blk0, int nblk,
                         int grp, const EpiBias* pre = nullptr) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const float* bias = P.bias + (int64_t)grp * P.bias_group_stride;
  if constexpr (EPI == EPI_QKV) {
    // One item = (token row m, 16-row block b): dims j0 .. j0 + 7 and
    // d/2 + j0 .. d/2 + j0 + 7 of one head, so the token's position and page
    // are looked up once per 8 rotary pairs and q and k leave in 8-element
    // stores (a K page keeps 8 consecutive dims of a slot together).
    const int D = P.head_dim, tph = D / 16, half = D / 2;
    for (int idx = tid; idx < mrows * nblk; idx += nt) {
      const int b = idx % nblk, m = idx / nblk, t = m0 + m;
      const int blk = blk0 + b, head = blk / tph, ti = blk - head * tph;
      const int j0 = 8 * ti;  // dim within the head, < D/2
      const int f_lo = head * D + j0, f_hi = f_lo + half;
      float lo[8], hi[8];
      {
        // the tile rows need not be 16-byte aligned (odd strides avoid bank
        // conflicts in some kernels): 4-byte reads; bias rows are aligned
        const float* c = cr + m * ld + 16 * b;
        const float4* bl = reinterpret_cast<const float4*>(bias + f_lo);
        const float4* bh = reinterpret_cast<const float4*>(bias + f_hi);
        const float4 b0 = bl[0], b1 = bl[1], b2 = bh[0], b3 = bh[1];
        const float bb[16] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w,
                              b2.x, b2.y, b2.z, b2.w, b3.x, b3.y, b3.z, b3.w};
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          lo[i] = c[i] + bb[i];
          hi[i] = c[8 + i] + bb[8 + i];
        }
      }
      const int pos = P.tok_pos[t];
      if (head < P.hq + P.hkv) {  // q or k: rotate the pairs (j, j + d/2)
        if (pos < 0 || pos >= P.rope_max_pos) {
          set_error(P.err, 2);
          continue;
        }
        const float4* cp = reinterpret_cast<const float4*>(P.rope_cos + (int64_t)pos * half + j0);
        const float4* sp = reinterpret_cast<const float4*>(P.rope_sin + (int64_t)pos * half + j0);
        const float4 ca = cp[0], cb = cp[1], sa = sp[0], sb = sp[1];
        const float cs[8] = {ca.x, ca.y, ca.z, ca.w, cb.x, cb.y, cb.z, cb.w};
        const float sn[8] = {sa.x, sa.y, sa.z, sa.w, sb.x, sb.y, sb.z, sb.w};
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float a = lo[i], bb = hi[i];
          lo[i] = a * cs[i] - bb * sn[i];
          hi[i] = a * sn[i] + bb * cs[i];
        }
      }
      if (head < P.hq) {
        T* q = reinterpret_cast<T*>(P.q_out) + ((int64_t)t * P.hq + head) * D;
        store8(q + j0, lo);
        store8(q + j0 + half, hi);
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
        T* kp = reinterpret_cast<T*>(P.k_pool) + ((int64_t)page * P.hkv + (head - P.hq)) * PAGE * D;
        store8(kp + k_off(slot, j0), lo);
        store8(kp + k_off(slot, j0 + half), hi);
      } else {
        T* vp = reinterpret_cast<T*>(P.v_pool) + ((int64_t)page * P.hkv + (head - P.hq - P.hkv)) * PAGE * D;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          Elem<T>::store(vp, v_off(slot, j0 + i), lo[i]);
          Elem<T>::store(vp, v_off(slot, j0 + half + i), hi[i]);
        }
      }
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    // A thread keeps one output column (its two bias values read once) and
    // walks the rows, so no global load waits behind an earlier iteration's
    // store (a loop that re-read the bias per element did, one L2 round trip
    // per element). A wavefront's consecutive columns leave as one store per row.
    T* out = reinterpret_cast<T*>(P.out);
    const int half_n = P.n / 2, cols = nblk * 8;
    if (cols <= nt) {
      const int lanes = nt / cols;
      if (tid < lanes * cols) {
        const int c = tid % cols, b = c >> 3, j = c & 7;
        const int col = (blk0 + b) * 16 + 2 * j;
        const float bg = pre ? pre->v.x : bias[col], bu = pre ? pre->v.y : bias[col + 1];
        const float* cp = cr + 16 * b + 2 * j;
        T* op = out + (int64_t)m0 * half_n + (blk0 + b) * 8 + j;
        for (int m = tid / cols; m < mrows; m += lanes)
          Elem<T>::store(op, (int64_t)m * half_n,
                         swiglu(cp[m * ld] + bg, cp[m * ld + 1] + bu, P.swiglu_alpha, P.swiglu_limit, P.swiglu_beta));
      }
    } else {
      for (int idx = tid; idx < mrows * cols; idx += nt) {
        const int j = idx & 7, b = (idx >> 3) % nblk, m = (idx >> 3) / nblk;
        const int col = (blk0 + b) * 16 + 2 * j;
        const float gate = cr[m * ld + 16 * b + 2 * j] + bias[col];
        const float up = cr[m * ld + 16 * b + 2 * j + 1] + bias[col + 1];
        Elem<T>::store(out, (int64_t)(m0 + m) * half_n + (blk0 + b) * 8 + j,
                       swiglu(gate, up, P.swiglu_alpha, P.swiglu_limit, P.swiglu_beta));
      }
    }
  } else if constexpr (EPI == EPI_LOGITS) {
    // Sixteen lanes per (row, 64-column slot), four consecutive columns each
    // (one Philox draw gives their four noise words): the slot's maximum of s,
    // its sum of exp(s - max), the largest s + g with its column (lowest
    // column on equal values) and the target's s, reduced across the sixteen
    // lanes and stored as one LogitSlot.
    LogitSlot* out = reinterpret_cast<LogitSlot*>(P.out);
    const int n_slots = (P.n + LOGIT_SLOT - 1) / LOGIT_SLOT;
    const int nslot = (nblk * 16 + LOGIT_SLOT - 1) / LOGIT_SLOT, c_end = (blk0 + nblk) * 16;
    const int sub = tid & 15;
    const float NEG = -__builtin_inff();
    const int items = mrows * nslot, stride = nt >> 4;
    auto slot = [&](int it, int pos, int seq, int tgt) __attribute__((always_inline)) {
      const int m = it / nslot, j = it - m * nslot, row = m0 + m;
      const int c0 = blk0 * 16 + j * LOGIT_SLOT + 4 * sub;
      const float* cp = cr + m * ld + j * LOGIT_SLOT + 4 * sub;
      float sv[4], g[4] = {0.f, 0.f, 0.f, 0.f};
      if (!P.greedy && c0 < c_end) {
        const U32x4 r = philox4x32_10(U32x4{(uint32_t)(c0 >> 2), (uint32_t)pos, (uint32_t)seq, LOGIT_RNG_TAG},
                                      (uint32_t)P.seed, (uint32_t)(P.seed >> 32));
        g[0] = gumbel_of(r.x); g[1] = gumbel_of(r.y); g[2] = gumbel_of(r.z); g[3] = gumbel_of(r.w);
      }
      float mx = NEG, pert = NEG, sb = NEG, st = NEG;
      int bi = 0x7FFFFFFF;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool ok = c0 + i < c_end;
        sv[i] = ok ? cp[i] * P.inv_temp : NEG;
        mx = fmaxf(mx, sv[i]);
        const float pv = sv[i] + g[i];
        if (ok && pv > pert) { pert = pv; sb = sv[i]; bi = c0 + i; }
        if (ok && c0 + i == tgt) st = sv[i];
      }
#pragma unroll
      for (int o = 8; o; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 16));
      float sum = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) sum += c0 + i < c_end ? __builtin_amdgcn_exp2f((sv[i] - mx) * 1.44269504088896341f) : 0.f;
#pragma unroll
      for (int o = 8; o; o >>= 1) {
        sum += __shfl_xor(sum, o, 16);
        const float p2 = __shfl_xor(pert, o, 16), s2 = __shfl_xor(sb, o, 16);
        const int i2 = __shfl_xor(bi, o, 16);
        if (p2 > pert || (p2 == pert && i2 < bi)) { pert = p2; sb = s2; bi = i2; }
        st = fmaxf(st, __shfl_xor(st, o, 16));
      }
      if (sub == 0) {
        LogitSlot r;
        r.m = mx; r.l = sum; r.pert = pert; r.s_best = sb; r.idx = bi; r.s_tgt = st; r.pad[0] = r.pad[1] = 0.f;
        out[(int64_t)row * n_slots + (c0 / LOGIT_SLOT)] = r;
      }
    };
    // two items per round: the rows' positions, sequence ids and targets are
    // loaded for both before either stores (a load may not pass a store to a
    // possibly aliasing address)
    for (int it = tid >> 4; it < items; it += 2 * stride) {
      const int it2 = it + stride;
      const bool two = it2 < items;  // uniform per 16 lanes
      const int r1 = m0 + it / nslot, r2 = m0 + (two ? it2 : it) / nslot;
      const bool draw = !P.greedy;
      const int pos1 = draw ? P.row_pos[r1] : 0, seq1 = draw ? P.row_seq[r1] : 0;
      const int pos2 = draw ? P.row_pos[r2] : 0, seq2 = draw ? P.row_seq[r2] : 0;
      const int tg1 = P.target ? P.target[r1] : -1, tg2 = P.target ? P.target[r2] : -1;
      slot(it, pos1, seq1, tg1);
      if (two) slot(it2, pos2, seq2, tg2);
    }
  } else {  // EPI_RESIDUAL, EPI_BIAS: fp32 rows, 4 consecutive features per thread
    // As above: fixed features per thread (bias read once); residual rows of
    // four passes are loaded before their stores.
    float* out = reinterpret_cast<float*>(P.out);
    const int nq = nblk * 4;
    auto row = [&](int m, int q, const float4& bv, const float4* r) __attribute__((always_inline)) {
      const int64_t o = (int64_t)(m0 + m) * P.n + blk0 * 16 + 4 * q;
      float4 v = make_float4(cr[m * ld + 4 * q] + bv.x, cr[m * ld + 4 * q + 1] + bv.y,
                             cr[m * ld + 4 * q + 2] + bv.z, cr[m * ld + 4 * q + 3] + bv.w);
      if constexpr (EPI == EPI_RESIDUAL) {
        v.x += r->x; v.y += r->y; v.z += r->z; v.w += r->w;
      }
      *reinterpret_cast<float4*>(out + o) = v;
    };
    if (nq <= nt) {
      const int lanes = nt / nq;
      if (tid < lanes * nq) {
        const int q = tid % nq, n = blk0 * 16 + 4 * q;
        const float4 bv = pre ? pre->v : make_float4(bias[n], bias[n + 1], bias[n + 2], bias[n + 3]);
        for (int m = tid / nq; m < mrows; m += 4 * lanes) {
          float4 r[4];
          if constexpr (EPI == EPI_RESIDUAL) {
#pragma unroll
            for (int u = 0; u < 4; ++u)
              if (m + u * lanes < mrows)
                r[u] = *reinterpret_cast<const float4*>(P.residual + (int64_t)(m0 + m + u * lanes) * P.n + n);
          }
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (m + u * lanes < mrows) row(m + u * lanes, q, bv, &r[u]);
        }
      }
    } else {
      for (int idx = tid; idx < mrows * nq; idx += nt) {
        const int q = idx % nq, m = idx / nq, n = blk0 * 16 + 4 * q;
        const float4 bv = make_float4(bias[n], bias[n + 1], bias[n + 2], bias[n + 3]);
        float4 r;
        if constexpr (EPI == EPI_RESIDUAL)
          r = *reinterpret_cast<const float4*>(P.residual + (int64_t)(m0 + m) * P.n + n);
        row(m, q, bv, &r);
      }
    }
  }
}

}  // namespace mcpu
