// Paged GQA attention with per-head sinks for gfx950.
//
// The step's attention (every new token attends to its sequence's cached keys,
// plus the sink logit of its head) is split three ways:
//   plan    one workgroup maps tokens to (sequence, position) and cuts each
//           token's visible page range into splits of `pps` pages;
//   split   one wavefront per (split, KV head) streams the split's K and V
//           pages and keeps a running max / sum / weighted value sum for the
//           G = Hq / Hkv query heads that share the KV head;
//   combine one workgroup per token merges the splits and adds the sink to
//           the normaliser.
// The score and value products run on the matrix cores: with keys as rows
// and the G query heads as columns (padded to 16), S^T = K q^T is one 16x16
// tile per page, and O^T += V^T P^T consumes it without any lane shuffle
// because the score tile's lane layout is exactly the value product's B
// operand layout. The page format (include/mcpu.h) makes every K and V
// fragment load a contiguous 512 B - 1 KiB segment per wavefront.
#include "device.h"
#include "kernels.h"

namespace mcpu {

constexpr float LOG2E = 1.4426950408889634f;

// ---------------------------------------------------------------------------
// plan
// ---------------------------------------------------------------------------

__device__ __forceinline__ int token_splits(int pos, int window, int pps) {
  int lo = window > 0 ? max(0, pos - window + 1) : 0;
  int pages = pos / PAGE - lo / PAGE + 1;
  return (pages + pps - 1) / pps;
}

__device__ __forceinline__ int seq_of_token(const int32_t* cu_q, int batch, int t) {
  // last b with cu_q[b] <= t
  int lo = 0, hi = batch - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (cu_q[mid] <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ bool is_prefill(const AttnPlan& P, int b) {
  return P.cu_q && P.prefill_min_q > 0 && P.cu_q[b + 1] - P.cu_q[b] >= P.prefill_min_q;
}

// Exclusive prefix of `local` over the 1024 threads of the block, and the total.
__device__ int block_exclusive_scan(int local, int* sums, int& total) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const int incl = wave_incl_scan(local);
  const int wave = tid >> 6, lane = tid & 63;
  if (lane == 63) sums[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    const int w = lane < (nt >> 6) ? sums[lane] : 0;
    const int wi = wave_incl_scan(w);
    if (lane < (nt >> 6)) sums[64 + lane] = wi - w;  // exclusive prefix of wave totals
    if (lane == (nt >> 6) - 1) sums[128] = wi;       // grand total
  }
  __syncthreads();
  const int excl = sums[64 + wave] + incl - local;
  total = sums[128];
  __syncthreads();  // sums is reused by the next scan
  return excl;
}

// Workgroups 1.. of the plan launch: the layer's first RMSNorm, y = x /
// sqrt(mean(x^2) + eps) * g, on four rows per workgroup (256 threads a row,
// float4 j of a thread at features 4 (t + 256 j)), so that the norm and the
// plan, both short and independent, share one launch.
template <typename T>
__device__ void plan_norm_rows(const RmsNorm& N) {
  __shared__ float part[16];
  constexpr int NVMAX = 8;  // hidden <= 8192
  const int tid = threadIdx.x, sub = tid & 255, grp = tid >> 8, H = N.hidden;
  const int row = (blockIdx.x - 1) * 4 + grp;
  const bool live = row < N.n_tokens;
  const float* x = N.x + (int64_t)(live ? row : 0) * H;
  float4 xv[NVMAX], gv[NVMAX];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NVMAX; ++j) {
    const int i = (sub + 256 * j) * 4;
    if (i < H) {
      xv[j] = *reinterpret_cast<const float4*>(x + i);
      gv[j] = *reinterpret_cast<const float4*>(N.g + i);
      ss += xv[j].x * xv[j].x + xv[j].y * xv[j].y + xv[j].z * xv[j].z + xv[j].w * xv[j].w;
    }
  }
  ss = wave_sum(ss);
  if (lane_id() == 0) part[tid >> 6] = ss;
  __syncthreads();
  const float tot = part[4 * grp] + part[4 * grp + 1] + part[4 * grp + 2] + part[4 * grp + 3];
  const float inv = 1.0f / sqrtf(tot / (float)H + N.eps);
  if (!live) return;
  T* out = reinterpret_cast<T*>(N.out) + (int64_t)row * H;
#pragma unroll
  for (int j = 0; j < NVMAX; ++j) {
    const int i = (sub + 256 * j) * 4;
    if (i < H)
      store4(out + i, make_float4(xv[j].x * inv * gv[j].x, xv[j].y * inv * gv[j].y,
                                xv[j].z * inv * gv[j].z, xv[j].w * inv * gv[j].w));
  }
}

__global__ __launch_bounds__(1024) void attn_plan_kernel(AttnPlan P) {
  if (blockIdx.x > 0) {
    if (P.norm_dtype == 0) plan_norm_rows<float>(P.norm);
    else plan_norm_rows<bf16>(P.norm);
    return;
  }
  __shared__ int sums[160];
  const int tid = threadIdx.x, nt = blockDim.x;
  for (int i = tid; i < P.n_zero; i += nt) P.zero[i] = 0;
  // tokens: positions and split counts (no splits for prefill sequences)
  const int per = (P.n_tokens + nt - 1) / nt;
  const int t0 = min(P.n_tokens, tid * per), t1 = min(P.n_tokens, t0 + per);
  int local = 0;
  for (int t = t0; t < t1; ++t) {
    int b = P.cu_q ? seq_of_token(P.cu_q, P.batch, t) : t;
    int pos = P.seq_lens[b] + (P.cu_q ? t - P.cu_q[b] : 0);
    local += is_prefill(P, b) ? 0 : token_splits(pos, P.window, P.pps);
  }
  int total = 0;
  int run = block_exclusive_scan(local, sums, total);
  for (int t = t0; t < t1; ++t) {
    int b = P.cu_q ? seq_of_token(P.cu_q, P.batch, t) : t;
    int pos = P.seq_lens[b] + (P.cu_q ? t - P.cu_q[b] : 0);
    P.tok_seq[t] = b;
    P.tok_pos[t] = pos;
    P.split_start[t] = run;
    const int ns = is_prefill(P, b) ? 0 : token_splits(pos, P.window, P.pps);
    // the token's ns splits share its np pages evenly (sizes differ by at most one)
    const int lo = P.window > 0 ? max(0, pos - P.window + 1) : 0;
    const int first = lo / PAGE, np = pos / PAGE - first + 1;
    for (int k = 0; k < ns && run + k < P.host_total_splits; ++k) {
      SplitDesc d;
      d.t = t; d.b = b; d.p = pos; d.lo = lo;
      d.pg0 = first + (int)((int64_t)k * np / ns);
      d.pg1 = first + (int)((int64_t)(k + 1) * np / ns);
      d.pad0 = d.pad1 = 0;
      P.split_desc[run + k] = d;
    }
    run += ns;
  }
  if (tid == 0) {
    P.split_start[P.n_tokens] = total;
    if (P.host_total_splits >= 0 && total != P.host_total_splits) set_error(P.err, 8);
  }
  if (!P.blk_start) return;
  // sequences: prefill blocks of prefill_qb tokens
  const int perb = (P.batch + nt - 1) / nt;
  const int b0 = min(P.batch, tid * perb), b1 = min(P.batch, b0 + perb);
  local = 0;
  for (int b = b0; b < b1; ++b)
    if (is_prefill(P, b)) local += (P.cu_q[b + 1] - P.cu_q[b] + P.prefill_qb - 1) / P.prefill_qb;
  run = block_exclusive_scan(local, sums, total);
  for (int b = b0; b < b1; ++b) {
    P.blk_start[b] = run;
    if (is_prefill(P, b)) run += (P.cu_q[b + 1] - P.cu_q[b] + P.prefill_qb - 1) / P.prefill_qb;
  }
  if (tid == 0) {
    P.blk_start[P.batch] = total;
    if (total != P.host_total_blocks) set_error(P.err, 8);
  }
}

hipError_t launch_attn_plan(const AttnPlan& p, hipStream_t s) {
  int blocks = 1;
  if (p.norm_dtype >= 0) {
    if (p.norm.hidden % 4 || p.norm.hidden > 8192) return hipErrorInvalidValue;
    blocks += (p.norm.n_tokens + 3) / 4;
  }
  hipLaunchKernelGGL(attn_plan_kernel, dim3(blocks), dim3(1024), 0, s, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// split: one wavefront per (split, KV head)
// ---------------------------------------------------------------------------

// One KV head's K and V of one page, loaded with the streaming policy: a page
// is read by one wavefront (C2 attention 218 -> 194 us).
template <typename T, int D>
struct PageFrags {
  Frag<T> k[D / 32];   // chunk c holds dims 32c + 8 * (lane / 16) .. +7 of key lane % 16
  Frag4<T> v[D / 16];  // block n holds V[4 * (lane / 16) + r][16n + lane % 16]
  __device__ __forceinline__ void load(const T* kp, const T* vp, int lane) {
#pragma unroll
    for (int c = 0; c < D / 32; ++c) k[c].load_stream(kp + (64 * c + lane) * 8);
#pragma unroll
    for (int n = 0; n < D / 16; ++n) v[n].load_stream(vp + (64 * n + lane) * 4);
  }
};

// Online-softmax state of one wavefront: the running maximum (log2 units), the
// running sum and the value accumulator (lane (hl, grp) holds dims
// 16 n + 4 grp .. + 3 of query head hl).
template <int D>
struct SoftmaxAcc {
  float m = -INFINITY, l = 0.f;
  f32x4 acc[D / 16];
  __device__ __forceinline__ SoftmaxAcc() {
#pragma unroll
    for (int n = 0; n < D / 16; ++n) acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // One page: S^T = K q^T on the matrix cores, mask keys outside [lo, p] (and
  // the whole page if `valid` is false), rescale, and O^T += V^T P^T.
  template <typename T>
  __device__ __forceinline__ void page(const PageFrags<T, D>& cur, const Frag<T> (&qf)[D / 32], bool valid,
                                       int key0, int lo, int p, float scale_log2) {
    f32x4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < D / 32; ++c) sc = mma32(cur.k[c], qf[c], sc);
    // sc[r] = score of key slot key0 + r for query head lane % 16
    float x[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int pos = key0 + r;
      x[r] = (valid && pos >= lo && pos <= p) ? sc[r] * scale_log2 : -INFINITY;
    }
    float mloc = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float m_new = fmaxf(m, mloc);
    // m_new is -inf only while every key so far was masked (missing pages)
    const bool live = m_new != -INFINITY;
    const float alpha = live ? __builtin_amdgcn_exp2f(m - m_new) : 1.0f;
    float pr[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) pr[r] = live ? __builtin_amdgcn_exp2f(x[r] - m_new) : 0.f;
    l *= alpha;
#pragma unroll
    for (int n = 0; n < D / 16; ++n) {
      acc[n] *= alpha;
      acc[n] = mma16_p(cur.v[n], pr, acc[n], n == 0 ? &l : nullptr);
    }
    m = m_new;
  }
  // the sum over the wavefront's four key-row groups
  __device__ __forceinline__ float l_total() const {
    float t = l + __shfl_xor(l, 16, 64);
    return t + __shfl_xor(t, 32, 64);
  }
};

// The token, position and page range of split s (shared by both kernels).
struct SplitRange {
  int t, b, p, lo, pg0, pg1;
};
// (the plan kernel wrote it as one 32-byte record: a single load, where a
// search over split_start would chain several dependent ones)
__device__ __forceinline__ SplitRange split_range(const AttnSplit& P, int s) {
  const SplitDesc d = P.split_desc[s];
  SplitRange r;
  r.t = uniform(d.t);
  r.b = uniform(d.b);
  r.p = uniform(d.p);
  r.lo = uniform(d.lo);
  r.pg0 = uniform(d.pg0);
  r.pg1 = uniform(d.pg1);
  // a record the plan did not write (device arrays disagree with the host's
  // plan) may be stale: every field is checked before it addresses memory
  if (r.t < 0 || r.t >= P.n_tokens || r.b < 0 || r.b >= P.batch || r.p < 0 || r.p / PAGE >= P.max_pages ||
      r.pg0 < 0 || r.pg0 >= r.pg1 || r.pg1 > P.max_pages) {
    if (lane_id() == 0) set_error(P.err, 1);
    r.t = 0;
    r.b = 0;
    r.pg0 = r.pg1 = 0;
  }
  return r;
}

template <typename T, int D>
__device__ __forceinline__ void load_q(Frag<T> (&qf)[D / 32], const AttnSplit& P, int t, int g) {
  const int lane = lane_id(), G = P.hq / P.hkv, hl = lane & 15, grp = lane >> 4;
  const T* qb = reinterpret_cast<const T*>(P.q) + ((int64_t)t * P.hq + g * G + hl) * D + 8 * grp;
#pragma unroll
  for (int c = 0; c < D / 32; ++c) {
    if (hl < G) qf[c].load(qb + 32 * c); else qf[c].zero();
  }
}

template <typename T, int D, int WAVES, int PF>
__global__ __launch_bounds__(64 * WAVES) void attn_split_kernel(AttnSplit P) {
  const int lane = lane_id();
  const int item = blockIdx.x * WAVES + uniform(threadIdx.x >> 6);
  const int s = item / P.hkv, g = item - (item / P.hkv) * P.hkv;
  if (s >= P.n_splits) return;
  const SplitRange R = split_range(P, s);
  const int pg0 = R.pg0, pg1 = R.pg1;
  const int G = P.hq / P.hkv;
  const int hl = lane & 15, grp = lane >> 4;
  Frag<T> qf[D / 32];
  load_q<T, D>(qf, P, R.t, g);

  const T* kpool = reinterpret_cast<const T*>(P.k_pool);
  const T* vpool = reinterpret_cast<const T*>(P.v_pool);
  const int32_t* ptab = P.page_table + (int64_t)R.b * P.max_pages;
  const int64_t head_off = (int64_t)g * PAGE * D, page_elems = (int64_t)P.hkv * PAGE * D;
  SoftmaxAcc<D> st;

  // PF-deep ring of pages: while page i is consumed, pages i+1 .. i+PF-1 are
  // in flight and page i+PF is issued into its slot. Loads are branch-free: a
  // slot past the split re-reads the last page, a missing page reads page 0,
  // and both are masked out of the softmax instead of skipped. (The wait for
  // each page-table entry also waits for the pages in flight; reading 64
  // entries with one vector load up front avoids that but costs 17 VGPRs,
  // five wavefronts per SIMD down to four, and was 4% slower at 64
  // sequences: this kernel hides its latency with occupancy.)
  const int npg = pg1 - pg0;
  PageFrags<T, D> ring[PF];
  bool ok[PF];
  auto fetch = [&](int slot, int i) {
    const int pg = pg0 + min(i, npg - 1);
    int id = uniform(ptab[pg]);
    const bool good = id >= 0 && id < P.n_pages;
    if (!good && lane == 0 && i < npg) set_error(P.err, 1);
    id = good ? id : 0;
    ok[slot] = good && i < npg;
    ring[slot].load(kpool + id * page_elems + head_off, vpool + id * page_elems + head_off, lane);
  };
  auto consume = [&](int slot, int i) {
    st.page(ring[slot], qf, ok[slot], (pg0 + i) * PAGE + 4 * grp, R.lo, R.p, P.scale_log2);
  };
  if (npg > 0) {
#pragma unroll
    for (int u = 0; u < PF; ++u) fetch(u, u);
    int i = 0;
    for (; i + PF <= npg; i += PF) {
#pragma unroll
      for (int u = 0; u < PF; ++u) {
        consume(u, i + u);
        fetch(u, i + u + PF);
      }
    }
#pragma unroll
    for (int u = 0; u < PF; ++u)
      if (i + u < npg) consume(u, i + u);
  }

  const float l_tot = st.l_total();
  if (hl < G) {
    const int64_t row = (int64_t)s * P.hq + g * G + hl;
    if (grp == 0) {
      P.part_ml[row * 2 + 0] = st.m;
      P.part_ml[row * 2 + 1] = l_tot;
    }
    float* pa = P.part_acc + row * D + 4 * grp;
#pragma unroll
    for (int n = 0; n < D / 16; ++n)
      *reinterpret_cast<float4*>(pa + 16 * n) = make_float4(st.acc[n][0], st.acc[n][1], st.acc[n][2], st.acc[n][3]);
  }
}

// Sliding-window layers: every decode token's window spans at most MAXP pages
// and is one split. One wavefront per (token, KV head) reads the window's page
// ids with one vector load (lane j: page j), issues every page's K and V loads
// at once, and finishes the token itself: the sink joins the normaliser and o
// is written in the layer dtype, so no partials and no combine pass are
// needed. (The split-K kernel, whose pages follow a page-table load each and
// keep two in flight, left short windows waiting on memory latency.)
//
// The KV heads of a token go to one workgroup of WW wavefronts (wavefront w:
// head w), the workgroups in eight contiguous ranges, one per XCD (workgroups
// are dealt to the XCDs round robin): a token's pages, which hold all its KV
// heads side by side, are then read by one compute unit.
template <typename T, int D, int MAXP, int WW>
__global__ __launch_bounds__(64 * WW) void attn_window_kernel(AttnSplit P) {
  const int lane = lane_id();
  const int items = P.n_splits * P.hkv;
  const int nblk = (items + WW - 1) / WW, chunk = (nblk + 7) >> 3;
  const int blk = (blockIdx.x & 7) * chunk + (blockIdx.x >> 3);
  if ((int)(blockIdx.x >> 3) >= chunk || blk >= nblk) return;
  const int item = blk * WW + uniform(threadIdx.x >> 6);
  if (item >= items) return;  // no barriers below: a wavefront may leave alone
  const int s = item / P.hkv, g = item - (item / P.hkv) * P.hkv;
  const SplitRange R = split_range(P, s);
  if (R.pg0 == R.pg1) return;  // an invalid record (error bit set): no token to finish
  const int npg = min(R.pg1 - R.pg0, MAXP);
  if (lane == 0 && R.pg1 - R.pg0 > MAXP) set_error(P.err, 8);  // the launch does not fit this plan
  const int G = P.hq / P.hkv;
  const int hl = lane & 15, grp = lane >> 4;
  const int my_id = lane < npg ? P.page_table[(int64_t)R.b * P.max_pages + R.pg0 + lane] : 0;
  Frag<T> qf[D / 32];
  load_q<T, D>(qf, P, R.t, g);
  const T* kpool = reinterpret_cast<const T*>(P.k_pool);
  const T* vpool = reinterpret_cast<const T*>(P.v_pool);
  const int64_t head_off = (int64_t)g * PAGE * D, page_elems = (int64_t)P.hkv * PAGE * D;
  // Every page is requested before the first is used, unconditionally (slots
  // past the window re-read its last page, a missing page reads page 0; both
  // masked), and the error bit is set after the loads: a conditional load or
  // atomic among them leaves the compiler unable to count the loads in
  // flight, and it then waits for each page before requesting the next.
  PageFrags<T, D> pages[MAXP];
  bool ok[MAXP];
  bool bad = false;
#pragma unroll
  for (int u = 0; u < MAXP; ++u) {
    int id = __shfl(my_id, min(u, npg - 1), 64);
    const bool good = id >= 0 && id < P.n_pages;
    bad = bad || (!good && u < npg);
    ok[u] = good && u < npg;
    id = good ? id : 0;
    pages[u].load(kpool + id * page_elems + head_off, vpool + id * page_elems + head_off, lane);
  }
  if (bad && lane == 0) set_error(P.err, 1);
  SoftmaxAcc<D> st;
#pragma unroll
  for (int u = 0; u < MAXP; ++u)
    if (u < npg) st.page(pages[u], qf, ok[u], (R.pg0 + u) * PAGE + 4 * grp, R.lo, R.p, P.scale_log2);
  const float l_tot = st.l_total();
  if (hl < G) {
    // o_h = 2^{m - M} acc / (2^{sink log2e - M} + 2^{m - M} l), M = max(sink log2e, m)
    const int h = g * G + hl;
    float M = P.sinks ? P.sinks[h] * LOG2E : -INFINITY;
    float L = P.sinks ? 1.0f : 0.0f;
    float f = 0.f;
    if (st.m != -INFINITY) {
      if (st.m > M) {
        L *= __builtin_amdgcn_exp2f(M - st.m);
        M = st.m;
      }
      f = __builtin_amdgcn_exp2f(st.m - M);
      L += f * l_tot;
    }
    T* o = reinterpret_cast<T*>(P.o) + ((int64_t)R.t * P.hq + h) * D + 4 * grp;
#pragma unroll
    for (int n = 0; n < D / 16; ++n)
#pragma unroll
      for (int r = 0; r < 4; ++r) Elem<T>::store(o, 16 * n + r, L > 0.f ? f * st.acc[n][r] / L : 0.f);
  }
}

#ifndef MCPU_WINDOW_WAVES
#define MCPU_WINDOW_WAVES 8
#endif
constexpr int WINDOW_WAVES = MCPU_WINDOW_WAVES;  // wavefronts per window workgroup

template <typename T, int D, int WAVES = 1, int PF = 2>
hipError_t split_impl(const AttnSplit& p, hipStream_t s) {
  int64_t items = (int64_t)p.n_splits * p.hkv;
  int blocks = (int)((items + WAVES - 1) / WAVES);
  if (blocks == 0) return hipSuccess;
  if (p.o) {
    constexpr int WW = WINDOW_WAVES;
    const int64_t nblk = (items + WW - 1) / WW, grid = (nblk + 7) / 8 * 8;
    hipLaunchKernelGGL((attn_window_kernel<T, D, WINDOW_MAX_PAGES, WW>), dim3((unsigned)grid), dim3(64 * WW), 0, s, p);
  } else {
    hipLaunchKernelGGL((attn_split_kernel<T, D, WAVES, PF>), dim3(blocks), dim3(64 * WAVES), 0, s, p);
  }
  return hipGetLastError();
}

hipError_t launch_attn_split(int dtype, int head_dim, const AttnSplit& p, hipStream_t s) {
  if (dtype == 0) return head_dim == 32 ? split_impl<float, 32>(p, s) : split_impl<float, 64>(p, s);
  return head_dim == 32 ? split_impl<bf16, 32>(p, s) : split_impl<bf16, 64>(p, s);
}

// ---------------------------------------------------------------------------
// combine: o_h = sum_s 2^{m_s - M} acc_s / (2^{sink_h log2e - M} + sum_s 2^{m_s - M} l_s)
// ---------------------------------------------------------------------------

// One wavefront per (token, query head); lane i owns dim i. The splits are
// merged in order with a running maximum, so one pass reads each partial once.
template <typename T, int D>
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnCombine P) {
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = lane_id();
  if (item >= P.n_tokens * P.hq) return;
  const int t = uniform(item / P.hq), h = uniform(item - (item / P.hq) * P.hq);
  const int s0 = min(uniform(P.split_start[t]), P.n_splits);
  const int s1 = min(uniform(P.split_start[t + 1]), P.n_splits);
  if (s0 == s1) return;  // a prefill token: its row comes from the prefill kernel
  float M = P.sinks ? P.sinks[h] * LOG2E : -INFINITY;
  float L = P.sinks ? 1.0f : 0.0f;  // the sink's own term, 2^(sink - M)
  float a = 0.f;
  const bool act = lane < D;
  constexpr int U = 4;
  int s = s0;
  for (; s + U <= s1; s += U) {
    float m[U], l[U], v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t row = (int64_t)(s + u) * P.hq + h;
      m[u] = P.part_ml[row * 2];
      l[u] = P.part_ml[row * 2 + 1];
      v[u] = act ? P.part_acc[row * D + lane] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (m[u] == -INFINITY) continue;  // a split whose pages were all missing
      if (m[u] > M) {
        const float r = __builtin_amdgcn_exp2f(M - m[u]);
        L *= r;
        a *= r;
        M = m[u];
      }
      const float f = __builtin_amdgcn_exp2f(m[u] - M);
      L += f * l[u];
      a += f * v[u];
    }
  }
  for (; s < s1; ++s) {
    const int64_t row = (int64_t)s * P.hq + h;
    const float m = P.part_ml[row * 2];
    if (m == -INFINITY) continue;
    if (m > M) {
      const float r = __builtin_amdgcn_exp2f(M - m);
      L *= r;
      a *= r;
      M = m;
    }
    const float f = __builtin_amdgcn_exp2f(m - M);
    L += f * P.part_ml[row * 2 + 1];
    a += f * (act ? P.part_acc[row * D + lane] : 0.f);
  }
  if (act) {
    T* o = reinterpret_cast<T*>(P.o) + ((int64_t)t * P.hq + h) * D;
    Elem<T>::store(o, lane, L > 0.f ? a / L : 0.f);
  }
}

hipError_t launch_attn_combine(int dtype, int head_dim, const AttnCombine& p, hipStream_t s) {
  if (p.n_tokens == 0) return hipSuccess;
  dim3 grid((p.n_tokens * p.hq + 3) / 4), block(256);
  if (dtype == 0) {
    if (head_dim == 32) hipLaunchKernelGGL((attn_combine_kernel<float, 32>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((attn_combine_kernel<float, 64>), grid, block, 0, s, p);
  } else {
    if (head_dim == 32) hipLaunchKernelGGL((attn_combine_kernel<bf16, 32>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((attn_combine_kernel<bf16, 64>), grid, block, 0, s, p);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// prefill: a chunk of new tokens attending causally to its sequence's pages
// ---------------------------------------------------------------------------

// A workgroup of four wavefronts owns QB consecutive new tokens of one
// sequence and one KV head. The matrix-core columns are (token, query head)
// pairs, 64 per wavefront: 64 / G tokens times the G query heads that share
// the KV head. The workgroup walks the pages from the first key any of its
// tokens sees to its last token's page, two pages (32 keys) per step, staged
// through LDS (double buffered) for all four wavefronts. Per step a wavefront
// forms S^T = K Q^T for both pages and its four 16-column tiles, masks keys
// outside each column's causal (and window) range, updates the running
// maximum and normaliser per column, and accumulates O^T += V^T P^T with one
// 16x16x32 product per tile that consumes both pages' scores as they sit in
// the lanes. The sink enters the normaliser at the end.
template <int G>
struct PrefillShape {
  static constexpr int TPW = 64 / G;    // tokens per wavefront
  static constexpr int QB = 4 * TPW;    // tokens per workgroup
};

// Only the groupings with a kernel instance (prefill_impl) report a block
// size; for the others the planner sends every chunk to split-K attention.
int prefill_block_tokens(int group) {
  switch (group) {
    case 4: return PrefillShape<4>::QB;
    case 8: return PrefillShape<8>::QB;
    default: return 0;
  }
}

template <typename T, int D, int G>
__global__ __launch_bounds__(256) void attn_prefill_kernel(AttnPrefill P) {
  using SH = PrefillShape<G>;
  constexpr int PE = PAGE * D;                          // elements of one page of one KV head
  constexpr int CH = 16 / sizeof(T);                    // elements per 16-byte chunk
  constexpr int NCH = 4 * PE / CH;                      // chunks per step (K and V of two pages)
  constexpr int PT = NCH / 256;                         // chunks per thread
  static_assert(NCH % 256 == 0, "a step's pages must split evenly over the workgroup");
  __shared__ __align__(16) T kv[2][4][PE];              // [buffer][K page a, K page b, V pages a and b interleaved]
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  const int g = blockIdx.x % P.hkv;
  const int blk = P.n_blocks - 1 - (int)(blockIdx.x / P.hkv);  // latest (heaviest) blocks first
  int lo_b = 0, hi_b = P.batch - 1;                            // sequence: last b with blk_start[b] <= blk
  while (lo_b < hi_b) {
    const int mid = (lo_b + hi_b + 1) >> 1;
    if (P.blk_start[mid] <= blk) lo_b = mid; else hi_b = mid - 1;
  }
  const int b = uniform(lo_b);
  const int q0 = P.cu_q[b], q1 = P.cu_q[b + 1];
  const int t0 = uniform(q0 + (blk - P.blk_start[b]) * SH::QB);
  const int ntok = min(SH::QB, q1 - t0);
  const int p_first = uniform(P.seq_lens[b] + (t0 - q0)), p_last = p_first + ntok - 1;
  const int lo = P.window > 0 ? max(0, p_first - P.window + 1) : 0;
  const int pg_lo = lo / PAGE;
  int n_steps = (p_last / PAGE - pg_lo + 2) / 2;
  if (ntok <= 0 || p_first < 0 || p_last / PAGE >= P.max_pages) {
    if (tid == 0) set_error(P.err, 1);
    n_steps = 0;
  }
  const int32_t* ptab = P.page_table + (int64_t)b * P.max_pages;
  const int64_t page_elems = (int64_t)P.hkv * PE;

  // this lane's column in each of the wavefront's four 16-column tiles
  const int fr = lane & 15, grp = lane >> 4;
  int pos[4], head[4];
  bool valid[4];
  Frag<T> qf[4][D / 32];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c = 16 * j + fr;
    const int ti = wave * SH::TPW + c / G;
    valid[j] = ti < ntok;
    pos[j] = p_first + ti;
    head[j] = g * G + c % G;
    const int trow = min(max(t0 + ti, 0), P.n_tokens - 1);  // in range even if the tables disagree
    const T* qp = reinterpret_cast<const T*>(P.q) + ((int64_t)trow * P.hq + head[j]) * D + 8 * grp;
#pragma unroll
    for (int cc = 0; cc < D / 32; ++cc) {
      qf[j][cc].load(qp + 32 * cc);
      qf[j][cc].keep_if(valid[j]);
    }
  }

  // staging: chunk i of a step is piece i / (PE / CH) (K a, K b, V a, V b) at
  // element offset (i % (PE / CH)) * CH; pages past the range repeat the last
  // one and missing pages read page 0 (both masked below)
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  struct Regs {
    u32x4 v[PT];
  };
  // page ids are wave-uniform: read them with scalar loads, whose wait counter
  // is separate from the vector loads kept in flight below
  auto page_id = [&](int step, int which, bool& ok) __attribute__((always_inline)) {
    const int pg = uniform(min(pg_lo + 2 * step + which, p_last / PAGE));
    const int id = load_uniform(ptab, pg);
    ok = id >= 0 && id < P.n_pages;
    return ok ? id : 0;
  };
  auto fetch = [&](Regs& st, int step) __attribute__((always_inline)) {
    step = min(step, max(n_steps - 1, 0));
    bool oka, okb;
    const int ida = page_id(step, 0, oka), idb = page_id(step, 1, okb);
#pragma unroll
    for (int u = 0; u < PT; ++u) {
      const int i = tid + 256 * u, piece = i / (PE / CH), off = (i % (PE / CH)) * CH;
      const T* pool = reinterpret_cast<const T*>(piece < 2 ? P.k_pool : P.v_pool);
      const int id = (piece & 1) ? idb : ida;
      st.v[u] = *reinterpret_cast<const u32x4*>(pool + id * page_elems + (int64_t)g * PE + off);
    }
  };
  // K pages keep the page format; the V pages of a step are interleaved in
  // blocks of 256 elements (the 64 lanes' 4-value fragments of one 16-dim
  // tile): [tile n][page a, page b], so the two halves of a PV operand are
  // 512 bytes apart and load as one register quadruple
  auto stage = [&](const Regs& st, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < PT; ++u) {
      const int i = tid + 256 * u, piece = i / (PE / CH), off = (i % (PE / CH)) * CH;
      T* dst = piece < 2 ? &kv[buf][piece][off] : &kv[buf][2][((off >> 8) * 2 + piece - 2) * 256 + (off & 255)];
      *reinterpret_cast<u32x4*>(dst) = st.v[u];
    }
  };

  // Per column: running maximum m (log2 units) and the accumulators of
  // O^T = V^T P^T, plus a tile against ones that sums the (rounded) weights.
  // The maximum is raised lazily: a step rescales only when some column's
  // scores exceed its m by more than RESCALE (weights then stay below
  // 2^RESCALE); every weight uses the same m as its normaliser, so the result
  // is the same quotient.
  constexpr float RESCALE = 8.0f;
  const float inv_scale = 1.0f / P.scale_log2;
  float m_run[4], m_sub[4], thr[4];
  f32x4 acc[D / 16][4], accl[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    m_run[j] = -INFINITY;
    m_sub[j] = 0.f;
    thr[j] = -INFINITY;
    accl[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int n = 0; n < D / 16; ++n) acc[n][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  Frag4<T> one;
  ones(one);
  // keys a step may need to mask: past the wave's first token (causal), before
  // its last token's window, or on a missing or out-of-range page
  const int pos_lo_w = p_first + wave * SH::TPW;
  const int pos_hi_w = min(pos_lo_w + SH::TPW - 1, p_last);
  const int pg_last = p_last / PAGE;

  auto compute = [&](int step, int buf) __attribute__((always_inline)) {
    bool ok[2];
    page_id(step, 0, ok[0]);
    page_id(step, 1, ok[1]);
    const int pg0 = pg_lo + 2 * step, k0 = pg0 * PAGE;
    const bool edge = k0 + 2 * PAGE - 1 > pos_lo_w || (P.window > 0 && k0 < pos_hi_w - P.window + 1) ||
                      !ok[0] || !ok[1] || pg0 + 1 > pg_last;
    // scores: sc[pg][j][r] = q(column j) . k(key 4 grp + r of page pg)
    f32x4 sc[2][4];
#pragma unroll
    for (int pg = 0; pg < 2; ++pg) {
      Frag<T> kf[D / 32];
#pragma unroll
      for (int cc = 0; cc < D / 32; ++cc) kf[cc].load(&kv[buf][pg][(64 * cc + lane) * 8]);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        sc[pg][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int cc = 0; cc < D / 32; ++cc) sc[pg][j] = mma32(kf[cc], qf[j][cc], sc[pg][j]);
      }
    }
    // wave-uniform: mask keys outside each column's range. The empty asm
    // keeps this a branch: if-converted, its compares and selects would run
    // on every step.
    if (__builtin_expect(edge, 0)) {
      asm volatile("");
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int hi = pos[j], lo_c = P.window > 0 ? pos[j] - P.window + 1 : 0;
#pragma unroll
        for (int pg = 0; pg < 2; ++pg)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int kp = k0 + pg * PAGE + 4 * grp + r;
            const bool in = ok[pg] && pg0 + pg <= pg_last && kp >= lo_c && kp <= hi;
            sc[pg][j][r] = in ? sc[pg][j][r] : -INFINITY;
          }
      }
    }
    // Each lane takes the largest of its 8 raw scores per column; the step
    // rescales only when one of them exceeds the column's threshold
    // (m + RESCALE in raw score units), and only then forms the column
    // maximum across the four row groups.
    float mloc[4];
    bool raise = false;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      mloc[j] = vmax(vmax(vmax(sc[0][j][0], sc[0][j][1]), vmax(sc[0][j][2], sc[0][j][3])),
                     vmax(vmax(sc[1][j][0], sc[1][j][1]), vmax(sc[1][j][2], sc[1][j][3])));
      raise = raise || mloc[j] > thr[j];
    }
    if (__builtin_expect(__builtin_amdgcn_ballot_w64(raise) != 0, 0)) {  // wave-uniform rescale (kept a branch)
      asm volatile("");
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float mstep = max_over_rows(mloc[j]) * P.scale_log2;
        const float m_new = fmaxf(m_run[j], mstep);
        const float alpha = m_new == -INFINITY ? 1.0f : __builtin_amdgcn_exp2f(m_run[j] - m_new);
        accl[j] *= alpha;
#pragma unroll
        for (int n = 0; n < D / 16; ++n) acc[n][j] *= alpha;
        m_run[j] = m_new;
        m_sub[j] = m_new == -INFINITY ? 0.f : m_new;  // masked scores give 2^-inf = 0
        thr[j] = (m_new + RESCALE) * inv_scale;
      }
    }
    PVFrag<T> vf[D / 16];
#pragma unroll
    for (int n = 0; n < D / 16; ++n) vf[n].load(&kv[buf][2][2 * n * 256 + lane * 4], &kv[buf][2][(2 * n + 1) * 256 + lane * 4]);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float msub = m_sub[j];
      float pa[4], pb[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        pa[r] = __builtin_amdgcn_exp2f(fmaf(sc[0][j][r], P.scale_log2, -msub));
        pb[r] = __builtin_amdgcn_exp2f(fmaf(sc[1][j][r], P.scale_log2, -msub));
      }
      accl[j] = mma32_pv(one, one, pa, pb, accl[j]);
#pragma unroll
      for (int n = 0; n < D / 16; ++n) acc[n][j] = mma32_pv(vf[n], pa, pb, acc[n][j]);
    }
  };

  // Step j's pages are loaded into register set j % R and staged into LDS
  // buffer j & 1: while step s is computed, steps s + 1 .. s + R are in flight
  // (L2 latency exceeds one step's products). The loop is unrolled R times so
  // set indices are constants; only the products are conditional (loads past
  // the last step are clamped and their staged copies never read).
  constexpr int R = 4;
  if (n_steps > 0) {
    Regs rs[R];
#pragma unroll
    for (int u = 0; u < R; ++u) {
      fetch(rs[u], u);
      __builtin_amdgcn_sched_barrier(0);
    }
    stage(rs[0], 0);
    fetch(rs[0], R);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    for (int step = 0; step < n_steps; step += R) {
#pragma unroll
      for (int u = 0; u < R; ++u) {
        if (step + u < n_steps) compute(step + u, u & 1);
        __builtin_amdgcn_sched_barrier(0);
        stage(rs[(u + 1) % R], (u + 1) & 1);
        fetch(rs[(u + 1) % R], step + u + 1 + R);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
      }
    }
  }

  // normalise with the sink and store this lane's 4 dims of each column
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float l_tot = accl[j][0];  // every row of the ones tile holds the column's sum
    float M = m_run[j], scale = 1.0f;
    if (P.sinks) {
      const float sk = P.sinks[head[j]] * LOG2E;
      const float Mt = fmaxf(M, sk);
      const float f = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(M - Mt);
      l_tot = l_tot * f + __builtin_amdgcn_exp2f(sk - Mt);
      scale = f;
    }
    const float inv = l_tot > 0.f ? scale / l_tot : 0.f;
    if (valid[j]) {
      T* o = reinterpret_cast<T*>(P.o) + ((int64_t)(t0 + wave * SH::TPW + (16 * j + fr) / G) * P.hq + head[j]) * D +
             4 * grp;
#pragma unroll
      for (int n = 0; n < D / 16; ++n)
#pragma unroll
        for (int r = 0; r < 4; ++r) Elem<T>::store(o, 16 * n + r, acc[n][j][r] * inv);
    }
  }
}

template <typename T, int D>
static hipError_t prefill_impl(int group, const AttnPrefill& p, hipStream_t s) {
  dim3 grid((unsigned)(p.n_blocks * p.hkv)), block(256);
  switch (group) {
    case 4: hipLaunchKernelGGL((attn_prefill_kernel<T, D, 4>), grid, block, 0, s, p); break;
    case 8: hipLaunchKernelGGL((attn_prefill_kernel<T, D, 8>), grid, block, 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attn_prefill(int dtype, int head_dim, int group, const AttnPrefill& p, hipStream_t s) {
  if (p.n_blocks == 0) return hipSuccess;
  if (dtype == 0) return head_dim == 32 ? prefill_impl<float, 32>(group, p, s) : prefill_impl<float, 64>(group, p, s);
  return head_dim == 32 ? prefill_impl<bf16, 32>(group, p, s) : prefill_impl<bf16, 64>(group, p, s);
}

// ---------------------------------------------------------------------------
// KV append: copy new keys / values into their pages, bit for bit
// ---------------------------------------------------------------------------

template <typename T, int D>
__global__ __launch_bounds__(256) void kv_append_kernel(KvAppend P) {
  const int t = blockIdx.x;
  const int b = P.cu_q ? seq_of_token(P.cu_q, P.batch, t) : t;
  const int pos = P.seq_lens[b] + (P.cu_q ? t - P.cu_q[b] : 0);
  const int lp = pos >= 0 ? pos / PAGE : -1;
  int page = (lp >= 0 && lp < P.max_pages) ? P.page_table[(int64_t)b * P.max_pages + lp] : -1;
  if (page < 0 || page >= P.n_pages) {
    if (threadIdx.x == 0) set_error(P.err, 1);
    return;
  }
  const int slot = pos % PAGE;
  const T* kn = reinterpret_cast<const T*>(P.k_new) + (int64_t)t * P.hkv * D;
  const T* vn = reinterpret_cast<const T*>(P.v_new) + (int64_t)t * P.hkv * D;
  T* kp = reinterpret_cast<T*>(P.k_pool) + (int64_t)page * P.hkv * PAGE * D;
  T* vp = reinterpret_cast<T*>(P.v_pool) + (int64_t)page * P.hkv * PAGE * D;
  for (int e = threadIdx.x; e < P.hkv * D; e += blockDim.x) {
    const int g = e / D, i = e - g * D;
    kp[(int64_t)g * PAGE * D + k_off(slot, i)] = kn[e];
    vp[(int64_t)g * PAGE * D + v_off(slot, i)] = vn[e];
  }
}

hipError_t launch_kv_append(int dtype, int head_dim, const KvAppend& p, hipStream_t s) {
  if (p.n_tokens == 0) return hipSuccess;
  dim3 grid(p.n_tokens), block(256);
  if (dtype == 0) {
    if (head_dim == 32) hipLaunchKernelGGL((kv_append_kernel<float, 32>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((kv_append_kernel<float, 64>), grid, block, 0, s, p);
  } else {
    if (head_dim == 32) hipLaunchKernelGGL((kv_append_kernel<bf16, 32>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((kv_append_kernel<bf16, 64>), grid, block, 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace mcpu
