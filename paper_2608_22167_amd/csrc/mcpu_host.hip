// Host side of the C ABI (include/mcpu.h): argument checks, the page
// allocator, launch planning from the caller's host copies of the sequence
// lengths, workspace carving and the launch order of each entry point.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <set>
#include <string>
#include <vector>

#include "../../include/mcpu.h"
#include "kernels.h"
#include "kernels_lm.h"

using namespace mcpu;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_TRY(expr)                                                              \
  do {                                                                             \
    hipError_t e_ = (expr);                                                        \
    if (e_ != hipSuccess) return fail(MCPU_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

constexpr int PAGE_SIZE = 16;
constexpr int SPLIT_EXTRA = 4096;   // splits beyond one per token that the workspace holds
constexpr int PPS_MIN = 16;         // minimum pages per attention split
constexpr int PPS_MAX = 256;        // maximum, unless the workspace's split count needs more
constexpr int TARGET_WAVES = 3072;  // (split, KV head) wavefronts the planner aims for (measured: ~100 pages per split)
constexpr int PREFILL_MIN_Q = 16;   // sequences adding this many tokens or more use the prefill kernel

size_t dtype_bytes(const mcpu_layer_cfg* c) { return c->dtype == MCPU_F32 ? 4 : 2; }

int check_cfg(const mcpu_layer_cfg* c) {
  if (!c) return fail(MCPU_EINVAL, "cfg is NULL");
  if (c->page_size != PAGE_SIZE) return fail(MCPU_EINVAL, "page_size must be 16 (got %d)", c->page_size);
  if (c->dtype != MCPU_F32 && c->dtype != MCPU_BF16) return fail(MCPU_EINVAL, "dtype %d", c->dtype);
  if (c->head_dim != 32 && c->head_dim != 64)
    return fail(MCPU_EUNSUPPORTED, "head_dim %d (supported: 32, 64)", c->head_dim);
  if (c->n_kv_heads <= 0 || c->n_q_heads <= 0 || c->n_q_heads % c->n_kv_heads)
    return fail(MCPU_EINVAL, "n_q_heads %d must be a positive multiple of n_kv_heads %d", c->n_q_heads,
                c->n_kv_heads);
  if (c->n_q_heads / c->n_kv_heads > 16)
    return fail(MCPU_EUNSUPPORTED, "more than 16 query heads per KV head");
  if (c->hidden <= 0 || c->hidden % 32 || c->hidden > 8192)
    return fail(MCPU_EINVAL, "hidden %d must be a multiple of 32 in (0, 8192]", c->hidden);
  if (c->ffn_dim <= 0 || c->ffn_dim % 32) return fail(MCPU_EINVAL, "ffn_dim %d must be a multiple of 32", c->ffn_dim);
  if ((c->n_q_heads * c->head_dim) % 32) return fail(MCPU_EINVAL, "n_q_heads * head_dim must be a multiple of 32");
  if (c->n_experts <= 0 || c->n_experts > 64) return fail(MCPU_EINVAL, "n_experts %d not in [1, 64]", c->n_experts);
  if (c->top_k <= 0 || c->top_k > std::min(8, c->n_experts)) return fail(MCPU_EINVAL, "top_k %d", c->top_k);
  if (c->window < 0) return fail(MCPU_EINVAL, "window %d", c->window);
  if (c->expert_fmt != MCPU_EXPERT_DENSE && c->expert_fmt != MCPU_EXPERT_MXFP4 &&
      c->expert_fmt != MCPU_EXPERT_MXFP4_NATIVE)
    return fail(MCPU_EINVAL, "expert_fmt %d", c->expert_fmt);
  if (c->expert_fmt != MCPU_EXPERT_DENSE && c->dtype != MCPU_BF16)
    return fail(MCPU_EUNSUPPORTED, "MXFP4 experts need a bf16 layer");
  if (c->expert_fmt == MCPU_EXPERT_MXFP4_NATIVE && (c->hidden % 64 || c->ffn_dim % 64))
    return fail(MCPU_EUNSUPPORTED, "native MXFP4 experts need hidden and ffn_dim multiples of 64");
  if (!(c->rms_eps >= 0.f)) return fail(MCPU_EINVAL, "rms_eps");
  return MCPU_OK;
}

// bump allocator over the workspace; a null base computes the size only
struct Carve {
  char* base;
  size_t off = 256;  // bytes 0..255: device error word
  explicit Carve(void* b) : base((char*)b) {}
  template <typename T> T* take(size_t count) {
    off = (off + 255) & ~size_t(255);
    T* p = base ? (T*)(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
  void* take_bytes(size_t n) { return take<char>(n); }
};

int32_t* err_word(void* ws) { return (int32_t*)ws; }

// ---- kernel timing (mcpu_timing_*) ------------------------------------------
struct KernelTimer {
  std::vector<hipEvent_t> start, stop;
  int armed = 0, next = 0;
};
KernelTimer g_timers[MCPU_KERNEL_COUNT];

// Records an event pair around the launch(es) made during its lifetime.
struct Timed {
  KernelTimer* t = nullptr;
  hipStream_t s;
  Timed(int kernel, hipStream_t st) : s(st) {
    KernelTimer& k = g_timers[kernel];
    if (k.next < k.armed) {
      t = &k;
      hipEventRecord(k.start[k.next], s);
    }
  }
  ~Timed() {
    if (t) {
      hipEventRecord(t->stop[t->next], s);
      ++t->next;
    }
  }
};

// per-token visible page count
int token_pages(int pos, int window) {
  int lo = window > 0 ? std::max(0, pos - window + 1) : 0;
  return pos / PAGE_SIZE - lo / PAGE_SIZE + 1;
}

struct AttnPlanHost {
  int n_tokens = 0, pps = PPS_MIN, n_splits = 0, max_pos = 0;
  int prefill_min_q = 0, prefill_qb = 0, n_blocks = 0;  // chunked-prefill work (0 blocks: none)
};

// Validate host positions and choose pages-per-split so that the split count
// fits the workspace (<= n_tokens + SPLIT_EXTRA) and fills the GPU.
int plan_attention(const mcpu_layer_cfg* c, int batch, int max_pages, const int32_t* hsl,
                   const int32_t* hcu, AttnPlanHost* out) {
  if (!hsl) return fail(MCPU_EINVAL, "host_seq_lens is NULL");
  int T = hcu ? hcu[batch] : batch;
  if (hcu && hcu[0] != 0) return fail(MCPU_EINVAL, "host_cu_q[0] must be 0");
  std::vector<int> pages;
  pages.reserve(T);
  long long total_pages = 0, blocks = 0;
  int max_pos = 0;
  // chunks of PREFILL_MIN_Q or more tokens go to the prefill kernel when it
  // supports the head grouping; everything else is split per token
  const int qb = hcu ? prefill_block_tokens(c->n_q_heads / c->n_kv_heads) : 0;
  const int min_q = qb > 0 ? PREFILL_MIN_Q : 0;
  for (int b = 0; b < batch; ++b) {
    int q = hcu ? hcu[b + 1] - hcu[b] : 1;
    if (q < 0) return fail(MCPU_EINVAL, "host_cu_q is not non-decreasing at %d", b);
    if (hsl[b] < 0) return fail(MCPU_EINVAL, "seq_lens[%d] = %d < 0", b, hsl[b]);
    const bool pre = min_q > 0 && q >= min_q;
    if (pre) blocks += (q + qb - 1) / qb;
    for (int i = 0; i < q; ++i) {
      int pos = hsl[b] + i;
      if (pos / PAGE_SIZE >= max_pages)
        return fail(MCPU_EINVAL, "sequence %d position %d beyond page table width %d", b, pos, max_pages);
      max_pos = std::max(max_pos, pos);
      if (pre) continue;
      int np = token_pages(pos, c->window);
      pages.push_back(np);
      total_pages += np;
    }
  }
  if (blocks * c->n_kv_heads > 0x7FFFFFFFLL) return fail(MCPU_EINVAL, "too many prefill blocks");
  out->prefill_min_q = min_q;
  out->prefill_qb = qb;
  out->n_blocks = (int)blocks;
  long long target = std::max<long long>(1, (long long)TARGET_WAVES / c->n_kv_heads);
  long long pps = std::max<long long>(PPS_MIN, (total_pages + target - 1) / target);
  // long contexts: more, shorter splits, so a token's splits are not much longer
  // than other tokens' single ones (the waves that finish last set the time)
  pps = std::min<long long>(pps, PPS_MAX);
  pps = std::max<long long>(pps, (total_pages + SPLIT_EXTRA - 1) / SPLIT_EXTRA);
  long long splits = 0;
  for (int np : pages) splits += (np + pps - 1) / pps;
  out->n_tokens = T;
  out->pps = (int)pps;
  out->n_splits = (int)splits;
  out->max_pos = max_pos;
  return MCPU_OK;
}

struct AttnBufs {
  int32_t *tok_seq, *tok_pos, *split_start, *blk_start;
  SplitDesc* split_desc;
  float *part_ml, *part_acc;
};

AttnBufs carve_attention(Carve& cv, const mcpu_layer_cfg* c, int max_tokens) {
  AttnBufs b;
  size_t S = (size_t)max_tokens + SPLIT_EXTRA;
  b.tok_seq = cv.take<int32_t>(max_tokens);
  b.tok_pos = cv.take<int32_t>(max_tokens);
  b.split_start = cv.take<int32_t>(max_tokens + 1);
  b.blk_start = cv.take<int32_t>(max_tokens + 1);  // max_tokens >= batch here
  b.split_desc = cv.take<SplitDesc>(S);
  b.part_ml = cv.take<float>(S * c->n_q_heads * 2);
  b.part_acc = cv.take<float>(S * c->n_q_heads * c->head_dim);
  return b;
}

// The plan kernel's arguments (one place for both launch sites).
AttnPlan make_plan(const mcpu_layer_cfg* c, int batch, const int32_t* seq_lens, const int32_t* cu_q,
                   const AttnPlanHost& ph, const AttnBufs& ab, int32_t* err) {
  AttnPlan pl{};
  pl.seq_lens = seq_lens; pl.cu_q = cu_q; pl.batch = batch; pl.n_tokens = ph.n_tokens;
  pl.window = c->window; pl.pps = ph.pps; pl.host_total_splits = ph.n_splits;
  pl.prefill_min_q = ph.prefill_min_q; pl.prefill_qb = ph.prefill_qb; pl.host_total_blocks = ph.n_blocks;
  pl.tok_seq = ab.tok_seq; pl.tok_pos = ab.tok_pos; pl.split_start = ab.split_start;
  pl.split_desc = ab.split_desc; pl.blk_start = ab.blk_start; pl.err = err;
  pl.norm_dtype = -1;  // no norm unless the caller adds one
  return pl;
}

struct MoeBufs {
  void* hn;
  int32_t* idx;
  float* w;
  int32_t *group_off, *pos_of, *src_tok, *chunk_cnt;
  void* act;
  float* y;
  // native MXFP4 experts: MXFP8 copies of hn and act (codes, scales)
  uint8_t *hq, *hs, *aq, *as;
};

MoeBufs carve_moe(Carve& cv, const mcpu_layer_cfg* c, int max_tokens) {
  MoeBufs m;
  size_t T = max_tokens, K = c->top_k, db = dtype_bytes(c);
  m.hn = cv.take_bytes(T * c->hidden * db);
  m.idx = cv.take<int32_t>(T * K);
  m.w = cv.take<float>(T * K);
  m.group_off = cv.take<int32_t>(c->n_experts + 1);
  m.pos_of = cv.take<int32_t>(T * K);
  m.src_tok = cv.take<int32_t>(T * K);
  m.chunk_cnt = cv.take<int32_t>((T * K + PERM_CHUNK - 1) / PERM_CHUNK * c->n_experts);
  const bool native = c->expert_fmt == MCPU_EXPERT_MXFP4_NATIVE;  // the SwiGLU output leaves in MXFP8
  m.act = native ? nullptr : cv.take_bytes(T * K * c->ffn_dim * db);
  m.y = cv.take<float>(T * K * c->hidden);
  m.hq = m.hs = m.aq = m.as = nullptr;
  if (native) {
    // in the GEMM operand layout, one row per (token, expert) assignment in
    // expert order
    m.hq = cv.take<uint8_t>(T * K * c->hidden);
    m.hs = cv.take<uint8_t>(mx_scale_bytes(T * K, c->hidden));
    m.aq = cv.take<uint8_t>(T * K * c->ffn_dim);
    m.as = cv.take<uint8_t>(mx_scale_bytes(T * K, c->ffn_dim));
  }
  return m;
}

int check_weights(const mcpu_layer_cfg* c, const mcpu_layer_weights* w, bool attn) {
  if (!w) return fail(MCPU_EINVAL, "weights is NULL");
  if (!w->g2 || !w->w_r || !w->b_r || !w->w_gu || !w->b_gu || !w->w_d || !w->b_d)
    return fail(MCPU_EINVAL, "a MoE weight pointer is NULL");
  if (c->expert_fmt != MCPU_EXPERT_DENSE && (!w->s_gu || !w->s_d))
    return fail(MCPU_EINVAL, "MXFP4 experts need the scale arrays s_gu and s_d");
  if (attn && (!w->g1 || !w->w_qkv || !w->b_qkv || !w->w_o || !w->b_o || !w->rope_cos || !w->rope_sin))
    return fail(MCPU_EINVAL, "an attention weight pointer is NULL");
  if (c->expert_fmt == MCPU_EXPERT_MXFP4_NATIVE) {
    if (!w->w_gu_packed || !w->w_d_packed)
      return fail(MCPU_EINVAL, "native MXFP4 experts need the slice-order copies w_gu_packed and w_d_packed");
    if ((uintptr_t)w->w_gu_packed % 256 || (uintptr_t)w->w_d_packed % 256)
      return fail(MCPU_EINVAL, "w_gu_packed and w_d_packed must be 256-byte aligned");
  } else if ((w->w_gu_packed || w->w_d_packed) && (c->expert_fmt != MCPU_EXPERT_DENSE || c->dtype != MCPU_BF16)) {
    return fail(MCPU_EINVAL, "packed expert weights need bf16 dense experts");
  }
  if (w->w_gu_packed && (2 * c->ffn_dim % 16 || c->hidden % 64))
    return fail(MCPU_EINVAL, "packed w_gu needs 2 * ffn_dim %% 16 == 0 and hidden %% 64 == 0");
  if (w->w_d_packed && (c->hidden % 16 || c->ffn_dim % 64))
    return fail(MCPU_EINVAL, "packed w_d needs hidden %% 16 == 0 and ffn_dim %% 64 == 0");
  if ((w->w_qkv_packed || w->w_o_packed) && c->dtype != MCPU_BF16)
    return fail(MCPU_EINVAL, "packed projection weights need a bf16 layer");
  if (w->w_qkv_packed && ((c->n_q_heads + 2 * c->n_kv_heads) * c->head_dim % 16 || c->hidden % 64))
    return fail(MCPU_EINVAL, "packed w_qkv needs (Hq + 2 Hkv) d %% 16 == 0 and hidden %% 64 == 0");
  if (w->w_o_packed && (c->hidden % 16 || c->n_q_heads * c->head_dim % 64))
    return fail(MCPU_EINVAL, "packed w_o needs hidden %% 16 == 0 and Hq d %% 64 == 0");
  if ((uintptr_t)w->w_qkv_packed % 16 || (uintptr_t)w->w_o_packed % 16)
    return fail(MCPU_EINVAL, "w_qkv_packed and w_o_packed must be 16-byte aligned");
  return MCPU_OK;
}

// MoE sub-block launches (router, permute, two grouped GEMMs, combine)
int run_moe(const mcpu_layer_cfg* c, const mcpu_layer_weights* w, int T, const float* h, float* out,
            int32_t* idx_user, float* w_user, const int32_t* force_idx, const MoeBufs& m, int32_t* err,
            hipStream_t st, float* logits_out = nullptr) {
  if (T == 0) return MCPU_OK;
  const int H = c->hidden, I = c->ffn_dim, E = c->n_experts, K = c->top_k;
  int32_t* idx = idx_user ? idx_user : m.idx;
  float* wt = w_user ? w_user : m.w;

  Router r{};
  r.h = h; r.g2 = w->g2; r.w_r = w->w_r; r.b_r = w->b_r; r.force_idx = force_idx;
  r.n_tokens = T; r.hidden = H; r.n_experts = E; r.top_k = K; r.eps = c->rms_eps;
  r.hn_out = m.hn; r.idx_out = idx; r.w_out = wt; r.logits_out = logits_out; r.err = err;
  {
    Timed tm(MCPU_KERNEL_ROUTER, st);
    HIP_TRY(launch_router(c->dtype, r, st));
  }

  Permute p{};
  p.idx = idx; p.n_tokens = T; p.top_k = K; p.n_experts = E;
  p.group_off = m.group_off; p.pos_of = m.pos_of; p.src_tok = m.src_tok; p.chunk_cnt = m.chunk_cnt; p.err = err;
  {
    Timed tm(MCPU_KERNEL_PERMUTE, st);
    HIP_TRY(launch_permute(p, st));
  }

  const int max_rows = force_idx ? T * K : T;  // a token picks each expert at most once
  // per-expert stride: elements for dense experts, bytes of E2M1 codes for MXFP4
  const int64_t fdiv = c->expert_fmt != MCPU_EXPERT_DENSE ? 2 : 1;
  const bool native = c->expert_fmt == MCPU_EXPERT_MXFP4_NATIVE;
  if (native) {  // the first product reads the normalised rows in MXFP8, in expert order
    MxQuant q{};
    q.in = m.hn; q.row_dst = m.pos_of; q.copies = K; q.rows = T; q.out_rows = (int64_t)T * K; q.cols = H;
    q.codes = m.hq; q.scales = m.hs; q.gemm_layout = 1;
    HIP_TRY(launch_mx_quant(q, st));
  }
  Gemm g1{};
  g1.w = w->w_gu; g1.w_scales = w->s_gu; g1.w_group_stride = (int64_t)2 * I * H / fdiv; g1.n = 2 * I; g1.k = H;
  g1.x = m.hn; g1.row_src = m.src_tok; g1.group_off = m.group_off; g1.n_rows = T * K; g1.n_groups = E;
  g1.epi = EPI_SWIGLU; g1.bias = w->b_gu; g1.bias_group_stride = 2 * I; g1.out = m.act;
  g1.swiglu_alpha = c->swiglu_alpha; g1.swiglu_limit = c->swiglu_limit; g1.swiglu_beta = c->swiglu_beta;
  g1.err = err; g1.max_rows_per_group = max_rows; g1.x_rows = T; g1.w_packed = w->w_gu_packed;
  if (native) {  // slice-order operands, rows already in expert order; the SwiGLU
                 // output leaves in MXFP8 for the second product
    g1.w = w->w_gu_packed; g1.w_packed = nullptr;
    g1.w_scales = (const uint8_t*)w->w_gu_packed + mx_packed_codes_bytes(E, 2 * I, H);
    g1.x = m.hq; g1.x_scales = m.hs; g1.row_src = nullptr; g1.x_rows = T * K;
    g1.epi = EPI_SWIGLU_MX; g1.out = m.aq; g1.out_scales = m.as;
  }
  {
    Timed tm(MCPU_KERNEL_EXPERT_GU, st);
    HIP_TRY(launch_gemm(c->dtype, c->expert_fmt, g1, st));
  }

  Gemm g2{};
  g2.w = w->w_d; g2.w_scales = w->s_d; g2.w_group_stride = (int64_t)H * I / fdiv; g2.n = H; g2.k = I;
  g2.x = m.act; g2.group_off = m.group_off; g2.n_rows = T * K; g2.n_groups = E;
  g2.epi = EPI_BIAS; g2.bias = w->b_d; g2.bias_group_stride = H; g2.out = m.y;
  g2.err = err; g2.max_rows_per_group = max_rows; g2.w_packed = w->w_d_packed;
  if (native) {
    g2.w = w->w_d_packed; g2.w_packed = nullptr;
    g2.w_scales = (const uint8_t*)w->w_d_packed + mx_packed_codes_bytes(E, H, I);
    g2.x = m.aq; g2.x_scales = m.as; g2.x_rows = T * K;
  }
  {
    Timed tm(MCPU_KERNEL_EXPERT_DOWN, st);
    HIP_TRY(launch_gemm(c->dtype, c->expert_fmt, g2, st));
  }

  MoeCombine mc{};
  mc.h = h; mc.y = m.y; mc.w = wt; mc.pos_of = m.pos_of; mc.n_tokens = T; mc.hidden = H; mc.top_k = K;
  mc.out = out;
  {
    Timed tm(MCPU_KERNEL_MOE_COMBINE, st);
    HIP_TRY(launch_moe_combine(mc, st));
  }
  return MCPU_OK;
}

int run_attention(const mcpu_layer_cfg* c, const float* sinks, mcpu_kv_pool* pool, int batch,
                  const int32_t* page_table, int max_pages, const int32_t* seq_lens, const int32_t* cu_q,
                  const AttnPlanHost& ph, const void* q, void* o, const AttnBufs& ab, int32_t* err,
                  hipStream_t st, bool plan_done);

}  // namespace

struct mcpu_kv_pool {
  mcpu_layer_cfg cfg;
  int32_t n_pages;
  void* k;
  void* v;
  std::set<int32_t> free_ids;
  std::vector<uint8_t> in_use;
};

namespace {
int run_attention(const mcpu_layer_cfg* c, const float* sinks, mcpu_kv_pool* pool, int batch,
                  const int32_t* page_table, int max_pages, const int32_t* seq_lens, const int32_t* cu_q,
                  const AttnPlanHost& ph, const void* q, void* o, const AttnBufs& ab, int32_t* err,
                  hipStream_t st, bool plan_done) {
  if (!plan_done) {
    Timed tm(MCPU_KERNEL_ATTN_PLAN, st);
    HIP_TRY(launch_attn_plan(make_plan(c, batch, seq_lens, cu_q, ph, ab, err), st));
  }
  AttnSplit sp{};
  sp.q = q; sp.k_pool = pool->k; sp.v_pool = pool->v; sp.page_table = page_table;
  sp.max_pages = max_pages; sp.n_pages = pool->n_pages;
  sp.tok_seq = ab.tok_seq; sp.tok_pos = ab.tok_pos; sp.split_start = ab.split_start; sp.split_desc = ab.split_desc;
  sp.batch = batch; sp.n_tokens = ph.n_tokens; sp.n_splits = ph.n_splits; sp.hq = c->n_q_heads; sp.hkv = c->n_kv_heads;
  sp.window = c->window; sp.pps = ph.pps;
  sp.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)c->head_dim));
  sp.part_ml = ab.part_ml; sp.part_acc = ab.part_acc; sp.err = err;
  // short windows: one split per token, finished in the split pass itself
  const bool one_pass = c->window > 0 && c->window <= WINDOW_MAX_KEYS && ph.pps >= WINDOW_MAX_PAGES;
  if (one_pass) { sp.o = o; sp.sinks = sinks; }
  {
    Timed tm(MCPU_KERNEL_ATTN_SPLIT, st);
    HIP_TRY(launch_attn_split(c->dtype, c->head_dim, sp, st));
  }
  if (!one_pass) {
    AttnCombine cb{};
    cb.part_ml = ab.part_ml; cb.part_acc = ab.part_acc; cb.split_start = ab.split_start; cb.sinks = sinks;
    cb.n_tokens = ph.n_tokens; cb.n_splits = ph.n_splits; cb.hq = c->n_q_heads; cb.o = o;
    Timed tm(MCPU_KERNEL_ATTN_COMBINE, st);
    HIP_TRY(launch_attn_combine(c->dtype, c->head_dim, cb, st));
  }
  if (ph.n_blocks > 0) {
    AttnPrefill pf{};
    pf.q = q; pf.k_pool = pool->k; pf.v_pool = pool->v; pf.page_table = page_table;
    pf.max_pages = max_pages; pf.n_pages = pool->n_pages;
    pf.seq_lens = seq_lens; pf.cu_q = cu_q; pf.blk_start = ab.blk_start;
    pf.batch = batch; pf.n_tokens = ph.n_tokens; pf.n_blocks = ph.n_blocks; pf.hq = c->n_q_heads; pf.hkv = c->n_kv_heads;
    pf.window = c->window; pf.scale_log2 = sp.scale_log2; pf.sinks = sinks; pf.o = o; pf.err = err;
    Timed tm(MCPU_KERNEL_ATTN_PREFILL, st);
    HIP_TRY(launch_attn_prefill(c->dtype, c->head_dim, c->n_q_heads / c->n_kv_heads, pf, st));
  }
  return MCPU_OK;
}

bool same_shape(const mcpu_layer_cfg* a, const mcpu_layer_cfg* b) {
  return a->n_kv_heads == b->n_kv_heads && a->head_dim == b->head_dim && a->dtype == b->dtype;
}
}  // namespace

extern "C" {

const char* mcpu_last_error(void) { return g_err.c_str(); }

int kv_pool_create(const mcpu_layer_cfg* cfg, int32_t n_pages, void* k_pool, void* v_pool, mcpu_kv_pool** out) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!out || !k_pool || !v_pool) return fail(MCPU_EINVAL, "NULL pointer");
  if (n_pages <= 0) return fail(MCPU_EINVAL, "n_pages %d", n_pages);
  mcpu_kv_pool* p = new (std::nothrow) mcpu_kv_pool();
  if (!p) return fail(MCPU_ENOMEM, "host allocation failed");
  p->cfg = *cfg;
  p->n_pages = n_pages;
  p->k = k_pool;
  p->v = v_pool;
  p->in_use.assign(n_pages, 0);
  for (int32_t i = 0; i < n_pages; ++i) p->free_ids.insert(p->free_ids.end(), i);
  *out = p;
  return MCPU_OK;
}

int kv_pool_destroy(mcpu_kv_pool* pool) {
  delete pool;
  return MCPU_OK;
}

int32_t kv_pool_free_pages(const mcpu_kv_pool* pool) { return pool ? (int32_t)pool->free_ids.size() : 0; }

int kv_pages_alloc(mcpu_kv_pool* pool, int32_t n, int32_t* out_ids) {
  if (!pool || (n > 0 && !out_ids) || n < 0) return fail(MCPU_EINVAL, "kv_pages_alloc: bad arguments");
  if ((size_t)n > pool->free_ids.size())
    return fail(MCPU_ENOMEM, "kv_pages_alloc: %d pages requested, %zu free", n, pool->free_ids.size());
  auto it = pool->free_ids.begin();
  for (int32_t i = 0; i < n; ++i) {
    out_ids[i] = *it;
    pool->in_use[*it] = 1;
    it = pool->free_ids.erase(it);
  }
  return MCPU_OK;
}

int kv_pages_free(mcpu_kv_pool* pool, int32_t n, const int32_t* ids) {
  if (!pool || (n > 0 && !ids) || n < 0) return fail(MCPU_EINVAL, "kv_pages_free: bad arguments");
  std::vector<uint8_t> seen;
  for (int32_t i = 0; i < n; ++i) {
    int32_t id = ids[i];
    if (id < 0 || id >= pool->n_pages) return fail(MCPU_EINVAL, "kv_pages_free: id %d out of range", id);
    if (!pool->in_use[id]) return fail(MCPU_EINVAL, "kv_pages_free: page %d is not allocated", id);
    if (seen.empty()) seen.assign(pool->n_pages, 0);
    if (seen[id]) return fail(MCPU_EINVAL, "kv_pages_free: page %d repeated", id);
    seen[id] = 1;
  }
  for (int32_t i = 0; i < n; ++i) {
    pool->in_use[ids[i]] = 0;
    pool->free_ids.insert(ids[i]);
  }
  return MCPU_OK;
}

int kv_pages_append(mcpu_kv_pool* pool, int32_t batch, const int32_t* page_table, int32_t max_pages,
                    const int32_t* seq_lens, const int32_t* cu_q, int32_t n_tokens, const void* k_new,
                    const void* v_new, void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (!pool) return fail(MCPU_EINVAL, "pool is NULL");
  if (batch < 0 || n_tokens < 0 || max_pages <= 0) return fail(MCPU_EINVAL, "bad sizes");
  if (!cu_q && n_tokens != batch) return fail(MCPU_EINVAL, "n_tokens must equal batch when cu_q is NULL");
  if (n_tokens == 0) return MCPU_OK;
  if (!page_table || !seq_lens || !k_new || !v_new || !workspace) return fail(MCPU_EINVAL, "NULL pointer");
  if (ws_bytes < 256) return fail(MCPU_ENOMEM, "workspace smaller than 256 bytes");
  KvAppend a{};
  a.k_new = k_new; a.v_new = v_new; a.k_pool = pool->k; a.v_pool = pool->v;
  a.page_table = page_table; a.max_pages = max_pages; a.n_pages = pool->n_pages;
  a.seq_lens = seq_lens; a.cu_q = cu_q; a.batch = batch; a.n_tokens = n_tokens;
  a.hkv = pool->cfg.n_kv_heads; a.err = err_word(workspace);
  {
    Timed tm(MCPU_KERNEL_KV_APPEND, stream);
    HIP_TRY(launch_kv_append(pool->cfg.dtype, pool->cfg.head_dim, a, stream));
  }
  return MCPU_OK;
}

size_t paged_attention_workspace_size(const mcpu_layer_cfg* cfg, int32_t max_batch, int32_t max_tokens) {
  if (check_cfg(cfg)) return 0;
  Carve cv(nullptr);
  carve_attention(cv, cfg, std::max(max_tokens, max_batch));
  return (cv.off + 255) & ~size_t(255);
}

int paged_attention(const mcpu_layer_cfg* cfg, const float* sinks, mcpu_kv_pool* pool, int32_t batch,
                    const int32_t* page_table, int32_t max_pages, const int32_t* seq_lens, const int32_t* cu_q,
                    const int32_t* host_seq_lens, const int32_t* host_cu_q, const void* q, void* o,
                    void* workspace, size_t ws_bytes, hipStream_t stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!pool || !same_shape(cfg, &pool->cfg)) return fail(MCPU_EINVAL, "pool missing or of another shape");
  if (batch <= 0 || max_pages <= 0) return fail(MCPU_EINVAL, "batch %d, max_pages %d", batch, max_pages);
  if (!page_table || !seq_lens || !q || !o || !workspace) return fail(MCPU_EINVAL, "NULL pointer");
  if ((cu_q == nullptr) != (host_cu_q == nullptr)) return fail(MCPU_EINVAL, "cu_q and host_cu_q must both be given or both NULL");
  AttnPlanHost ph;
  if ((rc = plan_attention(cfg, batch, max_pages, host_seq_lens, host_cu_q, &ph))) return rc;
  if (ph.n_tokens == 0) return MCPU_OK;
  size_t need = paged_attention_workspace_size(cfg, batch, ph.n_tokens);
  if (ws_bytes < need) return fail(MCPU_ENOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  Carve cv(workspace);
  AttnBufs ab = carve_attention(cv, cfg, std::max(ph.n_tokens, batch));
  return run_attention(cfg, sinks, pool, batch, page_table, max_pages, seq_lens, cu_q, ph, q, o, ab,
                       err_word(workspace), stream, false);
}

size_t mcpu_packed_weights_bytes(int32_t n_groups, int32_t rows, int32_t cols) {
  if (n_groups <= 0 || rows <= 0 || cols <= 0 || rows % 16 || cols % 64) return 0;
  return (size_t)n_groups * (rows / 16) * ((cols + 127) / 128) * 4096;
}

int mcpu_pack_weights(int32_t dtype, const void* src, void* dst, int32_t n_groups, int32_t rows, int32_t cols,
                      hipStream_t stream) {
  if (dtype != MCPU_BF16) return fail(MCPU_EUNSUPPORTED, "streaming-order weights are bf16 only (dtype %d)", dtype);
  const size_t bytes = mcpu_packed_weights_bytes(n_groups, rows, cols);
  if (bytes == 0) return fail(MCPU_EINVAL, "groups %d, rows %d (multiple of 16), cols %d (multiple of 64)", n_groups, rows, cols);
  if (!src || !dst) return fail(MCPU_EINVAL, "NULL pointer");
  if ((uintptr_t)src % 16 || (uintptr_t)dst % 16) return fail(MCPU_EINVAL, "src and dst must be 16-byte aligned");
  const uintptr_t s0 = (uintptr_t)src, s1 = s0 + (size_t)n_groups * rows * cols * 2;
  const uintptr_t d0 = (uintptr_t)dst, d1 = d0 + bytes;
  if (s0 < d1 && d0 < s1) return fail(MCPU_EINVAL, "src and dst overlap");
  HIP_TRY(launch_pack_weights(src, dst, n_groups, rows, cols, stream));
  return MCPU_OK;
}

size_t mcpu_packed_mxfp4_bytes(int32_t n_groups, int32_t rows, int32_t cols) {
  if (n_groups <= 0 || rows <= 0 || rows % 16 || cols <= 0 || cols % 64) return 0;
  return mx_packed_bytes(n_groups, rows, cols);
}

int mcpu_pack_mxfp4(const uint8_t* codes, const uint8_t* scales, void* dst, int32_t n_groups, int32_t rows,
                    int32_t cols, hipStream_t stream) {
  const size_t bytes = mcpu_packed_mxfp4_bytes(n_groups, rows, cols);
  if (bytes == 0) return fail(MCPU_EINVAL, "groups %d, rows %d (multiple of 16), cols %d (multiple of 64)", n_groups, rows, cols);
  if (!codes || !scales || !dst) return fail(MCPU_EINVAL, "NULL pointer");
  if ((uintptr_t)codes % 16 || (uintptr_t)dst % 256) return fail(MCPU_EINVAL, "codes must be 16-byte and dst 256-byte aligned");
  const uintptr_t d0 = (uintptr_t)dst, d1 = d0 + bytes;
  const uintptr_t c0 = (uintptr_t)codes, c1 = c0 + (size_t)n_groups * rows * (cols / 2);
  const uintptr_t s0 = (uintptr_t)scales, s1 = s0 + (size_t)n_groups * rows * (cols / 32);
  if ((c0 < d1 && d0 < c1) || (s0 < d1 && d0 < s1)) return fail(MCPU_EINVAL, "source and dst overlap");
  MxPack p{};
  p.codes = codes; p.scales = scales; p.dst = (uint8_t*)dst; p.groups = n_groups; p.rows = rows; p.cols = cols;
  HIP_TRY(launch_mx_pack(p, stream));
  return MCPU_OK;
}

size_t moe_forward_workspace_size(const mcpu_layer_cfg* cfg, int32_t max_tokens) {
  if (check_cfg(cfg)) return 0;
  Carve cv(nullptr);
  carve_moe(cv, cfg, max_tokens);
  return (cv.off + 255) & ~size_t(255);
}

int moe_forward(const mcpu_layer_cfg* cfg, const mcpu_layer_weights* w, int32_t n_tokens, const float* h,
                float* out, int32_t* topk_idx, float* topk_w, const int32_t* force_idx, void* workspace,
                size_t ws_bytes, hipStream_t stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if ((rc = check_weights(cfg, w, false))) return rc;
  if (n_tokens < 0) return fail(MCPU_EINVAL, "n_tokens %d", n_tokens);
  if (n_tokens == 0) return MCPU_OK;
  if (!h || !out || !workspace) return fail(MCPU_EINVAL, "NULL pointer");
  size_t need = moe_forward_workspace_size(cfg, n_tokens);
  if (ws_bytes < need) return fail(MCPU_ENOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  Carve cv(workspace);
  MoeBufs m = carve_moe(cv, cfg, n_tokens);
  return run_moe(cfg, w, n_tokens, h, out, topk_idx, topk_w, force_idx, m, err_word(workspace), stream);
}

// fp32 partial tiles of the dense projections when they split the reduction
// over workgroups (bf16 layers, a few rows): the most any row count up to
// max_rows needs, so the carve does not depend on the call's row count
size_t layer_split_floats(const mcpu_layer_cfg* c, int max_rows) {
  if (c->dtype != MCPU_BF16) return 0;
  const int H = c->hidden, D = c->head_dim;
  size_t m = 0;
  for (int r = 1; r <= std::min(max_rows, SPLIT_MAX_ROWS); ++r)
    m = std::max({m, slab_split_part_floats((c->n_q_heads + 2 * c->n_kv_heads) * D, H, r),
                  slab_split_part_floats(H, c->n_q_heads * D, r)});
  return m;
}

size_t decode_layer_workspace_size(const mcpu_layer_cfg* cfg, int32_t max_batch, int32_t max_tokens) {
  if (check_cfg(cfg)) return 0;
  int T = std::max(max_tokens, max_batch);
  Carve cv(nullptr);
  carve_attention(cv, cfg, T);
  size_t db = dtype_bytes(cfg);
  cv.take_bytes((size_t)T * cfg->hidden * db);                        // xn
  cv.take_bytes((size_t)T * cfg->n_q_heads * cfg->head_dim * db);     // q
  cv.take_bytes((size_t)T * cfg->n_q_heads * cfg->head_dim * db);     // o
  cv.take<float>((size_t)T * cfg->hidden);                            // h1
  carve_moe(cv, cfg, T);
  cv.take<float>(layer_split_floats(cfg, T));                         // split partial tiles
  cv.take<int32_t>(SPLIT_MAX_TILES);                                  // their arrival counters
  return (cv.off + 255) & ~size_t(255);
}

int decode_layer(const mcpu_layer_cfg* cfg, const mcpu_layer_weights* w, mcpu_kv_pool* pool, int32_t batch,
                 const int32_t* page_table, int32_t max_pages, const int32_t* seq_lens, const int32_t* cu_q,
                 const int32_t* host_seq_lens, const int32_t* host_cu_q, const float* x_in, float* x_out,
                 int32_t* topk_idx, float* topk_w, const mcpu_taps* taps, void* workspace, size_t ws_bytes,
                 hipStream_t stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if ((rc = check_weights(cfg, w, true))) return rc;
  if (!pool || !same_shape(cfg, &pool->cfg)) return fail(MCPU_EINVAL, "pool missing or of another shape");
  if (batch <= 0 || max_pages <= 0) return fail(MCPU_EINVAL, "batch %d, max_pages %d", batch, max_pages);
  if (!page_table || !seq_lens || !x_in || !x_out || !workspace) return fail(MCPU_EINVAL, "NULL pointer");
  if (x_in == x_out) return fail(MCPU_EINVAL, "x_in and x_out must not alias");
  if ((cu_q == nullptr) != (host_cu_q == nullptr)) return fail(MCPU_EINVAL, "cu_q and host_cu_q must both be given or both NULL");
  AttnPlanHost ph;
  if ((rc = plan_attention(cfg, batch, max_pages, host_seq_lens, host_cu_q, &ph))) return rc;
  const int T = ph.n_tokens;
  if (T == 0) return MCPU_OK;
  if (ph.max_pos >= w->rope_max_pos)
    return fail(MCPU_EINVAL, "position %d beyond the RoPE table (%d rows)", ph.max_pos, w->rope_max_pos);
  size_t need = decode_layer_workspace_size(cfg, batch, T);
  if (ws_bytes < need) return fail(MCPU_ENOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);

  const int H = cfg->hidden, D = cfg->head_dim, Hq = cfg->n_q_heads, Hkv = cfg->n_kv_heads;
  const size_t db = dtype_bytes(cfg);
  Carve cv(workspace);
  const int Tc = std::max(T, batch);
  AttnBufs ab = carve_attention(cv, cfg, Tc);
  void* xn = cv.take_bytes((size_t)Tc * H * db);
  void* q = cv.take_bytes((size_t)Tc * Hq * D * db);
  void* o = cv.take_bytes((size_t)Tc * Hq * D * db);
  float* h1 = cv.take<float>((size_t)Tc * H);
  MoeBufs mb = carve_moe(cv, cfg, Tc);
  const size_t split_floats = layer_split_floats(cfg, Tc);
  float* part = cv.take<float>(split_floats);
  int32_t* part_cnt = cv.take<int32_t>(SPLIT_MAX_TILES);
  int32_t* err = err_word(workspace);

  // the plan and RMSNorm_1 share one launch (the norm does not depend on it)
  RmsNorm rn{};
  rn.x = x_in; rn.g = w->g1; rn.n_tokens = T; rn.hidden = H; rn.eps = cfg->rms_eps; rn.out = xn;
  {
    Timed tm(MCPU_KERNEL_ATTN_PLAN, stream);
    AttnPlan pl = make_plan(cfg, batch, seq_lens, cu_q, ph, ab, err);
    if (split_floats) {  // the split GEMMs' counters start at zero
      pl.zero = part_cnt;
      pl.n_zero = SPLIT_MAX_TILES;
    }
    pl.norm = rn;
    pl.norm_dtype = cfg->dtype;
    HIP_TRY(launch_attn_plan(pl, stream));
  }

  Gemm gq{};
  gq.w = w->w_qkv; gq.n = (Hq + 2 * Hkv) * D; gq.k = H; gq.x = xn; gq.n_rows = T; gq.n_groups = 1;
  gq.epi = EPI_QKV; gq.bias = w->b_qkv; gq.hq = Hq; gq.hkv = Hkv; gq.head_dim = D; gq.q_out = q;
  gq.k_pool = pool->k; gq.v_pool = pool->v; gq.page_table = page_table; gq.max_pages = max_pages;
  gq.n_pages = pool->n_pages; gq.tok_seq = ab.tok_seq; gq.tok_pos = ab.tok_pos; gq.rope_cos = w->rope_cos;
  gq.rope_sin = w->rope_sin; gq.rope_max_pos = w->rope_max_pos; gq.err = err; gq.max_rows_per_group = T;
  gq.w_packed = cfg->dtype == MCPU_BF16 ? w->w_qkv_packed : nullptr;
  if (split_floats) { gq.part = part; gq.part_cnt = part_cnt; }
  {
    Timed tm(MCPU_KERNEL_QKV, stream);
    HIP_TRY(launch_gemm(cfg->dtype, MCPU_EXPERT_DENSE, gq, stream));
  }

  if ((rc = run_attention(cfg, w->sinks, pool, batch, page_table, max_pages, seq_lens, cu_q, ph, q, o, ab, err,
                          stream, true)))
    return rc;

  Gemm go{};
  go.w = w->w_o; go.n = H; go.k = Hq * D; go.x = o; go.n_rows = T; go.n_groups = 1; go.epi = EPI_RESIDUAL;
  go.bias = w->b_o; go.residual = x_in; go.out = h1; go.err = err; go.max_rows_per_group = T;
  go.w_packed = cfg->dtype == MCPU_BF16 ? w->w_o_packed : nullptr;
  if (split_floats) { go.part = part; go.part_cnt = part_cnt; }
  {
    Timed tm(MCPU_KERNEL_OPROJ, stream);
    HIP_TRY(launch_gemm(cfg->dtype, MCPU_EXPERT_DENSE, go, stream));
  }

  if ((rc = run_moe(cfg, w, T, h1, x_out, topk_idx, topk_w, nullptr, mb, err, stream,
                    taps ? taps->logits : nullptr)))
    return rc;

  if (taps) {
    if (taps->q) HIP_TRY(hipMemcpyAsync(taps->q, q, (size_t)T * Hq * D * db, hipMemcpyDeviceToDevice, stream));
    if (taps->o) HIP_TRY(hipMemcpyAsync(taps->o, o, (size_t)T * Hq * D * db, hipMemcpyDeviceToDevice, stream));
    if (taps->h1) HIP_TRY(hipMemcpyAsync(taps->h1, h1, (size_t)T * H * 4, hipMemcpyDeviceToDevice, stream));
  }
  return MCPU_OK;
}

size_t lm_head_workspace_size(int32_t hidden, int32_t vocab, int32_t max_tokens) {
  if (hidden <= 0 || vocab <= 0 || max_tokens < 0) return 0;
  Carve cv(nullptr);
  cv.take<int32_t>(2);                                                            // row range
  cv.take_bytes((size_t)std::max(max_tokens, 1) * hidden * 2);                     // normalised rows
  cv.take<LogitSlot>((size_t)std::max(max_tokens, 1) * ((vocab + LOGIT_SLOT - 1) / LOGIT_SLOT));
  return (cv.off + 255) & ~size_t(255);
}

int lm_head_sample(const mcpu_lm_head* lm, int32_t n_tokens, const float* x, const int32_t* x_rows,
                   float temperature, uint64_t seed,
                   const int32_t* seq_ids, const int32_t* positions, const int32_t* targets, int32_t* tokens_out,
                   float* logprob_out, float* target_logprob_out, float* lse_out, void* workspace,
                   size_t ws_bytes, hipStream_t stream) {
  if (!lm) return fail(MCPU_EINVAL, "lm is NULL");
  const int H = lm->hidden, V = lm->vocab;
  if (H <= 0 || H % 64 || H > 8192) return fail(MCPU_EINVAL, "hidden %d must be a multiple of 64 in (0, 8192]", H);
  if (V <= 0 || V % 16) return fail(MCPU_EINVAL, "vocab %d must be a positive multiple of 16", V);
  if ((int64_t)V * H * 2 >= (1LL << 31)) return fail(MCPU_EUNSUPPORTED, "vocab x hidden too large for one matrix");
  if (!(lm->rms_eps >= 0.f)) return fail(MCPU_EINVAL, "rms_eps");
  if (n_tokens < 0) return fail(MCPU_EINVAL, "n_tokens %d", n_tokens);
  if (n_tokens == 0) return MCPU_OK;
  if (!lm->g_final || !lm->w_lm || !x || !workspace) return fail(MCPU_EINVAL, "NULL pointer");
  const bool greedy = !(temperature > 0.f);
  // the draws are needed only when a sampled token (or its log-probability) is asked for
  const bool draws = !greedy && (tokens_out || logprob_out);
  if (draws && (!seq_ids || !positions)) return fail(MCPU_EINVAL, "sampling needs seq_ids and positions");
  if (!greedy && !(temperature < 1e30f)) return fail(MCPU_EINVAL, "temperature %g", (double)temperature);
  if (targets && !target_logprob_out) return fail(MCPU_EINVAL, "targets given without target_logprob_out");
  const size_t need = lm_head_workspace_size(H, V, n_tokens);
  if (ws_bytes < need) return fail(MCPU_ENOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  Carve cv(workspace);
  int32_t* goff = cv.take<int32_t>(2);
  void* xn = cv.take_bytes((size_t)n_tokens * H * 2);
  const int n_slots = (V + LOGIT_SLOT - 1) / LOGIT_SLOT;
  LogitSlot* slots = cv.take<LogitSlot>((size_t)n_tokens * n_slots);

  FinalNorm fn{};
  fn.x = x; fn.rows = x_rows; fn.g = lm->g_final; fn.n_tokens = n_tokens; fn.hidden = H; fn.eps = lm->rms_eps; fn.out = xn;
  fn.group_off = goff;
  HIP_TRY(launch_final_norm(fn, stream));

  Gemm g{};
  g.w = lm->w_lm; g.w_packed = lm->w_lm_packed; g.n = V; g.k = H; g.x = xn; g.group_off = goff;
  g.n_rows = n_tokens; g.n_groups = 1; g.epi = EPI_LOGITS; g.out = slots; g.err = err_word(workspace);
  g.max_rows_per_group = n_tokens; g.x_rows = n_tokens;
  g.inv_temp = greedy ? 1.f : 1.f / temperature; g.greedy = draws ? 0 : 1; g.seed = seed;
  g.row_seq = seq_ids; g.row_pos = positions; g.target = targets;
  {
    Timed tm(MCPU_KERNEL_LM_HEAD, stream);
    HIP_TRY(launch_gemm(MCPU_BF16, MCPU_EXPERT_DENSE, g, stream));
  }
  LmReduce r{};
  r.slots = slots; r.n_rows = n_tokens; r.n_slots = n_slots; r.tokens = tokens_out; r.logprob = logprob_out;
  r.lse = lse_out; r.target_logprob = targets ? target_logprob_out : nullptr;
  HIP_TRY(launch_lm_reduce(r, stream));
  return MCPU_OK;
}

int mcpu_mxfp8_quantize(const void* in, int64_t rows, int32_t cols, uint8_t* codes, uint8_t* scales,
                        hipStream_t stream) {
  if (rows < 0 || cols <= 0 || cols % 32) return fail(MCPU_EINVAL, "rows %lld, cols %d (a multiple of 32)", (long long)rows, cols);
  if (rows == 0) return MCPU_OK;
  if (!in || !codes || !scales) return fail(MCPU_EINVAL, "NULL pointer");
  if ((uintptr_t)in % 16 || (uintptr_t)codes % 16) return fail(MCPU_EINVAL, "in and codes must be 16-byte aligned");
  MxQuant q{};
  q.in = in; q.copies = 1; q.rows = q.out_rows = rows; q.cols = cols; q.codes = codes; q.scales = scales;
  HIP_TRY(launch_mx_quant(q, stream));
  return MCPU_OK;
}

int embed_tokens(const void* table, int32_t vocab, int32_t hidden, int32_t n_tokens, const int32_t* tokens,
                 float* x_out, void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (vocab <= 0 || hidden <= 0 || hidden % 8 || n_tokens < 0) return fail(MCPU_EINVAL, "bad sizes");
  if (n_tokens == 0) return MCPU_OK;
  if (!table || !tokens || !x_out || !workspace) return fail(MCPU_EINVAL, "NULL pointer");
  if ((uintptr_t)table % 16 || (uintptr_t)x_out % 16) return fail(MCPU_EINVAL, "table and x_out must be 16-byte aligned");
  if (ws_bytes < 256) return fail(MCPU_ENOMEM, "workspace smaller than 256 bytes");
  EmbedArgs a{};
  a.table = table; a.tokens = tokens; a.vocab = vocab; a.hidden = hidden; a.n_tokens = n_tokens; a.x = x_out;
  a.err = err_word(workspace);
  HIP_TRY(launch_embed(a, stream));
  return MCPU_OK;
}

}  // extern "C"

// ---- decode_layer without allocation ------------------------------------
// The workspace of decode_layer_noalloc is this file-scope device array. In
// host code its name is only a stand-in: the device address of each GPU's
// copy comes from hipGetSymbolAddress, looked up once per device and kept.
namespace {
constexpr size_t SCRATCH_BYTES = size_t(128) << 20;
static __device__ __align__(256) unsigned char scratch[SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

int scratch_for_current_device(void** out) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= MAX_DEVICES) return fail(MCPU_EUNSUPPORTED, "device %d beyond the scratch table", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    HIP_TRY(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
    if (!ptr) return fail(MCPU_EHIP, "hipGetSymbolAddress returned no address for the scratch array");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return MCPU_OK;
}

// Moves the call's device error word to the caller's output (or drops it)
// and clears it, so every call starts from zero without a memset.
__global__ void take_errors_kernel(int32_t* word, int32_t* out) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    if (out) *out = *word;
    *word = 0;
  }
}
}  // namespace

extern "C" {

int decode_layer_noalloc(const mcpu_layer_cfg* cfg, const mcpu_layer_weights* w, mcpu_kv_pool* pool,
                         int32_t batch, const int32_t* page_table, int32_t max_pages, const int32_t* seq_lens,
                         const int32_t* cu_q, const int32_t* host_seq_lens, const int32_t* host_cu_q,
                         const float* x_in, float* x_out, int32_t* topk_idx, float* topk_w, const mcpu_taps* taps,
                         int32_t* device_errors, hipStream_t stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (batch <= 0) return fail(MCPU_EINVAL, "batch %d", batch);
  if (!host_seq_lens) return fail(MCPU_EINVAL, "host_seq_lens is NULL");
  if (host_cu_q && host_cu_q[batch] < 0) return fail(MCPU_EINVAL, "host_cu_q[batch] < 0");
  const int T = host_cu_q ? host_cu_q[batch] : batch;
  const size_t need = decode_layer_workspace_size(cfg, batch, T);
  if (need == 0 || need > SCRATCH_BYTES)
    return fail(MCPU_ENOMEM, "decode_layer_noalloc: this step needs %zu bytes of scratch; the static scratch "
                "holds %zu (use decode_layer with a workspace)", need, SCRATCH_BYTES);
  void* ws = nullptr;
  if ((rc = scratch_for_current_device(&ws))) return rc;
  if ((rc = decode_layer(cfg, w, pool, batch, page_table, max_pages, seq_lens, cu_q, host_seq_lens, host_cu_q, x_in,
                         x_out, topk_idx, topk_w, taps, ws, SCRATCH_BYTES, stream)))
    return rc;
  hipLaunchKernelGGL(take_errors_kernel, dim3(1), dim3(64), 0, stream, err_word(ws), device_errors);
  HIP_TRY(hipGetLastError());
  return MCPU_OK;
}

int mcpu_timing_start(int kernel, int n) {
  if (kernel < 0 || kernel >= MCPU_KERNEL_COUNT || n < 0) return fail(MCPU_EINVAL, "timing kernel %d, n %d", kernel, n);
  KernelTimer& k = g_timers[kernel];
  while ((int)k.start.size() < n) {
    // timing only: no system-scope fence when an event is recorded (a fence
    // writes back and invalidates the caches, which would put about 6 us of
    // stall next to every timed launch)
    hipEvent_t a, b;
    HIP_TRY(hipEventCreateWithFlags(&a, hipEventDisableSystemFence));
    HIP_TRY(hipEventCreateWithFlags(&b, hipEventDisableSystemFence));
    k.start.push_back(a);
    k.stop.push_back(b);
  }
  k.armed = n;
  k.next = 0;
  return MCPU_OK;
}

int mcpu_timing_read(int kernel, float* ms, int n, int* n_recorded) {
  if (kernel < 0 || kernel >= MCPU_KERNEL_COUNT || n < 0 || (n > 0 && !ms))
    return fail(MCPU_EINVAL, "timing kernel %d", kernel);
  KernelTimer& k = g_timers[kernel];
  int m = std::min(n, k.next);
  for (int i = 0; i < m; ++i) {
    HIP_TRY(hipEventSynchronize(k.stop[i]));
    HIP_TRY(hipEventElapsedTime(&ms[i], k.start[i], k.stop[i]));
  }
  if (n_recorded) *n_recorded = m;
  return MCPU_OK;
}

int mcpu_check_device_errors(void* workspace, hipStream_t stream, int32_t* bits) {
  if (!workspace) return fail(MCPU_EINVAL, "workspace is NULL");
  int32_t v = 0;
  HIP_TRY(hipStreamSynchronize(stream));
  HIP_TRY(hipMemcpy(&v, workspace, sizeof v, hipMemcpyDeviceToHost));
  if (bits) *bits = v;
  if (v) {
    HIP_TRY(hipMemset(workspace, 0, sizeof v));
    return fail(MCPU_EDEVICE, "device error bits 0x%x", v);
  }
  return MCPU_OK;
}

}  // extern "C"
