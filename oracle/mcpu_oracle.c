/*
 * mcpu_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow CPU reference of one decode step of a gpt-oss-20b-shaped
 * decoder layer, the generation work that the paper's Run stage is bound by
 * (Sec. 3.2: the run stage is GPU bound and dominated by generation; the
 * policy is gpt-oss-20b, Sec. 4 and its training details appendix). Each
 * turn's tool observation joins the context (Sec. 1, Sec. 3.2), which is why
 * the step also takes multi-token chunks ("chunked prefill").
 *
 * The paper fixes none of the layer's arithmetic; the definitions below are
 * the public gpt-oss conventions, each stated where it is used. Everything is
 * computed in float64 with plain loops, in the order the definition gives, with
 * no blocking, splitting or reordering. Values are rounded only where the
 * layer stores them, to the layer's dtype (bfloat16 for bf16 layers, binary32
 * for fp32 layers): the normalised input of the QKV product, the rotated
 * queries, the new keys and values written to the paged cache, the attention
 * output, the normalised rows the experts read and the SwiGLU activations.
 * Everything between two such points (the products' sums, the softmax, the
 * residual stream, the router logits) stays in float64. A second mode
 * (kv_only) rounds the cache entries only and keeps every activation in
 * float64; it measures how much of the GPU's distance from the reference
 * comes from the activations it stores.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg use
 * this file. It shares no code, header or table with the GPU library.
 *
 * Paged cache format (the library's documented page format, restated here):
 * a pool holds n_pages pages; page p, KV head g holds 16 tokens x d dims at
 * base ((p * Hkv + g) * 16 * d). Within it, K element (slot s, dim i) sits at
 *   ((i / 8) * 16 + s) * 8 + i % 8
 * and V element (slot s, dim i) at
 *   (((i / 16) * 4 + s / 4) * 16 + i % 16) * 4 + s % 4.
 *
 * Parity pins: every function is checked by tests/test_oracle_pins.py against
 * brute force, closed forms, library routines and invariants.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_PAGE 16

typedef struct {
  int32_t hidden, n_q_heads, n_kv_heads, head_dim, n_experts, top_k, ffn_dim;
  int32_t page_size; /* must be 16 */
  int32_t window;    /* 0: full attention; else keys p-window+1 .. p */
  int32_t kv_bf16;   /* 1: the layer (cache and stored activations) is bfloat16 */
  int32_t kv_only;   /* 1: round only the cache entries; keep every activation unrounded */
  int32_t act_mx;    /* 1: the expert products read MXFP8 (E4M3) activations, see orc_mxfp8_quant */
  double rms_eps, swiglu_alpha, swiglu_limit, swiglu_beta;
} orc_cfg;

/* Layer parameters, all as fp32 arrays (bfloat16 values are exact in fp32). */
typedef struct {
  const float *g1, *w_qkv, *b_qkv, *w_o, *b_o, *g2, *w_r, *b_r;
  const float *w_gu, *b_gu, *w_d, *b_d, *sinks, *rope_cos, *rope_sin;
  int32_t rope_max_pos;
} orc_weights;

enum { ORC_OK = 0, ORC_EINVAL = -1 };

/* ------------------------------------------------------------------------ */
/* bfloat16: the upper 16 bits of binary32, rounded to nearest, ties to even */
/* ------------------------------------------------------------------------ */

double orc_round_bf16(double v) {
  if (v == 0.0 || !isfinite(v)) return v;
  int e;
  frexp(v, &e);              /* |v| = m * 2^e, 0.5 <= m < 1 */
  int q = e - 8;             /* 8 significant bits: ulp = 2^(e-8) */
  if (q < -133) q = -133;    /* binary32 exponent range: subnormal spacing 2^-133 */
  double r = ldexp(nearbyint(ldexp(v, -q)), q); /* default mode: nearest, ties even */
  if (fabs(r) > 3.3895313892515355e38) r = copysign(INFINITY, v);
  return r;
}

void orc_round_bf16_array(int64_t n, const double* in, double* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_round_bf16(in[i]);
}

/* a value as the layer stores it: bfloat16 or binary32 */
static double stored(const orc_cfg* c, double v) { return c->kv_bf16 ? orc_round_bf16(v) : (double)(float)v; }
void orc_mxfp8_round_row(int64_t n, double* v);

/* an activation the layer stores (not a cache entry): rounded unless kv_only */
static double stored_act(const orc_cfg* c, double v) { return c->kv_only ? v : stored(c, v); }
static void stored_array(const orc_cfg* c, int64_t n, double* v) {
  for (int64_t i = 0; i < n; ++i) v[i] = stored_act(c, v[i]);
}

/* ------------------------------------------------------------------------ */
/* page format                                                              */
/* ------------------------------------------------------------------------ */

static int64_t k_index(const orc_cfg* c, int64_t page, int g, int s, int i) {
  int64_t base = (page * c->n_kv_heads + g) * (int64_t)ORC_PAGE * c->head_dim;
  return base + ((i / 8) * ORC_PAGE + s) * 8 + i % 8;
}

static int64_t v_index(const orc_cfg* c, int64_t page, int g, int s, int i) {
  int64_t base = (page * c->n_kv_heads + g) * (int64_t)ORC_PAGE * c->head_dim;
  return base + (((i / 16) * (ORC_PAGE / 4) + s / 4) * 16 + i % 16) * 4 + s % 4;
}

/* physical page that holds position pos of sequence b, or -1 if not present */
static int64_t page_of(const int32_t* page_table, int max_pages, int n_pages, int b, int pos) {
  int lp = pos / ORC_PAGE;
  if (lp < 0 || lp >= max_pages) return -1;
  int32_t p = page_table[(int64_t)b * max_pages + lp];
  if (p < 0 || p >= n_pages) return -1;
  return p;
}

/* logical <-> page-format conversion of whole pools, for tests */
void orc_pool_to_logical(const orc_cfg* c, int n_pages, const float* k_pool, const float* v_pool,
                         float* k_out, float* v_out) {
  int d = c->head_dim;
  for (int64_t p = 0; p < n_pages; ++p)
    for (int g = 0; g < c->n_kv_heads; ++g)
      for (int s = 0; s < ORC_PAGE; ++s)
        for (int i = 0; i < d; ++i) {
          int64_t lin = ((p * c->n_kv_heads + g) * ORC_PAGE + s) * d + i;
          k_out[lin] = k_pool[k_index(c, p, g, s, i)];
          v_out[lin] = v_pool[v_index(c, p, g, s, i)];
        }
}

void orc_pool_from_logical(const orc_cfg* c, int n_pages, const float* k_in, const float* v_in,
                           float* k_pool, float* v_pool) {
  int d = c->head_dim;
  for (int64_t p = 0; p < n_pages; ++p)
    for (int g = 0; g < c->n_kv_heads; ++g)
      for (int s = 0; s < ORC_PAGE; ++s)
        for (int i = 0; i < d; ++i) {
          int64_t lin = ((p * c->n_kv_heads + g) * ORC_PAGE + s) * d + i;
          k_pool[k_index(c, p, g, s, i)] = k_in[lin];
          v_pool[v_index(c, p, g, s, i)] = v_in[lin];
        }
}

/* ------------------------------------------------------------------------ */
/* RMSNorm: y_i = x_i / sqrt(mean_j x_j^2 + eps) * g_i                       */
/* ------------------------------------------------------------------------ */

void orc_rmsnorm(int64_t rows, int dim, const double* x, const float* g, double eps, double* y) {
  for (int64_t r = 0; r < rows; ++r) {
    const double* xr = x + r * dim;
    double ss = 0.0;
    for (int i = 0; i < dim; ++i) ss += xr[i] * xr[i];
    double inv = 1.0 / sqrt(ss / dim + eps);
    for (int i = 0; i < dim; ++i) y[r * dim + i] = xr[i] * inv * (double)g[i];
  }
}

/* y[r][n] = sum_k x[r][k] * w[n][k] + (b ? b[n] : 0); w is [N][K] row-major */
static void linear(int64_t rows, int K, int N, const double* x, const float* w, const float* b,
                   double* y) {
  for (int64_t r = 0; r < rows; ++r)
    for (int n = 0; n < N; ++n) {
      double acc = 0.0;
      const float* wn = w + (int64_t)n * K;
      for (int k = 0; k < K; ++k) acc += x[r * K + k] * (double)wn[k];
      y[r * N + n] = acc + (b ? (double)b[n] : 0.0);
    }
}

/* ------------------------------------------------------------------------ */
/* Rotary position embedding on one head vector of length d at position pos: */
/* the pair (v_j, v_{j+d/2}) is rotated by the angle whose cosine and sine   */
/* are cos_tab[pos][j], sin_tab[pos][j].                                     */
/* ------------------------------------------------------------------------ */

void orc_rope(int d, int pos, const float* cos_tab, const float* sin_tab, double* v) {
  int h = d / 2;
  for (int j = 0; j < h; ++j) {
    double c = cos_tab[(int64_t)pos * h + j], s = sin_tab[(int64_t)pos * h + j];
    double a = v[j], b = v[j + h];
    v[j] = a * c - b * s;
    v[j + h] = a * s + b * c;
  }
}

/* ------------------------------------------------------------------------ */
/* KV append: token t of sequence tok_seq[t] at position tok_pos[t] stores   */
/* its key and value ([Hkv][d] each) into the pools, rounded to the cache    */
/* dtype.                                                                    */
/* ------------------------------------------------------------------------ */

int orc_kv_append(const orc_cfg* c, int T, const int32_t* tok_seq, const int32_t* tok_pos,
                  const double* k_new, const double* v_new, float* k_pool, float* v_pool,
                  const int32_t* page_table, int max_pages, int n_pages) {
  int d = c->head_dim, G = c->n_kv_heads;
  for (int t = 0; t < T; ++t) {
    int64_t page = page_of(page_table, max_pages, n_pages, tok_seq[t], tok_pos[t]);
    if (page < 0) return ORC_EINVAL;
    int s = tok_pos[t] % ORC_PAGE;
    for (int g = 0; g < G; ++g)
      for (int i = 0; i < d; ++i) {
        double kv = k_new[((int64_t)t * G + g) * d + i];
        double vv = v_new[((int64_t)t * G + g) * d + i];
        kv = stored(c, kv);
        vv = stored(c, vv);
        k_pool[k_index(c, page, g, s, i)] = (float)kv;
        v_pool[v_index(c, page, g, s, i)] = (float)vv;
      }
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Attention with a sink, one query token.                                   */
/*   Query head h reads KV head g = h / (Hq / Hkv).                           */
/*   Visible keys: j in [lo, p], lo = 0 (full) or max(0, p - window + 1).    */
/*   z_j = q_h . k_j / sqrt(d);  M = max(s_h, max_j z_j)                      */
/*   o_h = sum_j e^{z_j - M} v_j / (e^{s_h - M} + sum_j e^{z_j - M})          */
/* The sink logit s_h enters the normaliser only; it carries no value.       */
/* ------------------------------------------------------------------------ */

int orc_attention(const orc_cfg* c, int T, const int32_t* tok_seq, const int32_t* tok_pos,
                  const double* q, const float* k_pool, const float* v_pool,
                  const int32_t* page_table, int max_pages, int n_pages, const float* sinks,
                  double* o) {
  int d = c->head_dim, Hq = c->n_q_heads, Hkv = c->n_kv_heads, grp = Hq / Hkv;
  int bad = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : bad)
  for (int t = 0; t < T; ++t) {
    int b = tok_seq[t], p = tok_pos[t];
    int lo = c->window > 0 ? (p - c->window + 1 > 0 ? p - c->window + 1 : 0) : 0;
    int n = p - lo + 1;
    double* z = (double*)malloc(sizeof(double) * (size_t)n);
    for (int h = 0; h < Hq; ++h) {
      int g = h / grp;
      const double* qh = q + ((int64_t)t * Hq + h) * d;
      double M = sinks ? (double)sinks[h] : -INFINITY;
      for (int j = lo; j <= p; ++j) {
        int64_t page = page_of(page_table, max_pages, n_pages, b, j);
        if (page < 0) { bad = 1; z[j - lo] = -INFINITY; continue; }
        double dot = 0.0;
        for (int i = 0; i < d; ++i) dot += qh[i] * (double)k_pool[k_index(c, page, g, j % ORC_PAGE, i)];
        z[j - lo] = dot / sqrt((double)d);
        if (z[j - lo] > M) M = z[j - lo];
      }
      double L = sinks ? exp((double)sinks[h] - M) : 0.0;
      double* oh = o + ((int64_t)t * Hq + h) * d;
      for (int i = 0; i < d; ++i) oh[i] = 0.0;
      for (int j = lo; j <= p; ++j) {
        int64_t page = page_of(page_table, max_pages, n_pages, b, j);
        if (page < 0) continue;
        double e = exp(z[j - lo] - M);
        L += e;
        for (int i = 0; i < d; ++i) oh[i] += e * (double)v_pool[v_index(c, page, g, j % ORC_PAGE, i)];
      }
      for (int i = 0; i < d; ++i) oh[i] /= L;
    }
    free(z);
  }
  return bad ? ORC_EINVAL : ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Router and experts.                                                       */
/* ------------------------------------------------------------------------ */

/* SwiGLU in the clamped gpt-oss form: gate is capped above at L, up is      */
/* clamped to [-L, L]; a = gate * sigmoid(alpha * gate) * (up + beta).        */
/* alpha = 1, L = inf, beta = 0 is the plain SiLU(gate) * up.                 */
double orc_swiglu(double gate, double up, double alpha, double limit, double beta) {
  if (gate > limit) gate = limit;
  if (up > limit) up = limit;
  if (up < -limit) up = -limit;
  return gate / (1.0 + exp(-alpha * gate)) * (up + beta);
}

void orc_swiglu_array(int64_t n, const double* gate, const double* up, double alpha,
                      double limit, double beta, double* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_swiglu(gate[i], up[i], alpha, limit, beta);
}

/* Top-k selection over E logits: the k largest by value, ties to the lower   */
/* index; written in descending order. The comparison is made on the logits   */
/* rounded to fp32, the precision the GPU router decides in.                  */
void orc_topk(int E, int k, const double* logits, int32_t* idx) {
  int used[256] = {0};
  for (int s = 0; s < k; ++s) {
    int best = -1;
    float bv = 0.0f;
    for (int e = 0; e < E; ++e) {
      if (used[e]) continue;
      float v = (float)logits[e];
      if (best < 0 || v > bv) { best = e; bv = v; }
    }
    used[best] = 1;
    idx[s] = best;
  }
}

/* One token through one expert: gu = hn . W_gu[e]^T + b_gu[e], rows 2j/2j+1  */
/* are gate_j/up_j; a_j = swiglu(gate_j, up_j) (stored); y = a . W_d[e]^T +   */
/* b_d[e]. hn here is the stored copy of the normalised row.                  */
static void expert_ffn(const orc_cfg* c, const orc_weights* w, int e, const double* hn, double* y,
                       double* gu, double* act) {
  int H = c->hidden, I = c->ffn_dim;
  linear(1, H, 2 * I, hn, w->w_gu + (int64_t)e * 2 * I * H, w->b_gu + (int64_t)e * 2 * I, gu);
  for (int j = 0; j < I; ++j)
    act[j] = stored_act(c, orc_swiglu(gu[2 * j], gu[2 * j + 1], c->swiglu_alpha, c->swiglu_limit, c->swiglu_beta));
  if (c->act_mx) orc_mxfp8_round_row(I, act);  /* the second product reads the stored row in MXFP8 */
  linear(1, I, H, act, w->w_d + (int64_t)e * H * I, w->b_d + (int64_t)e * H, y);
}

/* MoE sub-block on the residual stream h [T][H]:                             */
/*   hn = RMSNorm(h; g2); logits = hn . W_r^T + b_r (hn unrounded);           */
/*   S = top-k set; w_e = softmax over {logits_e : e in S};                   */
/*   out = h + sum_{e in S} w_e * FFN_e(hn).                                  */
/* force_idx (optional [T][k]) replaces the selected set (used where the      */
/* k-th and (k+1)-th logits are within rounding of each other).              */
int orc_moe(const orc_cfg* c, const orc_weights* w, int T, const double* h, double* out,
            int32_t* idx_out, double* w_out, double* logits_out, double* moe_out,
            const int32_t* force_idx) {
  int H = c->hidden, E = c->n_experts, k = c->top_k, I = c->ffn_dim;
  if (k > E || E > 256) return ORC_EINVAL;
#pragma omp parallel for schedule(dynamic)
  for (int t = 0; t < T; ++t) {
    double* hn = (double*)malloc(sizeof(double) * (size_t)H);
    double* lg = (double*)malloc(sizeof(double) * (size_t)E);
    double* y = (double*)malloc(sizeof(double) * (size_t)H);
    double* acc = (double*)calloc((size_t)H, sizeof(double));
    double* gu = (double*)malloc(sizeof(double) * (size_t)2 * I);
    double* act = (double*)malloc(sizeof(double) * (size_t)I);
    int32_t sel[256];
    double wt[256];
    orc_rmsnorm(1, H, h + (int64_t)t * H, w->g2, c->rms_eps, hn);
    linear(1, H, E, hn, w->w_r, w->b_r, lg);
    stored_array(c, H, hn);  /* the router reads hn as computed; the experts its stored copy */
    if (c->act_mx) orc_mxfp8_round_row(H, hn);  /* ... in MXFP8 when the experts take MXFP8 rows */
    if (force_idx) memcpy(sel, force_idx + (int64_t)t * k, sizeof(int32_t) * (size_t)k);
    else orc_topk(E, k, lg, sel);
    double mx = -INFINITY, den = 0.0;
    for (int s = 0; s < k; ++s) if (lg[sel[s]] > mx) mx = lg[sel[s]];
    for (int s = 0; s < k; ++s) { wt[s] = exp(lg[sel[s]] - mx); den += wt[s]; }
    for (int s = 0; s < k; ++s) wt[s] /= den;
    for (int s = 0; s < k; ++s) {
      expert_ffn(c, w, sel[s], hn, y, gu, act);
      for (int n = 0; n < H; ++n) acc[n] += wt[s] * y[n];
    }
    for (int n = 0; n < H; ++n) out[(int64_t)t * H + n] = h[(int64_t)t * H + n] + acc[n];
    if (moe_out) memcpy(moe_out + (int64_t)t * H, acc, sizeof(double) * (size_t)H);
    if (idx_out) memcpy(idx_out + (int64_t)t * k, sel, sizeof(int32_t) * (size_t)k);
    if (w_out) memcpy(w_out + (int64_t)t * k, wt, sizeof(double) * (size_t)k);
    if (logits_out) memcpy(logits_out + (int64_t)t * E, lg, sizeof(double) * (size_t)E);
    free(hn); free(lg); free(y); free(acc); free(gu); free(act);
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* One decoder-layer step over a batch of sequences.                        */
/*   seq_lens[b]: tokens already cached; cu_q (optional, [B+1]): token b's    */
/*   new tokens are rows cu_q[b] .. cu_q[b+1]-1 of x_in, at positions         */
/*   seq_lens[b] + i. cu_q = NULL means one new token per sequence.           */
/* Per token at position p (xn, q, k, v and o are stored, i.e. rounded to    */
/* the layer dtype):                                                         */
/*   xn = RMSNorm(x; g1); [q | k | v] = xn . W_qkv^T + b_qkv;                 */
/*   q, k rotated at p; k, v stored in the cache;                            */
/*   o = attention with sink (after every new k, v is stored);               */
/*   h1 = x + o . W_o^T + b_o;  out = MoE(h1).                                */
/* ------------------------------------------------------------------------ */

/* n_eval / eval_rows (optional): every new token is projected and appended,  */
/* but attention, the output projection and the MoE are evaluated only for   */
/* the listed rows (ascending), whose results fill the outputs in that order */
/* (x_in and force_idx are still indexed by row). A token's result depends   */
/* only on its own row and the cache, so this changes no value.              */
static int decode_layer_rows(const orc_cfg* c, const orc_weights* w, int B, const int32_t* page_table,
                             int max_pages, int n_pages, const int32_t* seq_lens, const int32_t* cu_q,
                             float* k_pool, float* v_pool, const double* x_in, int n_eval,
                             const int32_t* eval_rows, double* x_out, double* q_out, double* o_out,
                             double* h1_out, int32_t* idx_out, double* w_out, double* logits_out,
                             double* moe_out, const int32_t* force_idx) {
  int H = c->hidden, d = c->head_dim, Hq = c->n_q_heads, Hkv = c->n_kv_heads;
  int QKV = (Hq + 2 * Hkv) * d, A = Hq * d;
  if (c->page_size != ORC_PAGE || Hq % Hkv) return ORC_EINVAL;
  int T = cu_q ? cu_q[B] : B;
  int32_t* tok_seq = (int32_t*)malloc(sizeof(int32_t) * (size_t)T);
  int32_t* tok_pos = (int32_t*)malloc(sizeof(int32_t) * (size_t)T);
  for (int b = 0; b < B; ++b) {
    int r0 = cu_q ? cu_q[b] : b, r1 = cu_q ? cu_q[b + 1] : b + 1;
    for (int r = r0; r < r1; ++r) { tok_seq[r] = b; tok_pos[r] = seq_lens[b] + (r - r0); }
  }
  int NE = eval_rows ? n_eval : T;
  int32_t* rows = (int32_t*)malloc(sizeof(int32_t) * (size_t)(NE > 0 ? NE : 1));
  for (int e = 0; e < NE; ++e) rows[e] = eval_rows ? eval_rows[e] : e;
  double* xn = (double*)malloc(sizeof(double) * (size_t)T * H);
  double* qkv = (double*)malloc(sizeof(double) * (size_t)T * QKV);
  double* q = (double*)malloc(sizeof(double) * (size_t)T * A);
  double* kn = (double*)malloc(sizeof(double) * (size_t)T * Hkv * d);
  double* vn = (double*)malloc(sizeof(double) * (size_t)T * Hkv * d);
  int32_t* e_seq = (int32_t*)malloc(sizeof(int32_t) * (size_t)(NE > 0 ? NE : 1));
  int32_t* e_pos = (int32_t*)malloc(sizeof(int32_t) * (size_t)(NE > 0 ? NE : 1));
  double* eq = (double*)malloc(sizeof(double) * (size_t)(NE > 0 ? NE : 1) * A);
  double* ex = (double*)malloc(sizeof(double) * (size_t)(NE > 0 ? NE : 1) * H);
  int32_t* ef = force_idx ? (int32_t*)malloc(sizeof(int32_t) * (size_t)(NE > 0 ? NE : 1) * c->top_k) : NULL;
  double* o = (double*)malloc(sizeof(double) * (size_t)(NE > 0 ? NE : 1) * A);
  double* h1 = (double*)malloc(sizeof(double) * (size_t)(NE > 0 ? NE : 1) * H);
  int rc = ORC_OK;

  for (int e = 0; e < NE; ++e)
    if (rows[e] < 0 || rows[e] >= T || (e > 0 && rows[e] <= rows[e - 1])) { rc = ORC_EINVAL; goto done; }
  orc_rmsnorm(T, H, x_in, w->g1, c->rms_eps, xn);
  stored_array(c, (int64_t)T * H, xn);
#pragma omp parallel for schedule(static)
  for (int t = 0; t < T; ++t) linear(1, H, QKV, xn + (int64_t)t * H, w->w_qkv, w->b_qkv, qkv + (int64_t)t * QKV);
  for (int t = 0; t < T; ++t) {
    if (tok_pos[t] >= w->rope_max_pos) { rc = ORC_EINVAL; goto done; }
    for (int h = 0; h < Hq; ++h) {
      double* qh = q + ((int64_t)t * Hq + h) * d;
      memcpy(qh, qkv + (int64_t)t * QKV + h * d, sizeof(double) * (size_t)d);
      orc_rope(d, tok_pos[t], w->rope_cos, w->rope_sin, qh);
      stored_array(c, d, qh);
    }
    for (int g = 0; g < Hkv; ++g) {
      double* kh = kn + ((int64_t)t * Hkv + g) * d;
      memcpy(kh, qkv + (int64_t)t * QKV + A + g * d, sizeof(double) * (size_t)d);
      orc_rope(d, tok_pos[t], w->rope_cos, w->rope_sin, kh);
      memcpy(vn + ((int64_t)t * Hkv + g) * d, qkv + (int64_t)t * QKV + A + Hkv * d + g * d,
             sizeof(double) * (size_t)d);
    }
  }
  rc = orc_kv_append(c, T, tok_seq, tok_pos, kn, vn, k_pool, v_pool, page_table, max_pages, n_pages);
  if (rc) goto done;
  for (int e = 0; e < NE; ++e) {
    e_seq[e] = tok_seq[rows[e]];
    e_pos[e] = tok_pos[rows[e]];
    memcpy(eq + (int64_t)e * A, q + (int64_t)rows[e] * A, sizeof(double) * (size_t)A);
    memcpy(ex + (int64_t)e * H, x_in + (int64_t)rows[e] * H, sizeof(double) * (size_t)H);
    if (ef) memcpy(ef + (int64_t)e * c->top_k, force_idx + (int64_t)rows[e] * c->top_k, sizeof(int32_t) * (size_t)c->top_k);
  }
  rc = orc_attention(c, NE, e_seq, e_pos, eq, k_pool, v_pool, page_table, max_pages, n_pages, w->sinks, o);
  if (rc) goto done;
  stored_array(c, (int64_t)NE * A, o);
#pragma omp parallel for schedule(static)
  for (int e = 0; e < NE; ++e) {
    linear(1, A, H, o + (int64_t)e * A, w->w_o, w->b_o, h1 + (int64_t)e * H);
    for (int n = 0; n < H; ++n) h1[(int64_t)e * H + n] += ex[(int64_t)e * H + n];
  }
  rc = orc_moe(c, w, NE, h1, x_out, idx_out, w_out, logits_out, moe_out, ef);
  if (q_out) memcpy(q_out, eq, sizeof(double) * (size_t)NE * A);
  if (o_out) memcpy(o_out, o, sizeof(double) * (size_t)NE * A);
  if (h1_out) memcpy(h1_out, h1, sizeof(double) * (size_t)NE * H);
done:
  free(tok_seq); free(tok_pos); free(rows); free(xn); free(qkv); free(q); free(kn); free(vn);
  free(e_seq); free(e_pos); free(eq); free(ex); free(ef); free(o); free(h1);
  return rc;
}

int orc_decode_layer(const orc_cfg* c, const orc_weights* w, int B, const int32_t* page_table,
                     int max_pages, int n_pages, const int32_t* seq_lens, const int32_t* cu_q,
                     float* k_pool, float* v_pool, const double* x_in, double* x_out,
                     double* q_out, double* o_out, double* h1_out, int32_t* idx_out,
                     double* w_out, double* logits_out, double* moe_out,
                     const int32_t* force_idx) {
  return decode_layer_rows(c, w, B, page_table, max_pages, n_pages, seq_lens, cu_q, k_pool, v_pool, x_in, 0,
                           NULL, x_out, q_out, o_out, h1_out, idx_out, w_out, logits_out, moe_out, force_idx);
}

int orc_decode_layer_rows(const orc_cfg* c, const orc_weights* w, int B, const int32_t* page_table,
                          int max_pages, int n_pages, const int32_t* seq_lens, const int32_t* cu_q,
                          float* k_pool, float* v_pool, const double* x_in, int n_eval,
                          const int32_t* eval_rows, double* x_out, double* q_out, double* o_out,
                          double* h1_out, int32_t* idx_out, double* w_out, double* logits_out,
                          double* moe_out, const int32_t* force_idx) {
  if (!eval_rows) return ORC_EINVAL;
  return decode_layer_rows(c, w, B, page_table, max_pages, n_pages, seq_lens, cu_q, k_pool, v_pool, x_in,
                           n_eval, eval_rows, x_out, q_out, o_out, h1_out, idx_out, w_out, logits_out,
                           moe_out, force_idx);
}

/* ------------------------------------------------------------------------ */
/* MXFP4 (OCP Microscaling Formats v1.0): blocks of 32 along a row share one  */
/* E8M0 scale 2^(s - 127); each element is FP4 E2M1 (sign, 2-bit exponent,   */
/* 1-bit mantissa, bias 1): magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6.            */
/* codes: [rows][cols/2], low nibble = even column. scales: [rows][cols/32].  */
/* ------------------------------------------------------------------------ */

double orc_e2m1(int code) {
  int sign = (code >> 3) & 1, ex = (code >> 1) & 3, man = code & 1;
  double mag = ex == 0 ? 0.5 * man : ldexp(1.0 + 0.5 * man, ex - 1);
  return sign ? -mag : mag;
}

int orc_mxfp4_dequant(int64_t rows, int cols, const uint8_t* codes, const uint8_t* scales,
                      float* out) {
  if (cols % 32) return ORC_EINVAL;
  double value[16];
  for (int c = 0; c < 16; ++c) value[c] = orc_e2m1(c);
  int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
  for (int64_t r = 0; r < rows; ++r)
    for (int blk = 0; blk < cols / 32; ++blk) {
      uint8_t s = scales[r * (cols / 32) + blk];
      if (s == 0xFF) { bad = 1; continue; } /* NaN scale is not a weight */
      double scale = ldexp(1.0, (int)s - 127);
      for (int j = 32 * blk; j < 32 * blk + 32; ++j) {
        uint8_t byte = codes[r * (cols / 2) + j / 2];
        int code = (j % 2 == 0) ? (byte & 0xF) : (byte >> 4);
        out[r * cols + j] = (float)(value[code] * scale);
      }
    }
  return bad ? ORC_EINVAL : ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Generation ends: the vocabulary head and next-token sampling.             */
/* The rollouts sample at a fixed temperature (0.7 in the paper's training   */
/* details) and the GRPO update rescores whole trajectories under the policy */
/* (Sec. 3.2, Sec. 4).                                                        */
/* ------------------------------------------------------------------------ */

/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011): a round maps counter  */
/* (c0, c1, c2, c3) under key (k0, k1) to                                    */
/*   (hi(B*c2) ^ c1 ^ k0, lo(B*c2), hi(A*c0) ^ c3 ^ k1, lo(A*c0))            */
/* with A = 0xD2511F53, B = 0xCD9E8D57 (hi/lo: upper and lower 32 bits of the */
/* 64-bit product); ten rounds, the key advanced by (0x9E3779B9, 0xBB67AE85)  */
/* before every round after the first.                                       */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3], k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    uint64_t pa = (uint64_t)0xD2511F53u * c0, pb = (uint64_t)0xCD9E8D57u * c2;
    uint32_t n0 = (uint32_t)(pb >> 32) ^ c1 ^ k0, n1 = (uint32_t)pb;
    uint32_t n2 = (uint32_t)(pa >> 32) ^ c3 ^ k1, n3 = (uint32_t)pa;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

#define ORC_SAMPLE_TAG 0x4C4D5330u

/* The uniform draw of vocabulary entry v for (seed, sequence, position):    */
/* word v % 4 of Philox at counter (v / 4, pos, seq, tag), key (seed low,     */
/* seed high); u = (w / 2^9 rounded down + 1/2) / 2^23, strictly in (0, 1).   */
double orc_sample_uniform(uint64_t seed, int seq, int pos, int v) {
  uint32_t ctr[4] = {(uint32_t)v / 4u, (uint32_t)pos, (uint32_t)seq, ORC_SAMPLE_TAG};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)}, w[4];
  orc_philox4x32_10(ctr, key, w);
  return ((double)(w[v % 4] >> 9) + 0.5) / 8388608.0;
}

/* Gumbel noise of a uniform: g = -log(-log u). */
double orc_gumbel(double u) { return -log(-log(u)); }

/* Vocabulary head for T rows of the residual stream x [T][H]:               */
/*   xn = RMSNorm(x; g_final), stored (bf16); l_v = xn . W_lm[v] (float64);   */
/*   s = l / temperature (temperature > 0), else s = l;                       */
/*   lse = log sum_v e^{s_v};                                                 */
/*   token = argmax_v (s_v + g_v) with g_v the Gumbel noise of the row's      */
/*   (seed, seq, pos) draws (temperature > 0), or argmax_v l_v (greedy);      */
/*   the maximum is taken over values rounded to fp32 (the precision the GPU  */
/*   decides in), the lower id on equal values;                               */
/*   logprob = s_token - lse; target_logprob = s_target - lse.                */
/* logits_out (optional) receives l [T][V]; pert_out (optional) the float64   */
/* perturbed scores s + g [T][V] before rounding.                              */
int orc_lm_head(int T, int H, int V, const double* x, const float* g_final, double eps, const float* w_lm,
                double temperature, uint64_t seed, const int32_t* seq_ids, const int32_t* positions,
                const int32_t* targets, int32_t* tokens, double* logprob, double* lse_out,
                double* target_logprob, double* logits_out, double* pert_out) {
  int greedy = !(temperature > 0.0);
  if (!greedy && (!seq_ids || !positions)) return ORC_EINVAL;
#pragma omp parallel for schedule(dynamic)
  for (int t = 0; t < T; ++t) {
    double* xn = (double*)malloc(sizeof(double) * (size_t)H);
    double* s = (double*)malloc(sizeof(double) * (size_t)V);
    orc_rmsnorm(1, H, x + (int64_t)t * H, g_final, eps, xn);
    for (int h = 0; h < H; ++h) xn[h] = orc_round_bf16(xn[h]);
    double mx = -INFINITY;
    for (int v = 0; v < V; ++v) {
      double l = 0.0;
      const float* w = w_lm + (int64_t)v * H;
      for (int h = 0; h < H; ++h) l += xn[h] * (double)w[h];
      if (logits_out) logits_out[(int64_t)t * V + v] = l;
      s[v] = greedy ? l : l / temperature;
      if (s[v] > mx) mx = s[v];
    }
    double sum = 0.0;
    for (int v = 0; v < V; ++v) sum += exp(s[v] - mx);
    double lse = mx + log(sum);
    int best = -1;
    float bv = 0.0f;
    for (int v = 0; v < V; ++v) {
      double p = s[v];
      if (!greedy) p += orc_gumbel(orc_sample_uniform(seed, seq_ids[t], positions[t], v));
      if (pert_out) pert_out[(int64_t)t * V + v] = p;
      float pf = (float)p;
      if (best < 0 || pf > bv) { best = v; bv = pf; }
    }
    if (tokens) tokens[t] = best;
    if (logprob) logprob[t] = s[best] - lse;
    if (lse_out) lse_out[t] = lse;
    if (target_logprob && targets) {
      int tg = targets[t];
      target_logprob[t] = (tg >= 0 && tg < V) ? s[tg] - lse : -INFINITY;
    }
    free(xn); free(s);
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* MXFP8 activations for the scaled matrix-core expert products (OCP        */
/* Microscaling Formats v1.0): blocks of 32 consecutive elements of a row    */
/* along the reduction axis share one E8M0 scale X = 2^e with                */
/*   e = floor(log2(max |v|)) - 8   (8: the largest exponent of E4M3),       */
/* and each element is v / X rounded to the nearest FP8 E4M3 value (ties to  */
/* the even code), saturating at +-448. E4M3: sign, 4 exponent bits (bias 7), */
/* 3 mantissa bits; exponent 0 holds the subnormals m / 8 * 2^-6; S.1111.111 */
/* is NaN (never produced). An all-zero block gets scale byte 0 and zeros.   */
/* The input is the stored bf16 row, so both sides quantize identical values. */
/* ------------------------------------------------------------------------ */

double orc_e4m3(int code) {
  int sign = (code >> 7) & 1, ex = (code >> 3) & 15, man = code & 7;
  if (ex == 15 && man == 7) return NAN;
  double mag = ex == 0 ? ldexp((double)man / 8.0, -6) : ldexp(1.0 + man / 8.0, ex - 7);
  return sign ? -mag : mag;
}

/* the nearest E4M3 code to x (ties to the even code), |x| saturating at 448 */
int orc_e4m3_encode(double x) {
  int sign = x < 0 ? 0x80 : 0;
  double a = fabs(x);
  int best = 0;
  double bd = INFINITY;
  for (int c = 0; c <= 0x7E; ++c) {  /* the 127 finite non-negative codes, ascending */
    double d = fabs(orc_e4m3(c) - a);
    if (d < bd || (d == bd && (c & 1) == 0)) { bd = d; best = c; }
  }
  if (best == 0) sign = 0;  /* no negative zero */
  return sign | best;
}

int orc_mxfp8_quant(int64_t rows, int cols, const double* in, uint8_t* codes, uint8_t* scales) {
  if (cols % 32) return ORC_EINVAL;
  for (int64_t r = 0; r < rows; ++r)
    for (int blk = 0; blk < cols / 32; ++blk) {
      const double* v = in + r * cols + 32 * blk;
      double amax = 0.0;
      for (int j = 0; j < 32; ++j) if (fabs(v[j]) > amax) amax = fabs(v[j]);
      int e = -127;
      if (amax > 0.0) {
        int ex;
        frexp(amax, &ex);  /* amax = f * 2^ex, f in [0.5, 1): floor(log2 amax) = ex - 1 */
        e = ex - 1 - 8;
        if (e < -127) e = -127;
        if (e > 127) e = 127;
      }
      scales[r * (cols / 32) + blk] = (uint8_t)(e + 127);
      for (int j = 0; j < 32; ++j) codes[r * cols + 32 * blk + j] = (uint8_t)orc_e4m3_encode(ldexp(v[j], -e));
    }
  return ORC_OK;
}

/* a row replaced by its MXFP8 value (quantize, then decode exactly) */
void orc_mxfp8_round_row(int64_t n, double* v) {
  uint8_t codes[32], scale;
  for (int64_t b = 0; b + 32 <= n; b += 32) {
    orc_mxfp8_quant(1, 32, v + b, codes, &scale);
    for (int j = 0; j < 32; ++j) v[b + j] = ldexp(orc_e4m3(codes[j]), (int)scale - 127);
  }
}
