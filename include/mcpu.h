/*
 * mcpu.h -- C ABI of the MI355X (gfx950) decode-layer library.
 *
 * What it computes. The paper's rollout pipeline keeps the GPU busy with
 * generation while trajectories wait on tools: the Run stage is GPU bound and
 * dominated by generation (Sec. 3.2), the policy is gpt-oss-20b (Sec. 4), and
 * each turn's tool observation is appended to the context (Sec. 1, Sec. 3.2).
 * This library runs that generation's per-layer work for a batch of
 * concurrent trajectories: one decoder-layer step of a gpt-oss-20b-shaped MoE
 * transformer over a paged KV cache, where every sequence brings one new token
 * (decode) or a chunk of new tokens (an appended tool observation).
 *
 * Conventions shared by every entry point:
 *  - All device buffers belong to the caller. The library never allocates
 *    device memory; scratch comes from a caller-provided workspace.
 *  - Launches are asynchronous on the caller's stream; no entry point except
 *    mcpu_check_device_errors synchronises or copies device data to the host.
 *  - Return value: MCPU_OK or a negative mcpu_status; on error nothing was
 *    launched (host-detected) and mcpu_last_error() describes the cause. No
 *    C++ exception crosses the ABI.
 *  - Results are deterministic: no floating-point atomics, fixed reduction
 *    orders, independent of the physical page placement.
 *  - Workspace: device memory of at least the *_workspace_size() bytes,
 *    256-byte aligned. Its first 256 bytes hold the device error word and must
 *    be zero before the first call (e.g. allocate it zero-filled); errors then
 *    accumulate until mcpu_check_device_errors() reads and clears them.
 *
 * Paged KV cache (the page format). A pool holds n_pages pages. Page p, KV
 * head g holds 16 consecutive token positions x head_dim dims, at element
 * base (p * n_kv_heads + g) * 16 * head_dim of the K pool and of the V pool.
 * Within that block:
 *   K(slot s, dim i) at ((i / 8) * 16 + s) * 8 + i % 8
 *   V(slot s, dim i) at (((i / 16) * 4 + s / 4) * 16 + i % 16) * 4 + s % 4
 * so one 64-lane wavefront reads a page as whole contiguous segments already
 * in matrix-core operand order. Token position pos of sequence b lives in page
 * page_table[b * max_pages + pos / 16], slot pos % 16. Unused page-table
 * entries are -1. The element type is the layer dtype (fp32 or bf16).
 *
 * Positions. seq_lens[b] counts the tokens of sequence b already in the cache
 * before the step. A step writes its new tokens at positions seq_lens[b] ..
 * seq_lens[b] + q_len_b - 1 and then attends; the caller advances seq_lens
 * afterwards. Pages covering the new positions must be allocated beforehand.
 * Sliding-window layers read only pages that intersect [pos - window + 1, pos],
 * so pages left of the window may be freed (page-table entry -1).
 */
#ifndef MCPU_H
#define MCPU_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MCPU_OK = 0,
  MCPU_EINVAL = -1,       /* bad shape, pointer, size or configuration */
  MCPU_ENOMEM = -2,       /* page pool exhausted (kv_pages_alloc) or workspace too small */
  MCPU_EHIP = -3,         /* a HIP runtime call or kernel launch failed */
  MCPU_EUNSUPPORTED = -4, /* valid but not implemented (e.g. head_dim other than 32/64) */
  MCPU_EDEVICE = -5       /* a kernel found invalid data (see mcpu_check_device_errors) */
} mcpu_status;

enum { MCPU_F32 = 0, MCPU_BF16 = 1 };               /* layer dtype */
/* expert weight format: dense (layer dtype); MXFP4 weights decoded to bf16
 * for bf16 products; or MXFP4 weights on the scaled matrix cores against
 * MXFP8 activations (the normalised rows and the SwiGLU activations are
 * quantized per 32 elements, see moe_forward) */
enum { MCPU_EXPERT_DENSE = 0, MCPU_EXPERT_MXFP4 = 1, MCPU_EXPERT_MXFP4_NATIVE = 2 };

/* Device error bits (mcpu_check_device_errors). */
enum {
  MCPU_DEVERR_PAGE = 1,  /* a needed page-table entry was -1 or >= n_pages; its keys were skipped */
  MCPU_DEVERR_ROPE = 2,  /* a position was >= rope_max_pos; that token's q/k were not written */
  MCPU_DEVERR_EXPERT = 4, /* a top-k expert id outside [0, n_experts) was passed in */
  MCPU_DEVERR_PLAN = 8,   /* device seq_lens / cu_q disagree with the host copies */
  MCPU_DEVERR_MXFP4 = 16, /* an MXFP4 block scale outside [2, 252]: scaled values would not be
                             normal bfloat16; that block contributed zero */
  MCPU_DEVERR_TOKEN = 32  /* a token id outside [0, vocab) (embed_tokens); its row was zeroed */
};

/* Layer configuration (host struct, by value semantics). Paper: the policy
 * is gpt-oss-20b (Sec. 4 and the training-details appendix); its layer
 * shape is one instance of this struct.
 *  hidden H, n_q_heads Hq, n_kv_heads Hkv (Hq % Hkv == 0, Hq / Hkv <= 16),
 *  head_dim d in {32, 64}, n_experts E <= 64, top_k k <= min(E, 8),
 *  ffn_dim I (expert SwiGLU width); H, I and Hq * d multiples of 32.
 *  page_size must be 16. window 0 = full attention, else keys
 *  [pos - window + 1, pos]. dtype: MCPU_F32 or MCPU_BF16 for the matrices,
 *  the KV cache and matrix-core operands. expert_fmt: MCPU_EXPERT_DENSE
 *  (experts in dtype), MCPU_EXPERT_MXFP4 or MCPU_EXPERT_MXFP4_NATIVE (bf16
 *  layers only).
 *  SwiGLU: a = min(gate, L) * sigmoid(alpha * min(gate, L)) * (clamp(up, -L, L) + beta)
 *  with alpha = swiglu_alpha, L = swiglu_limit (may be +inf), beta = swiglu_beta. */
typedef struct mcpu_layer_cfg {
  int32_t hidden, n_q_heads, n_kv_heads, head_dim, n_experts, top_k, ffn_dim;
  int32_t page_size, window, dtype, expert_fmt;
  float rms_eps, swiglu_alpha, swiglu_limit, swiglu_beta;
} mcpu_layer_cfg;

/* Layer parameters (the policy's weights, Sec. 4): device pointers owned by
 * the caller. Matrices are
 * row-major with the reduction dimension contiguous, in the layer dtype
 * ("T") unless stated. Vectors are fp32.
 *  g1, g2 [H]            RMSNorm gains before attention and before the MoE
 *  w_qkv [(Hq+2Hkv)d, H] T   rows: all Q heads, then K heads, then V heads
 *  b_qkv [(Hq+2Hkv)d]
 *  w_o [H, Hq d] T, b_o [H]
 *  w_r [E, H] T, b_r [E] router (logits are formed in fp32)
 *  w_gu [E, 2I, H], b_gu [E, 2I]  row 2j is gate_j, row 2j+1 is up_j
 *  w_d [E, H, I], b_d [E, H]
 *    dense experts: w_gu/w_d in T, s_gu = s_d = NULL.
 *    MXFP4 experts: w_gu/w_d hold E2M1 codes, [E, rows, cols/2] bytes, low
 *    nibble = even column; s_gu/s_d hold E8M0 block scales [E, rows, cols/32].
 *  sinks [Hq]            one attention-sink logit per query head
 *  rope_cos, rope_sin [rope_max_pos, d/2]  rotation of the pair (j, j + d/2)
 *  w_gu_packed, w_d_packed  optional (NULL): bf16 dense experts w_gu and w_d
 *    in the streaming order written by mcpu_pack_weights. The grouped GEMMs
 *    of short expert groups (decode batches of a few hundred tokens) then
 *    read each 16-row by 128-column block as 4 KiB in a row; w_gu and w_d
 *    stay required for the other tilings.
 *    MCPU_EXPERT_MXFP4_NATIVE: required, the slice-order copies of the MXFP4
 *    experts (codes and scales) written by mcpu_pack_mxfp4, 256-byte
 *    aligned; the products read only these.
 *  w_qkv_packed, w_o_packed  optional (NULL): bf16 w_qkv and w_o in the same
 *    streaming order (mcpu_pack_weights with one group, rows in their own
 *    order), read by the projections of steps of up to 64 tokens and by the
 *    O projection of prefill-sized steps; w_qkv and w_o stay required. */
typedef struct mcpu_layer_weights {
  const float* g1;
  const void* w_qkv;
  const float* b_qkv;
  const void* w_o;
  const float* b_o;
  const float* g2;
  const void* w_r;
  const float* b_r;
  const void* w_gu;
  const float* b_gu;
  const void* w_d;
  const float* b_d;
  const uint8_t* s_gu;
  const uint8_t* s_d;
  const float* sinks;
  const float* rope_cos;
  const float* rope_sin;
  int32_t rope_max_pos;
  const void* w_gu_packed;
  const void* w_d_packed;
  const void* w_qkv_packed;
  const void* w_o_packed;
} mcpu_layer_weights;

/* Weights in streaming order (bf16 only), a layout aid for the decode-sized
 * expert GEMMs of the Run stage's generation (Sec. 3.2). src is [n_groups, rows, cols]
 * row-major with cols contiguous; rows a multiple of 16, cols of 64. dst
 * (mcpu_packed_weights_bytes bytes, caller-owned, not aliasing src) receives,
 * per group, row block rb (16 rows) and column chunk c (128 columns), a
 * 4096-byte block at ((group * rows/16 + rb) * ceil(cols/128) + c) * 4096:
 * sixteen-byte piece t * 64 + lane (t = 0..3, lane = r + 16 j with r, j =
 * 0..15, 0..3) holds src[group][16 rb + r][128 c + 32 t + 8 j .. + 7], zero
 * past cols. That is the operand order of the 16 x 16 x 32 matrix-core
 * products, so each product's weight fragment is one contiguous KiB.
 * Asynchronous on stream; returns 0 on success or mcpu_status (EINVAL for
 * bad sizes or NULL pointers, EUNSUPPORTED for a non-bf16 dtype) and then
 * launches nothing. */
size_t mcpu_packed_weights_bytes(int32_t n_groups, int32_t rows, int32_t cols);
int mcpu_pack_weights(int32_t dtype, const void* src, void* dst, int32_t n_groups, int32_t rows, int32_t cols,
                      hipStream_t stream);

/* MXFP4 expert weights in slice order, for MCPU_EXPERT_MXFP4_NATIVE (written
 * once, like the streaming-order copies above). codes [n_groups, rows,
 * cols/2] (E2M1, low nibble = even column, 16-byte aligned) and scales
 * [n_groups, rows, cols/32] (E8M0) as for MCPU_EXPERT_MXFP4; rows a multiple
 * of 16, cols of 64. dst (mcpu_packed_mxfp4_bytes bytes, 256-byte aligned,
 * caller-owned, overlapping neither source) receives
 *   codes: group g, 64-column slice s, row r: the row's 32 code bytes of the
 *     slice at ((g * cols/64 + s) * rows + r) * 32;
 *   scales, from byte C = ceil(n_groups * rows * cols/2 / 256) * 256: group g,
 *     128-column group q, row r: the four scale bytes of blocks 4q .. 4q+3 at
 *     C + ((g * ceil(cols/128) + q) * rows + r) * 4 (127 past the last block),
 * so that one 64-wide reduction slice of 256 consecutive rows is one
 * contiguous run of codes and one of scales. Asynchronous on stream; returns
 * 0 or MCPU_EINVAL (bad sizes, NULL, misaligned or overlapping buffers, then
 * nothing is launched). */
size_t mcpu_packed_mxfp4_bytes(int32_t n_groups, int32_t rows, int32_t cols);
int mcpu_pack_mxfp4(const uint8_t* codes, const uint8_t* scales, void* dst, int32_t n_groups, int32_t rows,
                    int32_t cols, hipStream_t stream);

/* Opaque page pool: host-side free list over a caller-owned pair of device
 * pools (K and V, each n_pages * Hkv * 16 * d elements of the layer dtype).
 * Paper: trajectories are multi-turn and their contexts grow by every turn's
 * tool observation (Sec. 1, Sec. 3.2), so cache pages are taken as a
 * sequence grows and returned when it ends. */
typedef struct mcpu_kv_pool mcpu_kv_pool;

/* Thread-local description of the last non-OK return of this thread. */
const char* mcpu_last_error(void);

/* Create a pool handle over device buffers k_pool / v_pool. All pages start
 * free. The handle does not own the buffers. */
int kv_pool_create(const mcpu_layer_cfg* cfg, int32_t n_pages, void* k_pool, void* v_pool,
                   mcpu_kv_pool** out);
int kv_pool_destroy(mcpu_kv_pool* pool);
/* Number of free pages. */
int32_t kv_pool_free_pages(const mcpu_kv_pool* pool);

/* Allocate n pages, all or nothing, writing their ids to host array out_ids
 * (per-turn growth of a trajectory's context, Sec. 3.2).
 * MCPU_ENOMEM (nothing allocated) when fewer than n are free. Ids come out in
 * ascending order of the free list, lowest first. */
int kv_pages_alloc(mcpu_kv_pool* pool, int32_t n, int32_t* out_ids);
/* Return n pages (a finished trajectory, or sliding-window pages left behind
 * the window). MCPU_EINVAL, freeing nothing, if any id is out
 * of range, not allocated, or repeated. */
int kv_pages_free(mcpu_kv_pool* pool, int32_t n, const int32_t* ids);

/* Write new keys and values into the cache (the append of a step; Sec. 1 and
 * Sec. 3.2: generated tokens and tool observations join the context).
 *  batch sequences; page_table [batch, max_pages], seq_lens [batch] and cu_q
 *  [batch+1] are device int32; new token row r in [cu_q[b], cu_q[b+1]) of
 *  sequence b goes to position seq_lens[b] + r - cu_q[b]. cu_q == NULL means
 *  one token per sequence (row b). n_tokens = total rows.
 *  k_new, v_new: [n_tokens, Hkv, d] device arrays in the layer dtype, stored
 *  bit-exactly. Missing pages set MCPU_DEVERR_PAGE and skip that token.
 *  workspace: at least 256 bytes (error word). */
int kv_pages_append(mcpu_kv_pool* pool, int32_t batch, const int32_t* page_table,
                    int32_t max_pages, const int32_t* seq_lens, const int32_t* cu_q,
                    int32_t n_tokens, const void* k_new, const void* v_new, void* workspace,
                    size_t ws_bytes, hipStream_t stream);

/* Attention of already-appended queries over the paged cache, with sinks
 * (the attention of the policy's layers, Sec. 4, over contexts that grow by
 * appended observations, Sec. 1).
 *  q [n_tokens, Hq, d] (layer dtype, rotated), o [n_tokens, Hq * d] (layer dtype).
 *  Token row r of sequence b sits at position p = seq_lens[b] + (r - cu_q[b])
 *  and attends keys [lo, p] (lo = 0, or max(0, p - window + 1)):
 *    o_h = sum_j e^{z_j - M} v_j / (e^{s_h - M} + sum_j e^{z_j - M}),
 *    z_j = q_h . k_j / sqrt(d), M = max(s_h, max_j z_j), s_h = sinks[h],
 *  with query head h reading KV head h / (Hq / Hkv). sinks may be NULL (no sink).
 *  host_seq_lens / host_cu_q: host copies of the same arrays, used only to
 *  plan the launch (no device-to-host traffic). A sequence that adds 16 or
 *  more rows in the step (a tool observation appended as a prefill chunk,
 *  paper Section 1) is served by the chunked-prefill kernel, the other rows
 *  by split-K decode attention; the result is the same formula either way. */
size_t paged_attention_workspace_size(const mcpu_layer_cfg* cfg, int32_t max_batch,
                                      int32_t max_tokens);
int paged_attention(const mcpu_layer_cfg* cfg, const float* sinks, mcpu_kv_pool* pool,
                    int32_t batch, const int32_t* page_table, int32_t max_pages,
                    const int32_t* seq_lens, const int32_t* cu_q, const int32_t* host_seq_lens,
                    const int32_t* host_cu_q, const void* q, void* o, void* workspace,
                    size_t ws_bytes, hipStream_t stream);

/* MoE sub-block on the residual stream (the policy's mixture-of-experts
 * feed-forward, Sec. 4): h, out [n_tokens, H] fp32 (may alias).
 *  hn = RMSNorm(h; g2); logits = hn . w_r^T + b_r (fp32); S = the top_k
 *  experts by logit (ties to the lower index); w_e = softmax over S;
 *  out = h + sum_{e in S} w_e * (SwiGLU(hn . w_gu[e]^T + b_gu[e]) . w_d[e]^T + b_d[e]).
 *  topk_idx [n_tokens, k] int32 and topk_w [n_tokens, k] fp32 (device,
 *  nullable) receive the selection in descending logit order.
 *  force_idx (device, nullable, [n_tokens, k]): use these experts instead of
 *  the router's choice (weights still softmax of their logits).
 *  MCPU_EXPERT_MXFP4_NATIVE: the experts read hn (stored bf16) and the SwiGLU
 *  activations (stored bf16) as MXFP8 (OCP MX v1.0): per row, blocks of 32
 *  along the reduction share the E8M0 scale 2^(floor(log2 max|v|) - 8), and
 *  each element is v / scale rounded to nearest-even FP8 E4M3, saturating at
 *  448; products on the scaled matrix cores, fp32 accumulation (hidden and
 *  ffn_dim multiples of 64, else MCPU_EUNSUPPORTED; the weights come from
 *  w_gu_packed / w_d_packed). */
size_t moe_forward_workspace_size(const mcpu_layer_cfg* cfg, int32_t max_tokens);
int moe_forward(const mcpu_layer_cfg* cfg, const mcpu_layer_weights* w, int32_t n_tokens,
                const float* h, float* out, int32_t* topk_idx, float* topk_w,
                const int32_t* force_idx, void* workspace, size_t ws_bytes, hipStream_t stream);

/* Optional copies of intermediates of decode_layer (each nullable):
 *  q [T, Hq, d] layer dtype (after rotation), o [T, Hq * d] layer dtype
 *  (attention output), h1 [T, H] fp32 (residual after attention), logits
 *  [T, E] fp32 (router logits the top-k selection is made on). */
typedef struct mcpu_taps {
  void* q;
  void* o;
  float* h1;
  float* logits;
} mcpu_taps;

/* One decoder-layer step for a batch of sequences: the unit of the Run
 * stage's generation, which dominates rollout time (Sec. 3.2) and whose
 * throughput Sec. 4.2 measures in tokens/s:
 *  xn = RMSNorm(x_in; g1); [q|k|v] = xn . w_qkv^T + b_qkv; q, k rotated at
 *  their positions; k, v appended to the cache; o = paged_attention(q);
 *  h1 = x_in + o . w_o^T + b_o; x_out = moe_forward(h1).
 *  x_in, x_out [T, H] fp32 (must not alias); T = batch, or host_cu_q[batch].
 *  Arrays as in kv_pages_append / paged_attention / moe_forward. */
size_t decode_layer_workspace_size(const mcpu_layer_cfg* cfg, int32_t max_batch,
                                   int32_t max_tokens);
int decode_layer(const mcpu_layer_cfg* cfg, const mcpu_layer_weights* w, mcpu_kv_pool* pool,
                 int32_t batch, const int32_t* page_table, int32_t max_pages,
                 const int32_t* seq_lens, const int32_t* cu_q, const int32_t* host_seq_lens,
                 const int32_t* host_cu_q, const float* x_in, float* x_out, int32_t* topk_idx,
                 float* topk_w, const mcpu_taps* taps, void* workspace, size_t ws_bytes,
                 hipStream_t stream);

/* decode_layer for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * step, arguments and results as decode_layer, but its workspace is a static
 * device array inside the library (128 MiB per GPU, held until the process
 * ends) instead of a caller buffer. It calls
 * no allocating routine. A step whose decode_layer_workspace_size exceeds
 * that returns MCPU_ENOMEM and launches nothing (gpt-oss-20b shapes: up to
 * about 480 decode tokens). Every call on a GPU shares that GPU's array:
 * calls that overlap on one GPU (two streams, two threads) race and must be
 * serialised by the caller. device_errors (device int32, nullable) receives
 * the step's device error bits (MCPU_DEVERR_*), which are then cleared, so
 * each call reports only its own. */
int decode_layer_noalloc(const mcpu_layer_cfg* cfg, const mcpu_layer_weights* w, mcpu_kv_pool* pool,
                         int32_t batch, const int32_t* page_table, int32_t max_pages, const int32_t* seq_lens,
                         const int32_t* cu_q, const int32_t* host_seq_lens, const int32_t* host_cu_q,
                         const float* x_in, float* x_out, int32_t* topk_idx, float* topk_w, const mcpu_taps* taps,
                         int32_t* device_errors, hipStream_t stream);

/* ---- Generation around the layer stack --------------------------------- */
/* The Run stage generates each trajectory's next tokens at the rollout
 * temperature (0.7 in the paper's training details) and, for the GRPO update,
 * scores whole trajectories under the policy (Sec. 3.2 on the rollout
 * pipeline; Sec. 4 and its training-details appendix). These calls supply the
 * two ends of the stack for that: token embedding in front of it, the final
 * RMSNorm, the vocabulary projection and sampling behind it. */

/* Vocabulary head (host struct; device pointers owned by the caller).
 *  hidden H (multiple of 64), vocab V (multiple of 16), V * H * 2 < 2^31.
 *  g_final [H] fp32 RMSNorm gain; w_lm [V, H] bf16 row-major (the unembedding,
 *  no bias); w_lm_packed: optional (NULL) streaming-order copy of w_lm
 *  (mcpu_pack_weights with n_groups 1), read by few-row batches. */
typedef struct mcpu_lm_head {
  int32_t hidden, vocab;
  float rms_eps;
  const float* g_final;
  const void* w_lm;
  const void* w_lm_packed;
} mcpu_lm_head;

/* Next-token sampling and log-probabilities for n_tokens rows.
 *  x [*, H] fp32 residual rows (the stack's output); row t of the head reads
 *  x[x_rows[t]] (x_rows: device int32 [T], e.g. each sequence's last new
 *  token; the caller keeps them in range), or x[t] when x_rows is NULL.
 *  xn = RMSNorm(x; g_final) stored as bf16; logits l = xn . w_lm^T (fp32
 *  accumulation); s = l / temperature.
 *  temperature > 0: the sampled token is argmax_v (s_v + g_v) (the Gumbel-max
 *    form of drawing from softmax(s)), g_v = -log(-log u_v), u_v = ((w >> 9) +
 *    1/2) / 2^23 with w word v % 4 of Philox4x32-10 (key = seed low, high
 *    32 bits) at counter (v / 4, positions[t], seq_ids[t], 0x4C4D5330); so a
 *    row's draw depends only on (seed, sequence id, position), never on the
 *    batch it is in. Equal perturbed scores go to the lower id.
 *  temperature <= 0: greedy, argmax_v l_v (lower id on ties); s = l.
 *  Outputs (device, [T], each nullable): tokens_out the chosen id,
 *  logprob_out its log-probability s_tok - logsumexp(s), lse_out logsumexp(s),
 *  target_logprob_out s_target - logsumexp(s) for targets[t] (device [T],
 *  nullable; ids in [0, V), else the value is -inf).
 *  seq_ids / positions: device int32 [T], required when sampling (temperature
 *  > 0 with tokens_out or logprob_out requested); without those outputs no
 *  draws are made (scoring targets at a temperature).
 *  workspace >= lm_head_workspace_size(H, V, T) bytes (first 256 bytes: the
 *  error word, as for decode_layer). Host-detected errors launch nothing. */
size_t lm_head_workspace_size(int32_t hidden, int32_t vocab, int32_t max_tokens);
int lm_head_sample(const mcpu_lm_head* lm, int32_t n_tokens, const float* x, const int32_t* x_rows,
                   float temperature, uint64_t seed,
                   const int32_t* seq_ids, const int32_t* positions, const int32_t* targets, int32_t* tokens_out,
                   float* logprob_out, float* target_logprob_out, float* lse_out, void* workspace,
                   size_t ws_bytes, hipStream_t stream);

/* MXFP8 quantization of bf16 rows (OCP Microscaling Formats v1.0; the
 * policy's experts are MXFP4, Sec. 4), the activation format of the native
 * MXFP4 experts (see moe_forward): in [rows, cols] bf16 (16-byte aligned,
 * cols a multiple of 32) -> codes [rows, cols] FP8 E4M3 (16-byte aligned) and
 * scales [rows, cols / 32] E8M0; an all-zero block gets scale byte 0.
 * Asynchronous on stream. */
int mcpu_mxfp8_quantize(const void* in, int64_t rows, int32_t cols, uint8_t* codes, uint8_t* scales,
                        hipStream_t stream);

/* Token embedding: x_out[t] = table[tokens[t]] widened to fp32.
 *  table [vocab, hidden] bf16 (16-byte aligned), tokens device int32 [T],
 *  x_out [T, hidden] fp32 (16-byte aligned), hidden a multiple of 8. An id
 *  outside [0, vocab) writes a zero row and sets MCPU_DEVERR_TOKEN in the
 *  workspace's error word (workspace >= 256 bytes). */
int embed_tokens(const void* table, int32_t vocab, int32_t hidden, int32_t n_tokens, const int32_t* tokens,
                 float* x_out, void* workspace, size_t ws_bytes, hipStream_t stream);

/* Kernel timing, a profiling aid for the throughput measurements of the
 * generation step (Sec. 4.2). mcpu_timing_start(kernel, n) arms the
 * library to record a HIP event pair on the launching stream around each of
 * the next n launches of that kernel (n = 0 disarms it); mcpu_timing_read
 * waits for the recorded events and writes up to n durations in milliseconds
 * to host array ms, setting *n_recorded. Process-wide state: not thread-safe,
 * and recording adds two event records per timed launch. */
enum {
  MCPU_KERNEL_ATTN_PLAN = 0,   /* attention plan; in decode_layer also RMSNorm_1 (one launch) */
  MCPU_KERNEL_RMSNORM = 1,     /* not recorded: decode_layer runs RMSNorm_1 in the plan's launch */
  MCPU_KERNEL_QKV = 2,         /* QKV projection + RoPE + KV append */
  MCPU_KERNEL_ATTN_SPLIT = 3,  /* paged attention partials */
  MCPU_KERNEL_ATTN_COMBINE = 4,
  MCPU_KERNEL_OPROJ = 5,
  MCPU_KERNEL_ROUTER = 6,
  MCPU_KERNEL_PERMUTE = 7,
  MCPU_KERNEL_EXPERT_GU = 8,   /* expert gate/up GEMM + SwiGLU */
  MCPU_KERNEL_EXPERT_DOWN = 9,
  MCPU_KERNEL_MOE_COMBINE = 10,
  MCPU_KERNEL_KV_APPEND = 11,
  MCPU_KERNEL_ATTN_PREFILL = 12, /* chunked-prefill attention */
  MCPU_KERNEL_LM_HEAD = 13,      /* vocabulary projection + sampling summaries */
  MCPU_KERNEL_COUNT = 14
};
int mcpu_timing_start(int kernel, int n);
int mcpu_timing_read(int kernel, float* ms, int n, int* n_recorded);

/* Error reporting of every entry point above (not from the paper).
 * Synchronise the stream, read the workspace's device error word, clear it.
 * Returns MCPU_OK, MCPU_EDEVICE (bits in *bits if non-NULL) or MCPU_EHIP. */
int mcpu_check_device_errors(void* workspace, hipStream_t stream, int32_t* bits);

#ifdef __cplusplus
}
#endif
#endif /* MCPU_H */
