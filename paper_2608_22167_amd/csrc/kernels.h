// Internal launch interface between the host library (mcpu.cpp) and the
// gfx950 kernels. Not part of the public ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mcpu {

// ---- attention -----------------------------------------------------------

// One split of a token's visible pages: token t of sequence b at position p,
// keys from lo, pages pg0 .. pg1 - 1 (logical page indices).
struct SplitDesc {
  int32_t t, b, p, lo, pg0, pg1, pad0, pad1;
};

struct RmsNorm {
  const float* x;  // [T][H]
  const float* g;
  int n_tokens, hidden;
  float eps;
  void* out;       // [T][H] layer dtype
};

struct AttnPlan {
  const int32_t* seq_lens;  // [batch]
  const int32_t* cu_q;      // [batch+1] or nullptr (one token per sequence)
  int batch, n_tokens, window, pps;
  int host_total_splits;    // what the host planned; checked on the device
  // sequences adding prefill_min_q or more tokens go to the prefill kernel in
  // blocks of prefill_qb tokens; their tokens get no splits
  int prefill_min_q, prefill_qb, host_total_blocks;
  int32_t* tok_seq;         // [n_tokens] out
  int32_t* tok_pos;         // [n_tokens] out
  int32_t* split_start;     // [n_tokens + 1] out
  SplitDesc* split_desc;    // [host_total_splits] out
  int32_t* blk_start;       // [batch + 1] out: first prefill block of each sequence
  int32_t* err;
  int32_t* zero;            // [n_zero] words cleared for the layer's later kernels
  int n_zero;
  // optional RMSNorm riding on the same launch (the layer's first norm, which
  // does not depend on the plan): workgroups 1.. normalise four rows each
  RmsNorm norm;             // rows and output of the norm
  int norm_dtype;           // -1: no norm; else the layer dtype of its output
};

// Chunked prefill: the new tokens of a sequence attend causally to its pages
// (the cached keys and the chunk's own, already appended).
struct AttnPrefill {
  const void* q;  // [T][Hq][D]
  const void* k_pool;
  const void* v_pool;
  const int32_t* page_table;
  int max_pages, n_pages;
  const int32_t* seq_lens;
  const int32_t* cu_q;
  const int32_t* blk_start;
  int batch, n_tokens, n_blocks, hq, hkv, window;
  float scale_log2;     // log2(e) / sqrt(D)
  const float* sinks;   // [Hq] or nullptr
  void* o;              // [T][Hq * D]
  int32_t* err;
};

struct AttnSplit {
  const void* q;  // [T][Hq][D]
  const void* k_pool;
  const void* v_pool;
  const int32_t* page_table;
  int max_pages, n_pages;
  const int32_t* tok_seq;
  const int32_t* tok_pos;
  const int32_t* split_start;
  const SplitDesc* split_desc;  // [n_splits], written by the plan kernel
  int batch, n_tokens, n_splits, hq, hkv, window, pps;
  float scale_log2;  // log2(e) / sqrt(D)
  float* part_ml;    // [S][Hq][2] running max (log2 units) and sum
  float* part_acc;   // [S][Hq][D]
  int32_t* err;
  // Set o (and sinks) to finish each token in the split pass (sliding-window
  // layers whose window fits WINDOW_MAX_PAGES pages, one split per token):
  // o [T][Hq * D] is written directly and no partials are stored.
  const float* sinks;
  void* o;
};
// pages a window of at most WINDOW_MAX_KEYS keys can touch
constexpr int WINDOW_MAX_KEYS = 128;
constexpr int WINDOW_MAX_PAGES = (WINDOW_MAX_KEYS + 14) / 16 + 1;

struct AttnCombine {
  const float* part_ml;
  const float* part_acc;
  const int32_t* split_start;
  const float* sinks;  // [Hq] or nullptr
  int n_tokens, n_splits, hq;
  void* o;             // [T][Hq * D]
};

hipError_t launch_attn_plan(const AttnPlan& p, hipStream_t s);
hipError_t launch_attn_split(int dtype, int head_dim, const AttnSplit& p, hipStream_t s);
hipError_t launch_attn_combine(int dtype, int head_dim, const AttnCombine& p, hipStream_t s);
// tokens per prefill workgroup for G = Hq / Hkv query heads per KV head (0 if unsupported)
int prefill_block_tokens(int group);
hipError_t launch_attn_prefill(int dtype, int head_dim, int group, const AttnPrefill& p, hipStream_t s);

// ---- KV append -------------------------------------------------------------

struct KvAppend {
  const void* k_new;  // [T][Hkv][D]
  const void* v_new;
  void* k_pool;
  void* v_pool;
  const int32_t* page_table;
  int max_pages, n_pages;
  const int32_t* seq_lens;  // [batch]
  const int32_t* cu_q;      // [batch+1] or nullptr
  int batch, n_tokens, hkv;
  int32_t* err;
};
hipError_t launch_kv_append(int dtype, int head_dim, const KvAppend& p, hipStream_t s);

// ---- weight-streaming GEMMs with fused epilogues -------------------------

enum EpiKind { EPI_QKV = 0, EPI_RESIDUAL = 1, EPI_SWIGLU = 2, EPI_BIAS = 3, EPI_LOGITS = 4, EPI_SWIGLU_MX = 5 };

// EPI_LOGITS: the output columns are vocabulary logits l (no bias). Nothing
// [rows, n] is written; per row and 64-column slot the epilogue leaves one
// LogitSlot record summarising s = l * inv_temp over the slot, from which
// lm_sample_reduce forms the row's sample and log-probabilities.
constexpr int LOGIT_SLOT = 64;
struct LogitSlot {
  float m;       // max of s over the slot
  float l;       // sum of exp(s - m) over the slot
  float pert;    // max of s + g (Gumbel noise g; g = 0 when greedy)
  float s_best;  // s at that column
  int32_t idx;   // that column (the lowest one on equal values)
  float s_tgt;   // s at the row's target column if it lies in the slot, else -inf
  float pad[2];
};

struct Gemm {
  // Y[row][n] = sum_k X[src(row)][k] * W[group][n][k], rows of a group are
  // group_off[g] .. group_off[g+1] (or 0 .. n_rows for one group).
  const void* w;
  const void* w_packed;     // bf16 weights in streaming order (mcpu_pack_weights) or nullptr
  const uint8_t* w_scales;  // MXFP4 block scales or nullptr
  int64_t w_group_stride;   // elements (or bytes for MXFP4 codes) per group
  int n, k;
  const void* x;            // [*, k] layer dtype (MXFP8 experts: E4M3 codes)
  const uint8_t* x_scales;  // MXFP8 activations: E8M0 scales [*, k / 32], else nullptr
  const int32_t* row_src;   // nullptr = identity
  const int32_t* group_off; // nullptr = one group of n_rows rows
  int n_rows, n_groups;
  int epi;
  // epilogue operands
  const float* bias;        // [groups][n]
  int64_t bias_group_stride;
  const float* residual;    // EPI_RESIDUAL: [rows][n] fp32
  void* out;                // EPI_RESIDUAL/EPI_BIAS: fp32 [rows][n]; EPI_SWIGLU: dtype [rows][n/2];
                            // EPI_SWIGLU_MX (scaled matrix cores only): the SwiGLU rows stored as
                            // bf16 and quantized to MXFP8, codes here and scales in out_scales,
                            // both in slice order over n_rows rows
  uint8_t* out_scales;
  float swiglu_alpha, swiglu_limit, swiglu_beta;
  // EPI_QKV
  int hq, hkv, head_dim;
  void* q_out;              // [rows][Hq][D]
  void* k_pool;
  void* v_pool;
  const int32_t* page_table;
  int max_pages, n_pages;
  const int32_t* tok_seq;
  const int32_t* tok_pos;
  const float* rope_cos;
  const float* rope_sin;
  int rope_max_pos;
  int32_t* err;
  int max_rows_per_group;   // upper bound used to pick the m-tiling
  int x_rows;               // rows of x when row_src gathers from it (0: n_rows)
  // reduction split over workgroups (one matrix, few rows): fp32 partial
  // tiles, slab_split_part_floats(n, k, n_rows) of them, and SPLIT_MAX_TILES
  // per-tile arrival counters that are zero on entry and left zero; nullptr
  // disables the split
  float* part;
  int32_t* part_cnt;
  int k_splits;             // set by the launcher
  // EPI_LOGITS: LogitSlot records [rows][ceil(n / LOGIT_SLOT)] in `out`;
  // s = l * inv_temp (greedy: inv_temp = 1 and no noise); the noise of row r,
  // column v comes from Philox4x32-10 keyed by seed at counter
  // (v / 4, row_pos[r], row_seq[r], LOGIT_RNG_TAG), word v % 4
  float inv_temp;
  int greedy;
  uint64_t seed;
  const int32_t* row_seq;
  const int32_t* row_pos;
  const int32_t* target;    // [rows] column whose s is recorded, or nullptr
};
constexpr uint32_t LOGIT_RNG_TAG = 0x4C4D5330u;  // counter word 3 of the sampling draws
hipError_t launch_gemm(int dtype, int expert_fmt, const Gemm& g, hipStream_t s);
// Scaled matrix-core products (gemm_mx.hip): MXFP8 activations (x, x_scales)
// times MXFP4 weights (w, w_scales), k a multiple of 64, n of 16, every
// operand in slice order so that a 64-wide reduction slice of 256 rows is one
// contiguous run:
//   x: E4M3 code (row r, column k) at ((k / 64) * x_rows + r) * 64 + k % 64;
//   x_scales: dword (k / 128) * x_rows + r, byte j = block 4 (k / 128) + j;
//   w: per group, E2M1 bytes of (row r, slice s) at (s * n + r) * 32 (low
//      nibble first), groups w_group_stride bytes apart (n * k / 2);
//   w_scales: per group, dword (k / 128) * n + r, groups n * ceil(k / 128) * 4
//      bytes apart.
// The rows of a group are x rows group_off[g] .. (row_src must be null).
__host__ __device__ constexpr int64_t mx_scale_bytes(int64_t rows, int k) { return (int64_t)((k + 127) / 128) * rows * 4; }
bool mx_gemm_applies(const Gemm& g);
hipError_t launch_gemm_mx(const Gemm& g, hipStream_t s);
// bf16 rows -> MXFP8 (E4M3 codes, E8M0 scales per 32 columns); input row r
// is quantized once and written to output rows row_dst[r * copies + c],
// c < copies (row r, one copy, when row_dst is null)
struct MxQuant {
  const void* in;  // [rows][cols] bf16
  const int32_t* row_dst;
  int copies;
  int64_t rows;      // input rows
  int64_t out_rows;  // rows of the output (the slice order's row count)
  int cols;
  uint8_t* codes;
  uint8_t* scales;
  int gemm_layout;  // 0: codes [out_rows][cols], scales [out_rows][cols / 32]; 1: the slice order above
};
// MXFP4 weights [groups][rows][cols / 2] + scales [groups][rows][cols / 32]
// -> the slice order above (codes, then scales at mx_packed_scales_offset)
struct MxPack {
  const uint8_t* codes;
  const uint8_t* scales;
  uint8_t* dst;
  int groups, rows, cols;
};
__host__ __device__ inline size_t mx_packed_codes_bytes(int groups, int rows, int cols) {
  return ((size_t)groups * rows * (cols / 2) + 255) & ~size_t(255);
}
__host__ __device__ inline size_t mx_packed_bytes(int groups, int rows, int cols) {
  return mx_packed_codes_bytes(groups, rows, cols) + (size_t)groups * mx_scale_bytes(rows, cols);
}
hipError_t launch_mx_pack(const MxPack& p, hipStream_t s);
hipError_t launch_mx_quant(const MxQuant& p, hipStream_t s);
// LDS-tiled path (gemm_tiled.hip): bf16, k a multiple of 64, at least
// TILED_MIN_TOTAL_ROWS rows in all and groups averaging TILED_MIN_ROWS rows;
// n_rows must then hold the total row count.
constexpr int TILED_MIN_ROWS = 16;
constexpr int TILED_MIN_TOTAL_ROWS = 128;
bool tiled_gemm_applies(int dtype, const Gemm& g);
hipError_t launch_gemm_tiled(int expert_fmt, const Gemm& g, hipStream_t s);
// Software-pipelined 256 x 256 tiles once groups average 256 rows and the
// launch has at least two tiles per compute unit (bf16 activations, k % 32 == 0).
bool pipe_gemm_applies(int dtype, const Gemm& g);
hipError_t launch_gemm_pipe(int expert_fmt, const Gemm& g, hipStream_t s);
// Weight slabs (gemm_slab.hip): grouped GEMMs with bf16 activations whose
// groups are too short for tiles (bf16 weights, under TILED_MIN_ROWS rows per
// group) or whose MXFP4 weights dominate the traffic (up to SLAB_MAX_ROWS_FP4
// rows per group on average); k a multiple of 64.
constexpr int SLAB_MAX_ROWS_FP4 = 96;
bool slab_gemm_applies(int dtype, int expert_fmt, const Gemm& g);
// One bf16 matrix against at most SPLIT_MAX_ROWS token rows: the slabs also
// split the reduction so that every compute unit streams weights; the last
// workgroup of a tile to finish sums the partial tiles in split order.
constexpr int SPLIT_MAX_ROWS = 64;
// Up to SLAB_WIDE_MAX_ROWS rows, a matrix of at least SLAB_WIDE_MIN_N output
// rows whose streaming-order copy is given also takes the slabs (unsplit: the
// launch already has a few hundred workgroups); narrower ones stay on tiles.
constexpr int SLAB_WIDE_MAX_ROWS = 512;
constexpr int SLAB_WIDE_MIN_N = 4096;
constexpr int SPLIT_MAX_TILES = 1024;
size_t slab_split_part_floats(int n, int k, int n_rows);  // 0: no split for this shape
// bf16 [groups][rows][cols] -> streaming order (the layout mcpu_pack_weights documents)
hipError_t launch_pack_weights(const void* src, void* dst, int groups, int rows, int cols, hipStream_t s);
hipError_t launch_gemm_slab(int expert_fmt, const Gemm& g, hipStream_t s);

// ---- norms, router, permutation, combine --------------------------------



struct Router {
  const float* h;      // [T][H] residual stream
  const float* g2;
  const void* w_r;     // [E][H] layer dtype
  const float* b_r;
  const int32_t* force_idx;
  int n_tokens, hidden, n_experts, top_k;
  float eps;
  void* hn_out;        // [T][H] layer dtype (expert GEMM input)
  int32_t* idx_out;    // [T][k]
  float* w_out;        // [T][k]
  float* logits_out;   // [T][E] fp32 router logits, or nullptr
  int32_t* err;
};
hipError_t launch_router(int dtype, const Router& p, hipStream_t s);

struct Permute {
  const int32_t* idx;  // [T][k]
  int n_tokens, top_k, n_experts;
  int32_t* group_off;  // [E+1]
  int32_t* pos_of;     // [T*k] sorted position of assignment t*k+s
  int32_t* src_tok;    // [T*k] token of sorted row
  int32_t* chunk_cnt;  // workspace: [ceil(T*k / PERM_CHUNK)][E] (batches above PERM_CHUNK)
  int32_t* err;
};
constexpr int PERM_CHUNK = 4096;  // assignments one permute workgroup ranks
hipError_t launch_permute(const Permute& p, hipStream_t s);

struct MoeCombine {
  const float* h;        // [T][H]
  const float* y;        // [T*k][H] sorted rows
  const float* w;        // [T][k]
  const int32_t* pos_of; // [T*k]
  int n_tokens, hidden, top_k;
  float* out;            // [T][H]
};
hipError_t launch_moe_combine(const MoeCombine& p, hipStream_t s);

}  // namespace mcpu
