// Internal launch interface of the token-embedding and vocabulary-head
// kernels (lm_head.hip). Not part of the public ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace mcpu {

struct EmbedArgs {
  const void* table;      // [vocab][hidden] bf16
  const int32_t* tokens;  // [n_tokens]
  int vocab, hidden, n_tokens;
  float* x;               // [n_tokens][hidden] fp32
  int32_t* err;
};
hipError_t launch_embed(const EmbedArgs& p, hipStream_t s);

struct FinalNorm {
  const float* x;  // [*][hidden] fp32 residual stream
  const int32_t* rows;  // [n_tokens] rows of x to normalise, or nullptr (row t)
  const float* g;  // [hidden]
  int n_tokens, hidden;
  float eps;
  void* out;           // [n_tokens][hidden] bf16
  int32_t* group_off;  // [2] out: {0, n_tokens}
};
hipError_t launch_final_norm(const FinalNorm& p, hipStream_t s);

struct LmReduce {
  const LogitSlot* slots;  // [n_rows][n_slots]
  int n_rows, n_slots;
  int32_t* tokens;         // [n_rows] sampled (or greedy) column, nullable
  float* logprob;          // [n_rows] its log-probability under softmax(s), nullable
  float* lse;              // [n_rows] log-sum-exp of s, nullable
  float* target_logprob;   // [n_rows] the target column's log-probability, nullable
};
hipError_t launch_lm_reduce(const LmReduce& p, hipStream_t s);

}  // namespace mcpu
