// Host-side launcher of the fused loss-head kernels (internal; the public
// interface is cattn_lmhead_fwd in cattn.h).  Arguments are validated by the
// caller before the launcher runs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cattn {

struct LmheadArgs {
  const void* x;       // [M, K] bf16 hidden states
  const void* w;       // [N, K] bf16 projection (one row per vocabulary entry)
  const int* targets;  // [M] target ids, or nullptr
  float* logits;       // [M, N]
  float* lse;          // [M]
  float* row_loss;     // [M] (with targets)
  float* loss;         // [1] mean of row_loss (with targets; may be nullptr)
  float* part;         // workspace: [M][N / 64] pairs (maximum, sum of exponentials)
  int M, N, K;
};

hipError_t launch_lmhead(const LmheadArgs& a, hipStream_t st);

}  // namespace cattn
