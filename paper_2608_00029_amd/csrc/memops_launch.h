// Host-side launchers of the memory-bound operators (internal; the public
// interface is the cattn_layernorm_*, cattn_gelu_* and cattn_sce_* entry
// points in cattn.h).  Arguments are validated by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cattn {

constexpr int kLnMaxC = 4096;  // widest LayerNorm row kept in registers (16 float4 per lane)

// Work groups of the LayerNorm backward's first kernel; each leaves one
// partial row of (dgamma, dbeta) in the workspace.
constexpr int ln_bwd_groups(int rows) { return rows <= 0 ? 0 : (rows + 15) / 16 < 512 ? (rows + 15) / 16 : 512; }

hipError_t launch_layernorm_fwd(const float* x, const float* gamma, const float* beta, float* y, float* mean,
                                float* rstd, int rows, int C, float eps, hipStream_t st);
hipError_t launch_layernorm_bwd(const float* x, const float* gamma, const float* mean, const float* rstd,
                                const float* dy, float* dx, float* dgamma, float* dbeta, float* part, int rows, int C,
                                hipStream_t st);
hipError_t launch_gelu(const float* x, const float* dy, float* out, int64_t n, bool backward, hipStream_t st);
hipError_t launch_sce_fwd(const float* z, const int* targets, float* lse, float* row_loss, int rows, int V,
                          hipStream_t st);
hipError_t launch_sce_bwd(const float* z, const int* targets, const float* lse, float scale, float* dz, int rows,
                          int V, hipStream_t st);
// loss[0] = (1/M) sum_i v[i], summed in a fixed order by one work group.
hipError_t launch_row_mean(const float* v, float* loss, int M, hipStream_t st);

}  // namespace cattn
