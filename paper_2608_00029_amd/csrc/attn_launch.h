// Host-side launchers of the attention kernels (internal to the library; the
// public interface is the C ABI in cattn.h).  Arguments are validated by the
// caller before any launcher runs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn_sched.h"

namespace cattn {

struct FwdArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;
  int BH, S, D;
  float scale;
  bool causal;
  bool bf16;
  int H;           // heads (BH = B * H)
  bool seq_major;  // tensors stored [B, S, H, D] instead of [B, H, S, D]
};

struct BwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* o;
  const void* dout;
  const float* lse;
  void* dq;
  void* dk;
  void* dv;
  float* ws;  // workspace, per head: D = rowsum(dO * O) row, then -LSE/scale row, ws_rows(S) floats each
  int BH, S, D;
  float scale;
  bool causal;
  bool bf16;
  int H;           // heads (BH = B * H)
  bool seq_major;  // tensors stored [B, S, H, D] instead of [B, H, S, D]
};

hipError_t launch_fwd(const FwdArgs& a, hipStream_t st);
// phase: 0 = dq kernel then dkdv kernel, 1 = dq kernel only, 2 = dkdv kernel only
hipError_t launch_bwd(const BwdArgs& a, int phase, hipStream_t st);
// bf16 kernels (attn_bf16.hip); launch_fwd / launch_bwd route bf16 calls here
hipError_t launch_fwd_bf16(const FwdArgs& a, hipStream_t st);
hipError_t launch_bwd_bf16(const BwdArgs& a, int phase, hipStream_t st);
int64_t fwd_grid_blocks(int BH, int S);
int64_t bwd_grid_blocks(int BH, int S);

}  // namespace cattn
