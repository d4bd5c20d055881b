// C ABI entry points (declared and documented in include/cattn.h): argument
// validation on the host, then dispatch to the kernel launchers on the
// caller's stream.  Nothing is allocated and no state survives a call except
// the per-thread text of the last error.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "../../include/cattn.h"
#include "attn_launch.h"
#include "lmhead_launch.h"
#include "memops_launch.h"

extern "C" size_t cattn_bwd_workspace_bytes(int B, int H, int S, int D);

namespace {

thread_local char g_last_error[256] = "";

constexpr float kMinScale = 1e-20f, kMaxScale = 1e6f;

cattn_status fail(cattn_status st, const char* msg) {
  snprintf(g_last_error, sizeof(g_last_error), "%s", msg);
  return st;
}

struct Range {
  uintptr_t lo, hi;  // [lo, hi)
};

Range range_of(const void* p, size_t bytes) {
  const uintptr_t a = (uintptr_t)p;
  return Range{a, a + bytes};
}

bool overlap(Range a, Range b) { return a.lo < b.hi && b.lo < a.hi; }

// Shape checks shared by both entry points.  Returns CATTN_OK with *empty set
// when the problem is empty.
cattn_status check_shape(int B, int H, int S, int D, float scale, int dtype, bool* empty) {
  *empty = false;
  if (B < 0 || H < 0 || S < 0) return fail(CATTN_ERR_INVALID_ARG, "negative B, H or S");
  if (D <= 0) return fail(CATTN_ERR_INVALID_ARG, "D must be positive");
  if (dtype != CATTN_F32 && dtype != CATTN_BF16) return fail(CATTN_ERR_INVALID_ARG, "dtype must be CATTN_F32 or CATTN_BF16");
  if (!(scale > 0.f) || !isfinite(scale)) return fail(CATTN_ERR_INVALID_ARG, "scale must be finite and > 0");
  // Masked scores take a finite sentinel (-1e30) whose base-2 exponential must
  // underflow to exactly 0 after the scale is applied, and sentinel * scale
  // must stay finite: both hold with a wide margin inside this range.
  if (scale < kMinScale || scale > kMaxScale)
    return fail(CATTN_ERR_INVALID_ARG, "scale must lie in [1e-20, 1e6]");
  if (D != 64 && D != 128) return fail(CATTN_ERR_UNSUPPORTED, "head dimension D must be 64 or 128");
  if (B == 0 || H == 0 || S == 0) {
    *empty = true;
    return CATTN_OK;
  }
  if ((int64_t)S * D > (int64_t(1) << 30)) return fail(CATTN_ERR_UNSUPPORTED, "S * D exceeds 2^30");
  if ((int64_t)B * H > INT32_MAX) return fail(CATTN_ERR_UNSUPPORTED, "B * H exceeds 2^31 - 1");
  const int64_t BH = (int64_t)B * H;
  if (cattn::fwd_grid_blocks((int)BH, S) >= (int64_t(1) << 31) || cattn::bwd_grid_blocks((int)BH, S) >= (int64_t(1) << 31))
    return fail(CATTN_ERR_UNSUPPORTED, "grid too large");
  return CATTN_OK;
}

cattn_status hip_status(hipError_t e) {
  if (e == hipSuccess) return CATTN_OK;
  snprintf(g_last_error, sizeof(g_last_error), "HIP error %d: %s", (int)e, hipGetErrorString(e));
  return CATTN_ERR_HIP;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// Every output range against every input range and against the other outputs.
bool any_overlap(const Range* ins, int ni, const Range* outs, int no) {
  for (int i = 0; i < no; ++i) {
    for (int j = 0; j < ni; ++j)
      if (overlap(outs[i], ins[j])) return true;
    for (int j = i + 1; j < no; ++j)
      if (overlap(outs[i], outs[j])) return true;
  }
  return false;
}

}  // namespace

extern "C" {

cattn_status cattn_attn_fwd_ex(const void* q, const void* k, const void* v, void* o, float* lse, int B, int H, int S,
                               int D, float scale, int causal, int dtype, int layout, void* stream) {
  g_last_error[0] = '\0';
  if (layout != CATTN_BHSD && layout != CATTN_BSHD) return fail(CATTN_ERR_INVALID_ARG, "unknown layout");
  bool empty;
  cattn_status st = check_shape(B, H, S, D, scale, dtype, &empty);
  if (st != CATTN_OK || empty) return st;
  if (!q || !k || !v || !o || !lse) return fail(CATTN_ERR_INVALID_ARG, "NULL tensor pointer");
  // the kernels move rows in 16-byte pieces
  for (const void* p : {q, k, v, (const void*)o})
    if (!aligned16(p)) return fail(CATTN_ERR_INVALID_ARG, "q, k, v and o must be 16-byte aligned");
  if (((uintptr_t)lse & 3) != 0) return fail(CATTN_ERR_INVALID_ARG, "lse must be 4-byte aligned");
  const size_t esz = dtype == CATTN_BF16 ? 2 : 4;
  const size_t n = (size_t)B * H * S * D, nrow = (size_t)B * H * S;
  const Range rq = range_of(q, n * esz), rk = range_of(k, n * esz), rv = range_of(v, n * esz);
  const Range ro = range_of(o, n * esz), rl = range_of(lse, nrow * 4);
  for (Range out : {ro, rl})
    for (Range in : {rq, rk, rv})
      if (overlap(out, in)) return fail(CATTN_ERR_INVALID_ARG, "an output overlaps an input");
  if (overlap(ro, rl)) return fail(CATTN_ERR_INVALID_ARG, "o overlaps lse");

  cattn::FwdArgs a{q, k, v, o, lse, B * H, S, D, scale, causal != 0, dtype == CATTN_BF16, H, layout == CATTN_BSHD};
  (void)hipGetLastError();  // do not report an earlier, unrelated error as ours
  return hip_status(cattn::launch_fwd(a, (hipStream_t)stream));
}

cattn_status cattn_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int B, int H, int S,
                            int D, float scale, int causal, int dtype, void* stream) {
  return cattn_attn_fwd_ex(q, k, v, o, lse, B, H, S, D, scale, causal, dtype, CATTN_BHSD, stream);
}

}  // extern "C"

namespace {

// Validation + launch shared by the three backward entry points.  `ins` and
// `outs` list the buffers each phase reads and writes; the workspace is an
// output of phases 0 and 1 and an input of phase 2.
cattn_status bwd_common(const void* q, const void* k, const void* v, const void* o, const void* dout,
                        const float* lse, void* dq, void* dk, void* dv, float* workspace, int B, int H, int S,
                        int D, float scale, int causal, int dtype, int layout, void* stream, int phase) {
  g_last_error[0] = '\0';
  if (layout != CATTN_BHSD && layout != CATTN_BSHD) return fail(CATTN_ERR_INVALID_ARG, "unknown layout");
  bool empty;
  cattn_status st = check_shape(B, H, S, D, scale, dtype, &empty);
  if (st != CATTN_OK || empty) return st;
  const bool need_o = phase != 2, need_dq = phase != 2, need_dkdv = phase != 1;
  if (!q || !k || !v || !dout || !lse || !workspace || (need_o && !o) || (need_dq && !dq) ||
      (need_dkdv && (!dk || !dv)))
    return fail(CATTN_ERR_INVALID_ARG, "NULL tensor pointer");
  // the kernels move rows (and workspace rows) in 16-byte pieces
  for (const void* p : {q, k, v, dout, (const void*)workspace, need_o ? o : q, need_dq ? (const void*)dq : q,
                        need_dkdv ? (const void*)dk : q, need_dkdv ? (const void*)dv : q})
    if (!aligned16(p)) return fail(CATTN_ERR_INVALID_ARG, "tensors and the workspace must be 16-byte aligned");
  if (((uintptr_t)lse & 3) != 0) return fail(CATTN_ERR_INVALID_ARG, "lse must be 4-byte aligned");
  const size_t esz = dtype == CATTN_BF16 ? 2 : 4;
  const size_t n = (size_t)B * H * S * D, nrow = (size_t)B * H * S;
  const size_t wsb = cattn_bwd_workspace_bytes(B, H, S, D);
  Range ins[7], outs[4];
  int ni = 0, no = 0;
  ins[ni++] = range_of(q, n * esz);
  ins[ni++] = range_of(k, n * esz);
  ins[ni++] = range_of(v, n * esz);
  ins[ni++] = range_of(dout, n * esz);
  ins[ni++] = range_of(lse, nrow * 4);
  if (need_o) ins[ni++] = range_of(o, n * esz);
  if (phase == 2) ins[ni++] = range_of(workspace, wsb);
  else outs[no++] = range_of(workspace, wsb);
  if (need_dq) outs[no++] = range_of(dq, n * esz);
  if (need_dkdv) {
    outs[no++] = range_of(dk, n * esz);
    outs[no++] = range_of(dv, n * esz);
  }
  for (int i = 0; i < no; ++i)
    for (int j = 0; j < ni; ++j)
      if (overlap(outs[i], ins[j])) return fail(CATTN_ERR_INVALID_ARG, "an output or the workspace overlaps an input");
  for (int i = 0; i < no; ++i)
    for (int j = i + 1; j < no; ++j)
      if (overlap(outs[i], outs[j])) return fail(CATTN_ERR_INVALID_ARG, "outputs or workspace overlap each other");

  cattn::BwdArgs a{q, k, v, o, dout, lse, dq, dk, dv, workspace, B * H, S, D, scale, causal != 0,
                   dtype == CATTN_BF16, H, layout == CATTN_BSHD};
  (void)hipGetLastError();
  return hip_status(cattn::launch_bwd(a, phase, (hipStream_t)stream));
}

}  // namespace

extern "C" {

cattn_status cattn_attn_bwd(const void* q, const void* k, const void* v, const void* o, const void* dout,
                            const float* lse, void* dq, void* dk, void* dv, float* workspace, int B, int H, int S,
                            int D, float scale, int causal, int dtype, void* stream) {
  return bwd_common(q, k, v, o, dout, lse, dq, dk, dv, workspace, B, H, S, D, scale, causal, dtype, CATTN_BHSD,
                    stream, 0);
}

cattn_status cattn_attn_bwd_ex(const void* q, const void* k, const void* v, const void* o, const void* dout,
                               const float* lse, void* dq, void* dk, void* dv, float* workspace, int B, int H,
                               int S, int D, float scale, int causal, int dtype, int layout, void* stream) {
  return bwd_common(q, k, v, o, dout, lse, dq, dk, dv, workspace, B, H, S, D, scale, causal, dtype, layout, stream,
                    0);
}

cattn_status cattn_attn_bwd_dq(const void* q, const void* k, const void* v, const void* o, const void* dout,
                               const float* lse, void* dq, float* workspace, int B, int H, int S, int D,
                               float scale, int causal, int dtype, void* stream) {
  return bwd_common(q, k, v, o, dout, lse, dq, nullptr, nullptr, workspace, B, H, S, D, scale, causal, dtype,
                    CATTN_BHSD, stream, 1);
}

cattn_status cattn_attn_bwd_dkdv(const void* q, const void* k, const void* v, const void* dout, const float* lse,
                                 const float* workspace, void* dk, void* dv, int B, int H, int S, int D,
                                 float scale, int causal, int dtype, void* stream) {
  return bwd_common(q, k, v, nullptr, dout, lse, nullptr, dk, dv, const_cast<float*>(workspace), B, H, S, D,
                    scale, causal, dtype, CATTN_BHSD, stream, 2);
}

}  // extern "C"

namespace {

// Backward workspace of cattn_attn_bwd_noalloc: a fixed device array, one copy
// per GPU the library runs on, held until the process ends.  Host code never
// uses the array's name as an address: the device address of each GPU's copy
// comes from hipGetSymbolAddress, looked up once per device with that device
// current, and is what the kernels receive.
constexpr size_t kNoAllocWsBytes = size_t(8) << 20;
__device__ __align__(256) float scratch[kNoAllocWsBytes / sizeof(float)];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch`, or NULL after writing the error.
float* scratch_on_current_device(cattn_status* st) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    *st = hip_status(e);
    return nullptr;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    *st = fail(CATTN_ERR_UNSUPPORTED, "device index beyond the static scratch table");
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      *st = e != hipSuccess ? hip_status(e) : fail(CATTN_ERR_HIP, "no device address for the static scratch");
      return nullptr;
    }
    g_scratch_ptr[dev] = (float*)p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

cattn_status cattn_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o, const void* dout,
                                    const float* lse, void* dq, void* dk, void* dv, int B, int H, int S, int D,
                                    float scale, int causal, int dtype, int layout, void* stream) {
  g_last_error[0] = '\0';
  bool empty;
  cattn_status st = check_shape(B, H, S, D, scale, dtype, &empty);
  if (st != CATTN_OK || empty) return st;
  if (cattn_bwd_workspace_bytes(B, H, S, D) > kNoAllocWsBytes)
    return fail(CATTN_ERR_UNSUPPORTED, "the backward workspace this shape needs exceeds the 8 MiB static scratch "
                                       "(2 * B * H * ceil(S / 32) * 32 floats)");
  st = CATTN_OK;
  float* ws = scratch_on_current_device(&st);
  if (!ws) return st;
  return bwd_common(q, k, v, o, dout, lse, dq, dk, dv, ws, B, H, S, D, scale, causal, dtype, layout, stream, 0);
}

size_t cattn_lmhead_workspace_bytes(int M, int N, int K) {
  if (M <= 0 || N <= 0 || K <= 0 || M % 128 || N % 128 || K % 64) return 0;
  return (size_t)M * (size_t)(N / 64) * 2 * sizeof(float);
}

cattn_status cattn_lmhead_fwd(const void* x, const void* w, const int* targets, float* logits, float* lse,
                              float* row_loss, float* loss, float* workspace, int M, int N, int K, void* stream) {
  g_last_error[0] = '\0';
  if (M < 0 || N < 0 || K < 0) return fail(CATTN_ERR_INVALID_ARG, "negative M, N or K");
  if (M == 0 || N == 0 || K == 0) return CATTN_OK;
  if (M % 128 || N % 128 || K % 64) return fail(CATTN_ERR_UNSUPPORTED, "M and N must be multiples of 128, K of 64");
  if ((int64_t)M * N > (int64_t(1) << 40) || M > (1 << 24) || N > (1 << 23))
    return fail(CATTN_ERR_UNSUPPORTED, "problem too large");
  if (!x || !w || !logits || !lse || !workspace || (targets && !row_loss))
    return fail(CATTN_ERR_INVALID_ARG, "NULL tensor pointer");
  if (((uintptr_t)workspace & 3) != 0) return fail(CATTN_ERR_INVALID_ARG, "workspace must be 4-byte aligned");
  Range ins[3], outs[5];
  int ni = 0, no = 0;
  ins[ni++] = range_of(x, (size_t)M * K * 2);
  ins[ni++] = range_of(w, (size_t)N * K * 2);
  if (targets) ins[ni++] = range_of(targets, (size_t)M * 4);
  outs[no++] = range_of(logits, (size_t)M * N * 4);
  outs[no++] = range_of(lse, (size_t)M * 4);
  outs[no++] = range_of(workspace, cattn_lmhead_workspace_bytes(M, N, K));
  if (targets) outs[no++] = range_of(row_loss, (size_t)M * 4);
  if (targets && loss) outs[no++] = range_of(loss, 4);
  for (int i = 0; i < no; ++i)
    for (int j = 0; j < ni; ++j)
      if (overlap(outs[i], ins[j])) return fail(CATTN_ERR_INVALID_ARG, "an output or the workspace overlaps an input");
  for (int i = 0; i < no; ++i)
    for (int j = i + 1; j < no; ++j)
      if (overlap(outs[i], outs[j])) return fail(CATTN_ERR_INVALID_ARG, "outputs or workspace overlap each other");
  cattn::LmheadArgs a{x, w, targets, logits, lse, row_loss, targets ? loss : nullptr, workspace, M, N, K};
  (void)hipGetLastError();
  return hip_status(cattn::launch_lmhead(a, (hipStream_t)stream));
}

cattn_status cattn_layernorm_fwd(const float* x, const float* gamma, const float* beta, float* y, float* mean,
                                 float* rstd, int rows, int C, float eps, void* stream) {
  g_last_error[0] = '\0';
  if (rows < 0 || C < 0) return fail(CATTN_ERR_INVALID_ARG, "negative rows or C");
  if (!(eps >= 0.f) || !isfinite(eps)) return fail(CATTN_ERR_INVALID_ARG, "eps must be finite and >= 0");
  if (rows == 0 || C == 0) return CATTN_OK;
  if (C % 4 || C > cattn::kLnMaxC) return fail(CATTN_ERR_UNSUPPORTED, "C must be a multiple of 4 and at most 4096");
  if (!x || !gamma || !beta || !y || !mean || !rstd) return fail(CATTN_ERR_INVALID_ARG, "NULL tensor pointer");
  for (const void* p : {(const void*)x, (const void*)gamma, (const void*)beta, (const void*)y, (const void*)mean,
                        (const void*)rstd})
    if (!aligned16(p)) return fail(CATTN_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
  const size_t n = (size_t)rows * C * 4;
  const Range ins[3] = {range_of(x, n), range_of(gamma, (size_t)C * 4), range_of(beta, (size_t)C * 4)};
  const Range outs[3] = {range_of(y, n), range_of(mean, (size_t)rows * 4), range_of(rstd, (size_t)rows * 4)};
  if (any_overlap(ins, 3, outs, 3)) return fail(CATTN_ERR_INVALID_ARG, "outputs overlap inputs or each other");
  (void)hipGetLastError();
  return hip_status(cattn::launch_layernorm_fwd(x, gamma, beta, y, mean, rstd, rows, C, eps, (hipStream_t)stream));
}

size_t cattn_layernorm_bwd_workspace_bytes(int rows, int C) {
  if (rows <= 0 || C <= 0) return 0;
  return (size_t)cattn::ln_bwd_groups(rows) * 2 * (size_t)C * sizeof(float);
}

cattn_status cattn_layernorm_bwd(const float* x, const float* gamma, const float* mean, const float* rstd,
                                 const float* dy, float* dx, float* dgamma, float* dbeta, float* workspace, int rows,
                                 int C, void* stream) {
  g_last_error[0] = '\0';
  if (rows < 0 || C < 0) return fail(CATTN_ERR_INVALID_ARG, "negative rows or C");
  if (rows == 0 || C == 0) return CATTN_OK;
  if (C % 4 || C > cattn::kLnMaxC) return fail(CATTN_ERR_UNSUPPORTED, "C must be a multiple of 4 and at most 4096");
  if (!x || !gamma || !mean || !rstd || !dy || !dx || !dgamma || !dbeta || !workspace)
    return fail(CATTN_ERR_INVALID_ARG, "NULL tensor pointer");
  for (const void* p : {(const void*)x, (const void*)gamma, (const void*)mean, (const void*)rstd, (const void*)dy,
                        (const void*)dx, (const void*)dgamma, (const void*)dbeta, (const void*)workspace})
    if (!aligned16(p)) return fail(CATTN_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
  const size_t n = (size_t)rows * C * 4;
  const Range ins[5] = {range_of(x, n), range_of(gamma, (size_t)C * 4), range_of(mean, (size_t)rows * 4),
                        range_of(rstd, (size_t)rows * 4), range_of(dy, n)};
  const Range outs[4] = {range_of(dx, n), range_of(dgamma, (size_t)C * 4), range_of(dbeta, (size_t)C * 4),
                         range_of(workspace, cattn_layernorm_bwd_workspace_bytes(rows, C))};
  if (any_overlap(ins, 5, outs, 4)) return fail(CATTN_ERR_INVALID_ARG, "outputs overlap inputs or each other");
  (void)hipGetLastError();
  return hip_status(cattn::launch_layernorm_bwd(x, gamma, mean, rstd, dy, dx, dgamma, dbeta, workspace, rows, C,
                                                (hipStream_t)stream));
}

static cattn_status gelu_common(const float* x, const float* dy, float* out, long long n, bool bwd, void* stream) {
  g_last_error[0] = '\0';
  if (n < 0) return fail(CATTN_ERR_INVALID_ARG, "negative n");
  if (n == 0) return CATTN_OK;
  if (n > (1LL << 40)) return fail(CATTN_ERR_UNSUPPORTED, "n exceeds 2^40");
  if (!x || !out || (bwd && !dy)) return fail(CATTN_ERR_INVALID_ARG, "NULL tensor pointer");
  if (!aligned16(x) || !aligned16(out) || (bwd && !aligned16(dy)))
    return fail(CATTN_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
  const size_t b = (size_t)n * 4;
  const Range ins[2] = {range_of(x, b), range_of(dy, bwd ? b : 0)};
  const Range outs[1] = {range_of(out, b)};
  if (any_overlap(ins, bwd ? 2 : 1, outs, 1)) return fail(CATTN_ERR_INVALID_ARG, "output overlaps an input");
  (void)hipGetLastError();
  return hip_status(cattn::launch_gelu(x, dy, out, (int64_t)n, bwd, (hipStream_t)stream));
}

cattn_status cattn_gelu_fwd(const float* x, float* y, long long n, void* stream) {
  return gelu_common(x, nullptr, y, n, false, stream);
}

cattn_status cattn_gelu_bwd(const float* x, const float* dy, float* dx, long long n, void* stream) {
  return gelu_common(x, dy, dx, n, true, stream);
}

cattn_status cattn_sce_fwd(const float* logits, const int* targets, float* lse, float* row_loss, float* loss, int rows,
                           int V, void* stream) {
  g_last_error[0] = '\0';
  if (rows < 0 || V < 0) return fail(CATTN_ERR_INVALID_ARG, "negative rows or V");
  if (rows == 0 || V == 0) return CATTN_OK;
  if (V % 4) return fail(CATTN_ERR_UNSUPPORTED, "V must be a multiple of 4");
  if (!logits || !lse || (targets && !row_loss)) return fail(CATTN_ERR_INVALID_ARG, "NULL tensor pointer");
  if (!targets) row_loss = loss = nullptr;
  for (const void* p : {(const void*)logits, (const void*)targets, (const void*)lse, (const void*)row_loss,
                        (const void*)loss})
    if (!aligned16(p)) return fail(CATTN_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
  const Range ins[2] = {range_of(logits, (size_t)rows * V * 4), range_of(targets, targets ? (size_t)rows * 4 : 0)};
  const Range outs[3] = {range_of(lse, (size_t)rows * 4), range_of(row_loss, row_loss ? (size_t)rows * 4 : 0),
                         range_of(loss, loss ? 4 : 0)};
  if (any_overlap(ins, 2, outs, 3)) return fail(CATTN_ERR_INVALID_ARG, "outputs overlap inputs or each other");
  (void)hipGetLastError();
  hipError_t e = cattn::launch_sce_fwd(logits, targets, lse, row_loss, rows, V, (hipStream_t)stream);
  if (e == hipSuccess && loss) e = cattn::launch_row_mean(row_loss, loss, rows, (hipStream_t)stream);
  return hip_status(e);
}

cattn_status cattn_sce_bwd(const float* logits, const int* targets, const float* lse, float scale, float* dlogits,
                           int rows, int V, void* stream) {
  g_last_error[0] = '\0';
  if (rows < 0 || V < 0) return fail(CATTN_ERR_INVALID_ARG, "negative rows or V");
  if (!isfinite(scale)) return fail(CATTN_ERR_INVALID_ARG, "scale must be finite");
  if (rows == 0 || V == 0) return CATTN_OK;
  if (V % 4) return fail(CATTN_ERR_UNSUPPORTED, "V must be a multiple of 4");
  const int64_t chunks = ((int64_t)V / 4 + 1023) / 1024;
  if ((int64_t)rows * chunks >= (int64_t(1) << 31)) return fail(CATTN_ERR_UNSUPPORTED, "grid too large");
  if (!logits || !targets || !lse || !dlogits) return fail(CATTN_ERR_INVALID_ARG, "NULL tensor pointer");
  for (const void* p : {(const void*)logits, (const void*)targets, (const void*)lse, (const void*)dlogits})
    if (!aligned16(p)) return fail(CATTN_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
  const size_t n = (size_t)rows * V * 4;
  const Range ins[3] = {range_of(logits, n), range_of(targets, (size_t)rows * 4), range_of(lse, (size_t)rows * 4)};
  const Range outs[1] = {range_of(dlogits, n)};
  if (any_overlap(ins, 3, outs, 1)) return fail(CATTN_ERR_INVALID_ARG, "output overlaps an input");
  (void)hipGetLastError();
  return hip_status(cattn::launch_sce_bwd(logits, targets, lse, scale, dlogits, rows, V, (hipStream_t)stream));
}

size_t cattn_bwd_workspace_bytes(int B, int H, int S, int D) {
  if (B <= 0 || H <= 0 || S <= 0 || D <= 0) return 0;
  return 2 * (size_t)B * H * (size_t)cattn::ws_rows(S) * sizeof(float);
}

const char* cattn_status_string(int status) {
  switch (status) {
    case CATTN_OK: return "CATTN_OK";
    case CATTN_ERR_INVALID_ARG: return "CATTN_ERR_INVALID_ARG";
    case CATTN_ERR_UNSUPPORTED: return "CATTN_ERR_UNSUPPORTED";
    case CATTN_ERR_HIP: return "CATTN_ERR_HIP";
    default: return "unknown status";
  }
}

const char* cattn_last_error_string(void) { return g_last_error; }

}  // extern "C"
