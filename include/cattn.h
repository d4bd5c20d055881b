/*
 * cattn.h -- C ABI of the MI355X (gfx950) fused causal multi-head attention
 * library: forward (O, LSE) and backward (dQ, dK, dV).
 *
 * What is computed (Nova paper, section 4.2 "Attention as a First-Class
 * Lowering", and its backward paragraph): for every batch b and head h,
 *
 *     S   = scale * Q K^T                  scores, never written to memory
 *     S[i,j] excluded for j > i            when causal (the diagonal is kept)
 *     LSE = log(sum_j exp(S[i,j]))         per row, natural log
 *     P   = exp(S - LSE)
 *     O   = P V
 *
 * and, for an upstream gradient dO, with D = rowsum(dO * O):
 *
 *     dV = P^T dO,  dS = P * (dO V^T - D),  dQ = scale * dS K,  dK = scale * dS^T Q
 *
 * The forward streams key/value tiles through an online (running max / running
 * sum) base-2 softmax and keeps S and P in registers; the backward recomputes P
 * from LSE in two kernels -- one reduces over keys (dQ, and writes D), one over
 * queries (dK, dV) -- so the S x S matrix never reaches HBM in either direction
 * and no atomics are used (results are bitwise reproducible).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensors Q, K, V, O, dO, dQ, dK, dV are contiguous row-major [B, H, S, D]
 *    arrays of the element type `dtype` (CATTN_F32: IEEE float; CATTN_BF16:
 *    bfloat16 stored as 16-bit words).  LSE and the workspace are float arrays
 *    [B, H, S].  Queries and keys share the sequence length S.
 *  - Every pointer is a DEVICE pointer on the current HIP device, allocated and
 *    freed by the caller; the library allocates nothing and keeps no state
 *    between calls, so concurrent calls on different streams are safe as long
 *    as their output buffers do not overlap.
 *  - `stream` is a hipStream_t (NULL = the legacy default stream).  Calls only
 *    enqueue work and return; there is no host synchronisation.  Results are
 *    ready when the stream reaches that point.
 *  - Precision: CATTN_BF16 multiplies bf16 operands on the matrix cores with
 *    float accumulation; P and dS are rounded to bf16 (round to nearest even)
 *    before they enter a contraction; softmax statistics, LSE, D and all
 *    accumulators are float.  CATTN_F32 runs every contraction in float.
 *  - Supported shapes: D in {64, 128}; any S >= 1 with S * D <= 2^30 (a ragged
 *    last tile is handled in the kernels); B * H * ceil(S / 128) < 2^31.
 *    B, H or S equal to 0 is an empty problem: the call returns CATTN_OK and
 *    touches no memory (pointers may then be NULL).
 *  - `scale` (the softmax scale, e.g. 1/sqrt(D)) must lie in [1e-20, 1e6]:
 *    masked scores take the finite sentinel -1e30 (section 4.2), whose
 *    base-2 exponential underflows to exactly 0 after scaling only for
 *    scales well above 1e-28, and sentinel * scale must stay finite.
 *  - Alignment: Q, K, V, O, dO, dQ, dK, dV and the backward workspace start
 *    on a 16-byte boundary (the kernels move rows in 16-byte pieces); LSE on
 *    a 4-byte boundary.  Any misaligned pointer is CATTN_ERR_INVALID_ARG.
 *  - `causal` != 0 selects the causal mask; 0 attends to every key.
 *
 * Errors: argument errors are detected on the host before anything is
 * enqueued and leave every buffer untouched.  CATTN_ERR_HIP means a launch was
 * rejected by the HIP runtime; cattn_last_error_string() then names the HIP
 * error (per calling thread).
 */
#ifndef CATTN_H
#define CATTN_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CATTN_OK = 0,
  CATTN_ERR_INVALID_ARG = 1,  /* NULL or misaligned pointer, negative size, bad
                                 dtype, scale outside [1e-20, 1e6] or not finite,
                                 an output overlapping an input */
  CATTN_ERR_UNSUPPORTED = 2,  /* valid but not implemented: D not in {64, 128},
                                 S * D > 2^30, grid too large */
  CATTN_ERR_HIP = 3           /* the HIP runtime rejected a launch */
} cattn_status;

typedef enum {
  CATTN_F32 = 0,
  CATTN_BF16 = 1
} cattn_dtype;

/* Storage order of Q, K, V, O, dO, dQ, dK, dV (LSE and the workspace are
 * [B, H, S] in both).  CATTN_BHSD: contiguous [B, H, S, D], one head's S x D
 * matrix contiguous.  CATTN_BSHD: contiguous [B, S, H, D], the order a
 * query/key/value projection of a [B, S, H*D] activation produces before the
 * usual head-major repack.  Section 4.2 (building the online softmax) absorbs
 * that repack into how the attention operator indexes its operands instead of
 * running transpose kernels; here the kernels likewise read and write
 * [B, S, H, D] in place (rows of one head H*D elements apart). */
typedef enum {
  CATTN_BHSD = 0,
  CATTN_BSHD = 1
} cattn_layout;

/*
 * Forward pass (section 4.2: online softmax over key tiles, base-2 exponent
 * with the scale folded in, finite mask sentinel, causal loop clamping, LSE
 * saved per row).
 *
 *   q, k, v : in,  [B, H, S, D] `dtype`
 *   o       : out, [B, H, S, D] `dtype`   (must not overlap q, k, v or lse)
 *   lse     : out, [B, H, S] float, natural-log log-sum-exp of each row of
 *             scale * Q K^T over the visible keys (must not overlap q, k, v, o)
 */
cattn_status cattn_attn_fwd(const void* q, const void* k, const void* v,
                            void* o, float* lse,
                            int B, int H, int S, int D,
                            float scale, int causal, int dtype, void* stream);

/*
 * Backward pass (section 4.2, backward paragraph: two fused kernels that
 * recompute P from the saved LSE -- a dQ kernel reducing over keys, which
 * also forms D = rowsum(dO * O) in float from the given O, then a dK/dV kernel
 * reducing over queries; the loop bounds are clamped to the causal triangle).
 *
 *   q, k, v  : in, [B, H, S, D] `dtype` -- the forward's inputs
 *   o        : in, [B, H, S, D] `dtype` -- the forward's output
 *   dout     : in, [B, H, S, D] `dtype` -- upstream gradient dO
 *   lse      : in, [B, H, S] float      -- the forward's LSE (natural log)
 *   dq,dk,dv : out, [B, H, S, D] `dtype` (must not overlap any input, each
 *              other, or the workspace)
 *   workspace: scratch of at least cattn_bwd_workspace_bytes(B, H, S, D)
 *              bytes, 16-byte aligned.  Its prior contents are ignored.  On
 *              return it holds, as float [B*H][2][Sp] with Sp = S rounded up
 *              to a multiple of 32: row 0 of head bh is D = rowsum(dO * O),
 *              row 1 is -LSE / scale; entries S..Sp-1 of both rows are 0.
 *   scale, causal: the values the forward was called with.
 */
cattn_status cattn_attn_bwd(const void* q, const void* k, const void* v,
                            const void* o, const void* dout, const float* lse,
                            void* dq, void* dk, void* dv, float* workspace,
                            int B, int H, int S, int D,
                            float scale, int causal, int dtype, void* stream);

/*
 * cattn_attn_fwd and cattn_attn_bwd with an explicit storage order `layout`
 * (cattn_layout) of the [.., D] tensors; everything else -- arguments,
 * sizes, the LSE and workspace layouts, error behaviour -- is as above.  An
 * unknown layout is CATTN_ERR_INVALID_ARG.  cattn_attn_fwd(...) is
 * cattn_attn_fwd_ex(..., CATTN_BHSD, stream), and likewise for the backward.
 */
cattn_status cattn_attn_fwd_ex(const void* q, const void* k, const void* v,
                               void* o, float* lse,
                               int B, int H, int S, int D,
                               float scale, int causal, int dtype, int layout, void* stream);

cattn_status cattn_attn_bwd_ex(const void* q, const void* k, const void* v,
                               const void* o, const void* dout, const float* lse,
                               void* dq, void* dk, void* dv, float* workspace,
                               int B, int H, int S, int D,
                               float scale, int causal, int dtype, int layout, void* stream);

/*
 * The two phases of cattn_attn_bwd as separate calls, for callers that
 * schedule or time them individually.  cattn_attn_bwd(...) is exactly
 * cattn_attn_bwd_dq(...) followed by cattn_attn_bwd_dkdv(...) on one stream.
 *
 * cattn_attn_bwd_dq: the kernel that reduces over keys.  Writes dq, and D =
 *   rowsum(dO * O) and -LSE / scale into `workspace` in the layout given
 *   above.  Same argument rules as cattn_attn_bwd for the arguments it takes.
 * cattn_attn_bwd_dkdv: the kernel that reduces over queries.  Reads D and
 *   -LSE / scale from `workspace` (bf16: both; float32: D, LSE from `lse`),
 *   which must hold what cattn_attn_bwd_dq wrote for the same
 *   inputs (ordered before this call on `stream`, or otherwise complete).
 *   Writes dk and dv.
 */
cattn_status cattn_attn_bwd_dq(const void* q, const void* k, const void* v,
                               const void* o, const void* dout, const float* lse,
                               void* dq, float* workspace,
                               int B, int H, int S, int D,
                               float scale, int causal, int dtype, void* stream);

cattn_status cattn_attn_bwd_dkdv(const void* q, const void* k, const void* v,
                                 const void* dout, const float* lse, const float* workspace,
                                 void* dk, void* dv,
                                 int B, int H, int S, int D,
                                 float scale, int causal, int dtype, void* stream);

/*
 * cattn_attn_bwd_ex without the workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The workspace is a fixed 8 MiB array in
 * the library's device memory instead, one per GPU, held until the process
 * ends; this call allocates nothing (no hipMalloc, no allocating library
 * routine).  Results are bit for bit those of cattn_attn_bwd_ex.
 *
 *   Limit: 2 * B * H * Sp * 4 <= 8 MiB, Sp = S rounded up to a multiple of 32
 *   (e.g. B*H*Sp <= 2^20: GPT-2 small B8 H12 S1024 uses 3 MiB); larger
 *   problems return CATTN_ERR_UNSUPPORTED before anything is enqueued.
 *   Sharing: every call on one GPU uses that GPU's one array.  The backward
 *   writes all of the part it reads before reading it, so nothing needs to
 *   be cleared between calls, but calls that overlap in time on one GPU (on
 *   different streams or threads) race on the array: order them.  The first
 *   call on a device looks up the array's device address (a HIP runtime
 *   query, no allocation).
 *   Everything else -- arguments, layouts, error behaviour -- as for
 *   cattn_attn_bwd_ex.
 */
cattn_status cattn_attn_bwd_noalloc(const void* q, const void* k, const void* v,
                                    const void* o, const void* dout, const float* lse,
                                    void* dq, void* dk, void* dv,
                                    int B, int H, int S, int D,
                                    float scale, int causal, int dtype, int layout, void* stream);

/*
 * Fused language-model loss head, forward (section 4.1, case study "Fusing a
 * Reduction into a Contraction Epilogue"; the fused loss-head evaluation).
 * For hidden states X, the head's weight W (no bias) and target ids y:
 *
 *     Z    = X W^T                          logits
 *     LSE  = log sum_j exp(Z[i, j])         per row, natural log
 *     l_i  = LSE_i - Z[i, y_i]              softmax cross entropy of row i
 *     loss = (1/M) sum_i l_i
 *
 * The projection keeps each row's maximum and sum of exponentials over every
 * 64 consecutive vocabulary entries in its epilogue (partials [M, N/64]); a
 * merge then combines the partials with the rescale-by-maximum-difference rule
 * into LSE and l, and a fixed-order reduction forms the mean.  Deterministic.
 *
 *   x        : in,  [M, K] bfloat16, row-major
 *   w        : in,  [N, K] bfloat16, row-major (one row per vocabulary entry)
 *   targets  : in,  [M] int32 ids in [0, N), or NULL (then row_loss and loss
 *              are not written and may be NULL); an id outside [0, N) makes
 *              that row's loss (and the mean) NaN
 *   logits   : out, [M, N] float (float32 accumulation of bf16 products)
 *   lse      : out, [M] float
 *   row_loss : out, [M] float (with targets)
 *   loss     : out, [1] float, the mean of row_loss (with targets; may be NULL)
 *   workspace: scratch of at least cattn_lmhead_workspace_bytes(M, N, K) bytes,
 *              4-byte aligned; on return it holds the partials, float
 *              [M][N/64][2] (maximum, sum of exp(z - maximum)).
 * Supported: M a multiple of 128, N a multiple of 128, K a multiple of 64
 * (GPT-2's head: M = 8192 tokens, K = 768, N = 50304, the vocabulary padded
 * to a multiple of 128); otherwise CATTN_ERR_UNSUPPORTED.  M, N or K equal
 * to 0 is an empty problem (CATTN_OK, nothing touched).  Outputs must not
 * overlap inputs, each other or the workspace (CATTN_ERR_INVALID_ARG).
 */
cattn_status cattn_lmhead_fwd(const void* x, const void* w, const int* targets,
                              float* logits, float* lse, float* row_loss, float* loss,
                              float* workspace, int M, int N, int K, void* stream);

/* Bytes of workspace cattn_lmhead_fwd needs: M * (N / 64) * 2 * sizeof(float)
 * (0 for an empty or unsupported shape). */
size_t cattn_lmhead_workspace_bytes(int M, int N, int K);

/*
 * Memory-bound operators of the GPT-2 step around attention (section 6,
 * "Memory-Bound Operators": LayerNorm, GELU and fused softmax cross entropy,
 * forward and backward, on float32 tensors; GELU and cross entropy with their
 * backward ops are the ops of the section 3 language-model-head IR example).
 * Every tensor is a contiguous float32 (targets: int32) device array whose
 * address is a multiple of 16 bytes (CATTN_ERR_INVALID_ARG otherwise);
 * outputs must not overlap inputs or each other.  Asynchronous on `stream`,
 * deterministic (fixed-order reductions).  A size of 0 is an empty problem.
 *
 * LayerNorm over the last axis of x [rows, C] (biased variance, eps inside the
 * square root):
 *     mean_r = (1/C) sum_c x[r,c],  rstd_r = 1 / sqrt((1/C) sum_c (x[r,c] - mean_r)^2 + eps)
 *     y = (x - mean_r) * rstd_r * gamma + beta
 *   x, y: [rows, C]; gamma, beta: [C]; mean, rstd: out, [rows].
 *   Supported: C a multiple of 4 and at most 4096 (CATTN_ERR_UNSUPPORTED
 *   otherwise); eps finite and >= 0.
 */
cattn_status cattn_layernorm_fwd(const float* x, const float* gamma, const float* beta,
                                 float* y, float* mean, float* rstd,
                                 int rows, int C, float eps, void* stream);

/* LayerNorm backward for upstream dy [rows, C], with the forward's mean and
 * rstd, xhat = (x - mean) * rstd and g = dy * gamma:
 *     dx = rstd * (g - mean_c(g) - xhat * mean_c(g * xhat))     [rows, C]
 *     dgamma = sum_r dy * xhat,  dbeta = sum_r dy               [C]
 * workspace: at least cattn_layernorm_bwd_workspace_bytes(rows, C) bytes,
 * 16-byte aligned (per-group partial sums of dgamma and dbeta). */
cattn_status cattn_layernorm_bwd(const float* x, const float* gamma, const float* mean,
                                 const float* rstd, const float* dy, float* dx,
                                 float* dgamma, float* dbeta, float* workspace,
                                 int rows, int C, void* stream);
size_t cattn_layernorm_bwd_workspace_bytes(int rows, int C);

/* GELU, the tanh form (GPT-2's activation), elementwise over n floats:
 *     y = 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))
 * and its backward dx = dy * dy/dx(x).  Any n >= 0. */
cattn_status cattn_gelu_fwd(const float* x, float* y, long long n, void* stream);
cattn_status cattn_gelu_bwd(const float* x, const float* dy, float* dx, long long n, void* stream);

/* Softmax cross entropy of logits z [rows, V] against targets [rows] (int32):
 *     lse_r = log sum_j exp(z[r,j]),  row_loss_r = lse_r - z[r, t_r],
 *     loss = (1/rows) sum_r row_loss_r
 * One read of the logits.  targets may be NULL (only lse is written; row_loss
 * and loss may then be NULL); loss may be NULL.  A target outside [0, V)
 * makes that row's loss (and the mean) NaN.  Supported: V a multiple of 4. */
cattn_status cattn_sce_fwd(const float* logits, const int* targets, float* lse,
                           float* row_loss, float* loss, int rows, int V, void* stream);

/* Softmax cross-entropy backward, the softmax recomputed from the logits and
 * the forward's lse (no softmax tensor is stored):
 *     dlogits[r, j] = scale * (exp(z[r,j] - lse_r) - [j == t_r])
 * (scale = dloss / rows for the mean loss).  A row whose target is outside
 * [0, V) gets NaN everywhere.  Supported: V a multiple of 4; scale finite. */
cattn_status cattn_sce_bwd(const float* logits, const int* targets, const float* lse,
                           float scale, float* dlogits, int rows, int V, void* stream);

/* Bytes of workspace cattn_attn_bwd needs: 2 * B * H * Sp * sizeof(float),
 * Sp = S rounded up to a multiple of 32 (0 for an empty or invalid shape). */
size_t cattn_bwd_workspace_bytes(int B, int H, int S, int D);

/* Static, NUL-terminated name of a status code ("unknown status" otherwise). */
const char* cattn_status_string(int status);

/* Description of the last CATTN_ERR_HIP / argument error on the calling
 * thread ("" if none).  Valid until the next call on the same thread. */
const char* cattn_last_error_string(void);

#ifdef __cplusplus
}
#endif

#endif /* CATTN_H */
