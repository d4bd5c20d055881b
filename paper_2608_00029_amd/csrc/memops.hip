// Memory-bound neighbours of attention in the GPT-2 training step, for gfx950:
// LayerNorm, GELU (tanh form) and softmax cross entropy, forward and backward,
// on float32 tensors (paper section 6, "Memory-Bound Operators"; the GELU and
// cross-entropy ops and their backward ops of its section 3 IR example).
//
// All of them move far more bytes than they compute on, so the design is about
// HBM: every access is a 16-byte vector load or store by consecutive lanes
// (a wave moves 1 KB per instruction), each thread keeps several loads in
// flight before it uses any of them, outputs and the streams read once are
// accessed non-temporally (where that measured faster on the MI355X: all
// stores, the loads of the GELU backward and of both cross-entropy kernels), intermediate values stay in registers
// (the softmax of the cross-entropy backward is recomputed from the logits and
// the saved LSE, never stored), and reductions are done in a fixed order so
// that results are bitwise reproducible.
//
//  * GELU: a flat grid over float4s; y = x * sigmoid(2u), u = sqrt(2/pi)
//    (x + 0.044715 x^3), which is 0.5 x (1 + tanh u) rewritten so that one
//    exponential and one reciprocal give both y and its derivative.
//  * LayerNorm forward: one wave per row, the row held in registers (up to
//    4096 columns), two-pass mean / variance over the registers.
//  * LayerNorm backward: one wave per row for dx; every wave also sums
//    dy * xhat and dy over its rows for dgamma / dbeta, the four waves of a
//    group add theirs in a fixed order through LDS into one partial row of the
//    workspace, and a second kernel sums the partial rows column by column.
//  * Cross-entropy forward: one work group per row; each lane keeps a running
//    (maximum, sum of exponentials) in base 2 and the lanes are merged with
//    the rescale-by-maximum-difference rule.  Mean loss: one work group.
//  * Cross-entropy backward: a flat grid of 4096-entry row chunks;
//    dz = scale * (exp(z - lse) - onehot).
#include <math.h>

#include "attn_device.h"
#include "memops_launch.h"

namespace cattn {

namespace {

constexpr int kUnroll = 4;  // 16-byte accesses per thread in flight

// GELU constants: K1 = 2 sqrt(2/pi) log2(e), K2 = K1 * 0.044715, so that
// 2u log2(e) = x (K1 + K2 x^2); KD1 = 2 sqrt(2/pi), KD2 = 6 sqrt(2/pi) 0.044715.
constexpr double kSqrt2OverPi = 0.79788456080286535588;
constexpr float kGeluK1 = (float)(2.0 * kSqrt2OverPi * 1.44269504088896340736);
constexpr float kGeluK2 = (float)(2.0 * kSqrt2OverPi * 1.44269504088896340736 * 0.044715);
constexpr float kGeluD1 = (float)(2.0 * kSqrt2OverPi);
constexpr float kGeluD2 = (float)(6.0 * kSqrt2OverPi * 0.044715);

// r = 1 / (1 + exp(2u)); then 0.5 (1 + tanh u) = 1 - r.
__device__ __forceinline__ float gelu_r(float x) {
  const float e = exp2_hw(x * fmaf(kGeluK2, x * x, kGeluK1));
  return __builtin_amdgcn_rcpf(1.f + e);
}
__device__ __forceinline__ float gelu_y(float x) {
  return fmaf(-x, gelu_r(x), x);  // x (1 - r)
}
// dy/dx = s + 0.5 x (1 - tanh^2 u) du/dx = s (1 + x r (KD1 + KD2 x^2)), s = 1 - r
__device__ __forceinline__ float gelu_dydx(float x) {
  const float r = gelu_r(x), s = 1.f - r;
  return s * fmaf(x * r, fmaf(kGeluD2, x * x, kGeluD1), 1.f);
}

template <bool BWD>
__global__ __launch_bounds__(256) void gelu_kernel(const float* __restrict__ x, const float* __restrict__ dy,
                                                   float* __restrict__ out, int64_t n4, int64_t n) {
  const f32x4* x4 = (const f32x4*)x;
  const f32x4* g4 = (const f32x4*)dy;
  f32x4* o4 = (f32x4*)out;
  const int64_t step = (int64_t)gridDim.x * 256 * kUnroll;
  for (int64_t i0 = (int64_t)blockIdx.x * 256 * kUnroll + threadIdx.x; i0 < n4; i0 += step) {
    f32x4 v[kUnroll], g[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = i0 + u * 256;
      if (i < n4) {
        if constexpr (BWD) {
          v[u] = __builtin_nontemporal_load(&x4[i]);
          g[u] = __builtin_nontemporal_load(&g4[i]);
        } else {
          v[u] = x4[i];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = i0 + u * 256;
      if (i < n4) {
        f32x4 r;
#pragma unroll
        for (int e = 0; e < 4; ++e) r[e] = BWD ? g[u][e] * gelu_dydx(v[u][e]) : gelu_y(v[u][e]);
        __builtin_nontemporal_store(r, &o4[i]);
      }
    }
  }
  // the last n % 4 elements
  if (blockIdx.x == 0 && (int64_t)threadIdx.x < n - 4 * n4) {
    const int64_t i = 4 * n4 + threadIdx.x;
    out[i] = BWD ? dy[i] * gelu_dydx(x[i]) : gelu_y(x[i]);
  }
}

__device__ __forceinline__ float sum4(const f32x4& v) { return (v[0] + v[1]) + (v[2] + v[3]); }

// LayerNorm forward: wave `gw` of the grid normalises rows gw, gw + nw, ...
template <int NPL>
__global__ __launch_bounds__(256) void layernorm_fwd_kernel(const float* __restrict__ x,
                                                            const float* __restrict__ gamma,
                                                            const float* __restrict__ beta, float* __restrict__ y,
                                                            float* __restrict__ mean, float* __restrict__ rstd,
                                                            int rows, int C, float eps) {
  const int lane = threadIdx.x & 63;
  const int nw = gridDim.x * 4;
  const int C4 = C >> 2;
  const float fc = (float)C;
  f32x4 g[NPL], b[NPL];
#pragma unroll
  for (int k = 0; k < NPL; ++k) {
    const int c = lane + 64 * k;
    g[k] = c < C4 ? ((const f32x4*)gamma)[c] : f32x4{};
    b[k] = c < C4 ? ((const f32x4*)beta)[c] : f32x4{};
  }
  for (int row = blockIdx.x * 4 + (threadIdx.x >> 6); row < rows; row += nw) {
    const f32x4* xr = (const f32x4*)(x + (int64_t)row * C);
    f32x4 v[NPL];
#pragma unroll
    for (int k = 0; k < NPL; ++k) v[k] = lane + 64 * k < C4 ? xr[lane + 64 * k] : f32x4{};
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < NPL; ++k) s += sum4(v[k]);
    const float mu = wave_sum(s) / fc;  // a divide, so that a constant row has d = 0 exactly
    float q = 0.f;
#pragma unroll
    for (int k = 0; k < NPL; ++k)
      if (lane + 64 * k < C4) {
        const f32x4 d = v[k] - mu;
        q += sum4(d * d);
      }
    const float rs = 1.f / sqrtf(wave_sum(q) / fc + eps);
    f32x4* yr = (f32x4*)(y + (int64_t)row * C);
#pragma unroll
    for (int k = 0; k < NPL; ++k)
      if (lane + 64 * k < C4) __builtin_nontemporal_store((v[k] - mu) * rs * g[k] + b[k], &yr[lane + 64 * k]);
    if (lane == 0) {
      mean[row] = mu;
      rstd[row] = rs;
    }
  }
}

// LayerNorm backward, dx and per-group partial (dgamma, dbeta).  Group `wg`
// owns a contiguous block of rows; its wave w takes rows w, w + 4, ... of it.
template <int NPL>
__global__ __launch_bounds__(256) void layernorm_bwd_kernel(const float* __restrict__ x,
                                                            const float* __restrict__ gamma,
                                                            const float* __restrict__ mean,
                                                            const float* __restrict__ rstd,
                                                            const float* __restrict__ dy, float* __restrict__ dx,
                                                            float* __restrict__ part, int rows, int C) {
  __shared__ f32x4 red[2 * kLnMaxC / 4];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int C4 = C >> 2;
  const float fc = (float)C;
  const int per = (rows + gridDim.x - 1) / gridDim.x;
  const int r0 = blockIdx.x * per, r1 = min(rows, r0 + per);
  f32x4 g[NPL], dg[NPL], db[NPL];
#pragma unroll
  for (int k = 0; k < NPL; ++k) {
    const int c = lane + 64 * k;
    g[k] = c < C4 ? ((const f32x4*)gamma)[c] : f32x4{};
    dg[k] = f32x4{};
    db[k] = f32x4{};
  }
  for (int row = r0 + w; row < r1; row += 4) {
    const f32x4* xr = (const f32x4*)(x + (int64_t)row * C);
    const f32x4* gr = (const f32x4*)(dy + (int64_t)row * C);
    f32x4 v[NPL], d[NPL];
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
      const bool ok = lane + 64 * k < C4;
      v[k] = ok ? xr[lane + 64 * k] : f32x4{};
      d[k] = ok ? gr[lane + 64 * k] : f32x4{};
    }
    const float mu = mean[row], rs = rstd[row];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
      v[k] = (v[k] - mu) * rs;  // xhat (padding lanes: garbage times zero gamma / dy below)
      const f32x4 gg = d[k] * g[k];
      s1 += sum4(gg);
      s2 += sum4(gg * v[k]);
    }
    const float a = wave_sum(s1) / fc, c2 = wave_sum(s2) / fc;
    f32x4* dxr = (f32x4*)(dx + (int64_t)row * C);
#pragma unroll
    for (int k = 0; k < NPL; ++k)
      if (lane + 64 * k < C4) {
        __builtin_nontemporal_store(rs * (d[k] * g[k] - a - v[k] * c2), &dxr[lane + 64 * k]);
        dg[k] += d[k] * v[k];
        db[k] += d[k];
      }
  }
  // waves 0, 1, 2, 3 add their sums in that order
  for (int ww = 0; ww < 4; ++ww) {
    if (w == ww) {
#pragma unroll
      for (int k = 0; k < NPL; ++k) {
        const int c = lane + 64 * k;
        if (c < C4) {
          red[c] = ww ? red[c] + dg[k] : dg[k];
          red[C4 + c] = ww ? red[C4 + c] + db[k] : db[k];
        }
      }
    }
    __syncthreads();
  }
  f32x4* pr = (f32x4*)(part + (int64_t)blockIdx.x * 2 * C);
  for (int c = threadIdx.x; c < 2 * C4; c += 256) pr[c] = red[c];
}

// dgamma / dbeta: work group k sums column quads 8k .. 8k+7 of the 2C/4 quads
// of a partial row over all partial rows.  Lane l of wave w takes quad
// 8k + (l & 7) of partial rows j, j + 128, ... with j = 8w + (l >> 3), so a
// thread issues all its loads at once; the eight row streams of a wave are
// then added by a fixed butterfly, and wave 0 adds the 16 wave sums in order.
__global__ __launch_bounds__(1024) void layernorm_bwd_reduce_kernel(const float* __restrict__ part,
                                                                    float* __restrict__ dgamma,
                                                                    float* __restrict__ dbeta, int n_part, int C) {
  __shared__ f32x4 red[16][8];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int C4 = C >> 2, q = blockIdx.x * 8 + (lane & 7);
  const bool ok = q < 2 * C4;
  f32x4 s = f32x4{};
  if (ok) {
    const f32x4* p4 = (const f32x4*)part;
    for (int i = 8 * w + (lane >> 3); i < n_part; i += 128) s += p4[(int64_t)i * 2 * C4 + q];
  }
#pragma unroll
  for (int d = 8; d < 64; d <<= 1)
#pragma unroll
    for (int e = 0; e < 4; ++e) s[e] += __shfl_xor(s[e], d, 64);
  if (lane < 8) red[w][lane] = s;
  __syncthreads();
  if (w == 0 && lane < 8 && ok) {
    f32x4 t = red[0][lane];
    for (int i = 1; i < 16; ++i) t += red[i][lane];
    if (q < C4)
      ((f32x4*)dgamma)[q] = t;
    else
      ((f32x4*)dbeta)[q - C4] = t;
  }
}

// (m, s) <- merge of two base-2 softmax statistics (the fold is not the merge:
// the smaller side's sum is rescaled by 2^(its maximum - the larger maximum)).
__device__ __forceinline__ void merge_stats(float& m, float& s, float m2, float s2) {
  const float mm = fmaxf(m, m2);
  if (mm == -INFINITY) return;  // both sides empty
  s = s * exp2_hw(m - mm) + s2 * exp2_hw(m2 - mm);
  m = mm;
}

__global__ __launch_bounds__(256) void sce_fwd_kernel(const float* __restrict__ z, const int* __restrict__ targets,
                                                      float* __restrict__ lse, float* __restrict__ row_loss, int V) {
  __shared__ float red[2][4];
  const int row = blockIdx.x, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const f32x4* zr = (const f32x4*)(z + (int64_t)row * V);
  const int V4 = V >> 2;
  float m = -INFINITY, s = 0.f;  // over z * log2(e)
  for (int i0 = threadIdx.x; i0 < V4; i0 += 256 * kUnroll) {
    f32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
      if (i0 + u * 256 < V4) v[u] = __builtin_nontemporal_load(&zr[i0 + u * 256]);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
      if (i0 + u * 256 < V4) {
        const f32x4 a = v[u] * kLog2e;
        const float mx = fmaxf(fmaxf(a[0], a[1]), fmaxf(a[2], a[3]));
        if (mx > m) {  // move the offset (rare once the row's large values are seen)
          s *= exp2_hw(m - mx);
          m = mx;
        }
        s += (exp2_hw(a[0] - m) + exp2_hw(a[1] - m)) + (exp2_hw(a[2] - m) + exp2_hw(a[3] - m));
      }
  }
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) merge_stats(m, s, __shfl_xor(m, d, 64), __shfl_xor(s, d, 64));
  if (lane == 0) {
    red[0][w] = m;
    red[1][w] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    m = red[0][0];
    s = red[1][0];
    for (int i = 1; i < 4; ++i) merge_stats(m, s, red[0][i], red[1][i]);
    const float l = (m + log2f(s)) * kLn2;
    lse[row] = l;
    if (row_loss) {
      const int t = targets[row];  // an id outside [0, V) gives NaN rather than a stray read
      row_loss[row] = (t >= 0 && t < V) ? l - z[(int64_t)row * V + t] : __builtin_nanf("");
    }
  }
}

constexpr int kSceChunk4 = 256 * kUnroll;  // float4s of a row per cross-entropy backward work group

__global__ __launch_bounds__(256) void sce_bwd_kernel(const float* __restrict__ z, const int* __restrict__ targets,
                                                      const float* __restrict__ lse, float scale,
                                                      float* __restrict__ dz, int V, int n_chunks) {
  const int row = blockIdx.x / n_chunks, chunk = blockIdx.x - row * n_chunks;
  const int V4 = V >> 2;
  const int t = targets[row];
  const bool valid = t >= 0 && t < V;
  const float nl = -lse[row] * kLog2e;
  const f32x4* zr = (const f32x4*)(z + (int64_t)row * V);
  f32x4* dr = (f32x4*)(dz + (int64_t)row * V);
  const int i0 = chunk * kSceChunk4 + threadIdx.x;
  f32x4 v[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u)
    if (i0 + u * 256 < V4) v[u] = __builtin_nontemporal_load(&zr[i0 + u * 256]);
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int i = i0 + u * 256;
    if (i < V4) {
      f32x4 p;
#pragma unroll
      for (int e = 0; e < 4; ++e) p[e] = exp2_hw(fmaf(v[u][e], kLog2e, nl));
      if (!valid) {
        p = f32x4{} + __builtin_nanf("");
      } else if ((t >> 2) == i) {
        p[t & 3] -= 1.f;
      }
      __builtin_nontemporal_store(p * scale, &dr[i]);
    }
  }
}

// Mean of M floats: thread i sums v[i], v[i + 1024], ... (loads issued four at
// a time), then a fixed tree over the 1024 partial sums.
__global__ __launch_bounds__(1024) void row_mean_kernel(const float* __restrict__ v, float* __restrict__ loss, int M) {
  __shared__ float red[1024];
  float s = 0.f;
  for (int i0 = threadIdx.x; i0 < M; i0 += 4096) {
    float a[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) a[u] = i0 + 1024 * u < M ? v[i0 + 1024 * u] : 0.f;
#pragma unroll
    for (int u = 0; u < 4; ++u) s += a[u];
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int d = 512; d > 0; d >>= 1) {
    if ((int)threadIdx.x < d) red[threadIdx.x] += red[threadIdx.x + d];
    __syncthreads();
  }
  if (threadIdx.x == 0) loss[0] = red[0] / (float)M;
}

// float4s per lane of a LayerNorm row, rounded up to an instantiated width
int ln_npl(int C) {
  const int need = (C / 4 + 63) / 64;
  for (int n : {1, 2, 3, 4, 6, 8, 12, 16})
    if (n >= need) return n;
  return 0;
}

}  // namespace

hipError_t launch_layernorm_fwd(const float* x, const float* gamma, const float* beta, float* y, float* mean,
                                float* rstd, int rows, int C, float eps, hipStream_t st) {
  const unsigned grid = (unsigned)((rows + 3) / 4);
#define LN_FWD(N)                                                                                            \
  case N:                                                                                                    \
    hipLaunchKernelGGL(layernorm_fwd_kernel<N>, dim3(grid), dim3(256), 0, st, x, gamma, beta, y, mean, rstd, \
                       rows, C, eps);                                                                        \
    break;
  switch (ln_npl(C)) {
    LN_FWD(1) LN_FWD(2) LN_FWD(3) LN_FWD(4) LN_FWD(6) LN_FWD(8) LN_FWD(12) LN_FWD(16)
    default: return hipErrorInvalidValue;
  }
#undef LN_FWD
  return hipGetLastError();
}

hipError_t launch_layernorm_bwd(const float* x, const float* gamma, const float* mean, const float* rstd,
                                const float* dy, float* dx, float* dgamma, float* dbeta, float* part, int rows, int C,
                                hipStream_t st) {
  const int groups = ln_bwd_groups(rows);
#define LN_BWD(N)                                                                                                \
  case N:                                                                                                        \
    hipLaunchKernelGGL(layernorm_bwd_kernel<N>, dim3((unsigned)groups), dim3(256), 0, st, x, gamma, mean, rstd, \
                       dy, dx, part, rows, C);                                                                   \
    break;
  switch (ln_npl(C)) {
    LN_BWD(1) LN_BWD(2) LN_BWD(3) LN_BWD(4) LN_BWD(6) LN_BWD(8) LN_BWD(12) LN_BWD(16)
    default: return hipErrorInvalidValue;
  }
#undef LN_BWD
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(layernorm_bwd_reduce_kernel, dim3((unsigned)((2 * (C / 4) + 7) / 8)), dim3(1024), 0, st,
                     (const float*)part, dgamma, dbeta, groups, C);
  return hipGetLastError();
}

hipError_t launch_gelu(const float* x, const float* dy, float* out, int64_t n, bool backward, hipStream_t st) {
  const int64_t n4 = n / 4;
  const int64_t blocks = (n4 + 256 * kUnroll - 1) / (256 * kUnroll);
  const unsigned grid = (unsigned)(blocks < 1 ? 1 : blocks > (1 << 20) ? (1 << 20) : blocks);
  if (backward)
    hipLaunchKernelGGL(gelu_kernel<true>, dim3(grid), dim3(256), 0, st, x, dy, out, n4, n);
  else
    hipLaunchKernelGGL(gelu_kernel<false>, dim3(grid), dim3(256), 0, st, x, dy, out, n4, n);
  return hipGetLastError();
}

hipError_t launch_sce_fwd(const float* z, const int* targets, float* lse, float* row_loss, int rows, int V,
                          hipStream_t st) {
  hipLaunchKernelGGL(sce_fwd_kernel, dim3((unsigned)rows), dim3(256), 0, st, z, targets, lse,
                     targets ? row_loss : nullptr, V);
  return hipGetLastError();
}

hipError_t launch_sce_bwd(const float* z, const int* targets, const float* lse, float scale, float* dz, int rows,
                          int V, hipStream_t st) {
  const int n_chunks = (V / 4 + kSceChunk4 - 1) / kSceChunk4;
  hipLaunchKernelGGL(sce_bwd_kernel, dim3((unsigned)((int64_t)rows * n_chunks)), dim3(256), 0, st, z, targets, lse,
                     scale, dz, V, n_chunks);
  return hipGetLastError();
}

hipError_t launch_row_mean(const float* v, float* loss, int M, hipStream_t st) {
  hipLaunchKernelGGL(row_mean_kernel, dim3(1), dim3(1024), 0, st, v, loss, M);
  return hipGetLastError();
}

}  // namespace cattn
