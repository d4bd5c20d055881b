// Fused language-model loss head for gfx950 (paper section 4.1, case study
// "Fusing a Reduction into a Contraction Epilogue", and its fused loss-head
// evaluation): the vocabulary projection Z = X W^T keeps, in its epilogue and
// while the output tile is still in registers, each row's maximum and sum of
// exponentials over the tile's columns; two small passes then merge the
// per-tile partials into LSE and the per-row cross entropy, and reduce the
// per-row losses to their mean.
//
// Kernel 1 (projection + statistics).  A work group owns 128 vocabulary rows
// x 128 tokens of Z and streams K in chunks of 64 through a ring of LDS slots
// (W tile and X tile of a chunk, 32 KB).  Each of its four waves computes a
// 64 x 64 block as 2 x 2 transposed 32 x 32 matrix-core blocks, Z^T = W X^T,
// so that every lane holds one token and 16 vocabulary entries of each block:
// the row statistics are then in-lane over 32 entries plus one swap between
// the wave halves, exactly as the attention kernels' row softmax.  A wave's
// partial covers its 64 vocabulary entries: partials are [M, N/64] pairs
// (maximum, sum of exp(z - maximum)).  Logits are written as float [M, N].
//
// Work groups are dealt to the GPU's chiplets round-robin by index; a
// chiplet's groups walk its vocabulary tiles eight at a time with the token
// tiles inside, so the W and X tiles in flight on one chiplet fit its L2.
//
// Kernel 2 (merge): one wave per token row combines the row's N/64 partials
// with the rescale-by-maximum-difference rule (the merge is not the fold),
// giving LSE, and with a target id the row loss LSE - Z[row, target].
// Kernel 3 (mean): one work group sums the M row losses in a fixed order.
#include <math.h>

#include "attn_device.h"
#include "bf16_stream.h"
#include "lmhead_launch.h"

namespace cattn {

#ifndef CATTN_LMH_NB
#define CATTN_LMH_NB 2
#endif

constexpr int kLmhTileV = 128;  // vocabulary rows per work group
constexpr int kLmhTileM = 128;  // tokens per work group
constexpr int kLmhKC = 64;      // K chunk per ring slot
constexpr int kLmhPartW = 64;   // vocabulary entries per partial

// Work group -> (vocabulary tile, token tile), or false for a padding group.
__device__ __forceinline__ bool lmh_tile_of_block(int bid, int n_vt, int n_mt, int& vt, int& mt) {
  const int x = bid % kXcdGroup, l = bid / kXcdGroup;
  const int nv_x = (n_vt - x + kXcdGroup - 1) / kXcdGroup;  // vocabulary tiles of chiplet x: x, x + 8, ...
  if (x >= n_vt || l >= nv_x * n_mt) return false;
  const int vb = l / (8 * n_mt);
  const int g = min(8, nv_x - 8 * vb);
  const int rem = l - vb * 8 * n_mt;
  mt = rem / g;
  vt = x + kXcdGroup * (8 * vb + rem % g);
  return true;
}

template <int NB>
__global__ __launch_bounds__(256) void lmhead_logits_stats_kernel(const bf16* __restrict__ X,
                                                                  const bf16* __restrict__ W,
                                                                  float* __restrict__ Z, float* __restrict__ part,
                                                                  int M, int N, int K, int n_vt, int n_mt) {
  constexpr int TILE = 32 * kLmhKC * 2;  // one 32-row tile of a chunk: 4 KB
  constexpr int SLOT = 8 * TILE;         // W: 4 tiles (128 rows), X: 4 tiles (128 rows)
  constexpr int AH = NB - 1, PER_CHUNK = 8 * TileGeom<kLmhKC>::DMA_PER_TENSOR;
  constexpr int KS = kLmhKC / 16;
  __shared__ __attribute__((aligned(16))) char smem[NB * SLOT];

  int vt, mt;
  if (!lmh_tile_of_block(blockIdx.x, n_vt, n_mt, vt, mt)) return;  // uniform over the group
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int vw = w & 1, tw = w >> 1;  // this wave: vocabulary half, token half
  const int v0 = vt * kLmhTileV, m0 = mt * kLmhTileM;
  const int n_chunks = K / kLmhKC;

  TileCopy<kLmhKC> tc;
  tc.init(w, lane, K);
  auto dma = [&](int c, auto slc) {  // chunk c into ring slot slc
    char* b = smem + decltype(slc)::value * SLOT;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      tc.copy_full(W + c * kLmhKC, v0 + 32 * i, b + i * TILE);
      tc.copy_full(X + c * kLmhKC, m0 + 32 * i, b + (4 + i) * TILE);
    }
  };
  unroll<AH>([&](auto I) {
    if (decltype(I)::value < n_chunks) dma(decltype(I)::value, I);
  });
  wait_vm(0);
  __syncthreads();

  f32x16 acc[2][2];  // [vocabulary block][token block] of Z^T
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};

  for (int c0 = 0; c0 < n_chunks; c0 += NB) {
    unroll<NB>([&](auto slc) {
      constexpr int sl = decltype(slc)::value;
      const int c = c0 + sl;
      if (c >= n_chunks) return;
      if (c > 0) {  // chunk c landed (copies of later chunks may stay in flight); slot of c-1 free
        if (c + AH - 1 < n_chunks) {
          tile_barrier_c<(AH - 1) * PER_CHUNK>();
        } else {
          tile_barrier(0);
        }
      }
      if (c + AH < n_chunks) dma(c + AH, IC<(sl + AH) % NB>{});
      const char* b = smem + sl * SLOT;
      MB::frag wf[2][KS], xf[2][KS];
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          wf[blk][ks] = read_row_frag<bf16, kLmhKC>(b + (2 * vw + blk) * TILE, r, ks, h);
          xf[blk][ks] = read_row_frag<bf16, kLmhKC>(b + (4 + 2 * tw + blk) * TILE, r, ks, h);
        }
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int t = 0; t < 2; ++t) acc[a][t] = MB::run(wf[a][ks], xf[t][ks], acc[a][t]);
    });
  }

  // Epilogue.  acc[a][t][e]: Z[token m0 + 64 tw + 32 t + r][vocab v0 + 64 vw + 32 a + acc_row(e, h)]
  const int n_part = N / kLmhPartW;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int tok = m0 + 64 * tw + 32 * t + r;
    float mx = acc[0][t][0];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, acc[a][t][e]);
    mx = halves_max(mx);
    float s = 0.f;
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int e = 0; e < 16; ++e) s += exp2_hw((acc[a][t][e] - mx) * kLog2e);
    s = halves_sum(s);
    if (h == 0) {
      float* p = part + ((int64_t)tok * n_part + (v0 + 64 * vw) / kLmhPartW) * 2;
      p[0] = mx;
      p[1] = s;
    }
    float* zrow = Z + (int64_t)tok * N + v0 + 64 * vw;
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        store4<float>(zrow + 32 * a + 8 * g + 4 * h, acc[a][t][4 * g], acc[a][t][4 * g + 1], acc[a][t][4 * g + 2],
                      acc[a][t][4 * g + 3]);
  }
}

// Wave-wide maximum / sum over 64 lanes in a fixed pattern (every lane gets the result).
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) x = fmaxf(x, __shfl_xor(x, d, 64));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) x += __shfl_xor(x, d, 64);
  return x;
}

// One wave per row: merge the row's partials (maximum, sum) into LSE; with
// targets, the row's loss LSE - Z[row, target].
__global__ __launch_bounds__(256) void lmhead_merge_kernel(const float* __restrict__ part,
                                                           const float* __restrict__ Z,
                                                           const int* __restrict__ targets, float* __restrict__ lse,
                                                           float* __restrict__ row_loss, int M, int N) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const int n_part = N / kLmhPartW;
  const float2* p = (const float2*)(part + (int64_t)row * n_part * 2);
  float m = -INFINITY;
  for (int i = lane; i < n_part; i += 64) m = fmaxf(m, p[i].x);
  m = wave_max(m);
  float s = 0.f;
  for (int i = lane; i < n_part; i += 64) s += p[i].y * exp2_hw((p[i].x - m) * kLog2e);
  s = wave_sum(s);
  const float l = m + logf(s);
  if (lane == 0) {
    lse[row] = l;
    if (targets) {
      const int t = targets[row];  // an id outside [0, N) gives NaN rather than a stray read
      row_loss[row] = (t >= 0 && t < N) ? l - Z[(int64_t)row * N + t] : __builtin_nanf("");
    }
  }
}

// One work group: mean of the M row losses, summed in a fixed order.
__global__ __launch_bounds__(256) void lmhead_mean_kernel(const float* __restrict__ row_loss, float* __restrict__ loss,
                                                          int M) {
  __shared__ float red[256];
  float s = 0.f;
  for (int i = threadIdx.x; i < M; i += 256) s += row_loss[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int d = 128; d > 0; d >>= 1) {
    if ((int)threadIdx.x < d) red[threadIdx.x] += red[threadIdx.x + d];
    __syncthreads();
  }
  if (threadIdx.x == 0) loss[0] = red[0] / (float)M;
}

int64_t lmhead_grid_blocks(int M, int N) {
  const int n_vt = N / kLmhTileV, n_mt = M / kLmhTileM;
  const int nv_max = (n_vt + kXcdGroup - 1) / kXcdGroup;
  return (int64_t)kXcdGroup * nv_max * n_mt;
}

hipError_t launch_lmhead(const LmheadArgs& a, hipStream_t st) {
  const int n_vt = a.N / kLmhTileV, n_mt = a.M / kLmhTileM;
  hipLaunchKernelGGL((lmhead_logits_stats_kernel<CATTN_LMH_NB>), dim3((unsigned)lmhead_grid_blocks(a.M, a.N)),
                     dim3(256), 0, st, (const bf16*)a.x, (const bf16*)a.w, a.logits, a.part, a.M, a.N, a.K, n_vt,
                     n_mt);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lmhead_merge_kernel, dim3((unsigned)((a.M + 3) / 4)), dim3(256), 0, st, (const float*)a.part,
                     (const float*)a.logits, a.targets, a.lse, a.row_loss, a.M, a.N);
  e = hipGetLastError();
  if (e != hipSuccess || !a.targets || !a.loss) return e;
  hipLaunchKernelGGL(lmhead_mean_kernel, dim3(1), dim3(256), 0, st, (const float*)a.row_loss, a.loss, a.M);
  return hipGetLastError();
}

}  // namespace cattn
