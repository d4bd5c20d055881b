// Fused language-model loss head for gfx950 (paper section 4.1, case study
// "Fusing a Reduction into a Contraction Epilogue", and its fused loss-head
// evaluation): the vocabulary projection Z = X W^T keeps, in its epilogue and
// while the output tile is still in registers, each row's maximum and sum of
// exponentials over the tile's columns; two small passes then merge the
// per-tile partials into LSE and the per-row cross entropy, and reduce the
// per-row losses to their mean.
//
// Kernel 1 (projection + statistics).  A persistent grid of one work group
// per compute unit; each walks its chiplet's 256 x 256 output tiles (256
// vocabulary rows x 256 tokens of Z) and streams K in chunks of 64 through two
// LDS slots (W and X rows of a chunk, 64 KB each): the copy of chunk c + 1 --
// or of the next tile's first chunk -- runs while chunk c computes, so the
// next tile's first copy also overlaps this tile's epilogue.  Each of the
// eight waves computes a 128 x 64 block as 4 x 2 transposed 32 x 32
// matrix-core blocks, Z^T = W X^T, so that every lane holds one token and 16
// vocabulary entries of each block: the row statistics are then in-lane over
// 32 entries plus one swap between the wave halves, exactly as the attention
// kernels' row softmax.  A partial covers 64 vocabulary entries: partials are
// [M, N/64] pairs (maximum, sum of exp(z - maximum)).  Logits are written as
// float [M, N].  A 256 x 256 tile does 128 FLOPs per byte it brings into LDS,
// twice what a 128 x 128 tile does, which is what keeps the chiplets' L2
// bandwidth from capping the matrix cores.
//
// Tiles are dealt to the GPU's chiplets by vocabulary tile (modulo 8); a
// chiplet walks its vocabulary tiles eight at a time with the token tiles
// inside (lmhead_sched.h), so the W and X rows in flight on it fit its L2.
// A ragged last tile (N or M not a multiple of 256; both are multiples of
// 128) leaves the waves past the end idle and skips their copies.
//
// Kernel 2 (merge): one wave per token row combines the row's N/64 partials
// with the rescale-by-maximum-difference rule (the merge is not the fold),
// giving LSE, and with a target id the row loss LSE - Z[row, target].
// Kernel 3 (mean, shared with the cross-entropy operator): one work group
// sums the M row losses in a fixed order.
#include <math.h>

#include "attn_device.h"
#include "bf16_stream.h"
#include "lmhead_launch.h"
#include "lmhead_sched.h"
#include "memops_launch.h"

namespace cattn {

__global__ __launch_bounds__(512) void lmhead_logits_stats_kernel(const bf16* __restrict__ X,
                                                                  const bf16* __restrict__ W,
                                                                  float* __restrict__ Z, float* __restrict__ part,
                                                                  int M, int N, int K, int per_xcd) {
  constexpr int TILE = 32 * kLmhKC * 2;  // one 32-row block of a chunk: 4 KB
  constexpr int SLOT = 16 * TILE;        // W: 8 blocks (256 rows), X: 8 blocks (256 rows)
  constexpr int KS = kLmhKC / 16;
  __shared__ __attribute__((aligned(16))) char smem[2 * SLOT];

  const int n_vt = lmh_vtiles(N), n_mt = lmh_mtiles(M);
  const int x = blockIdx.x % kXcdGroup;
  const int n_tiles = lmh_xcd_tiles(x, n_vt, n_mt);
  int l = blockIdx.x / kXcdGroup;
  if (l >= n_tiles) return;  // uniform over the group

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int vw = w & 1, tw = w >> 1;  // this wave: vocabulary half (128 rows), token quarter (64)
  const int n_chunks = K / kLmhKC;
  const int n_part = N / kLmhPartW;

  // Waves 0-3 copy the W rows of a chunk, waves 4-7 its X rows: eight 32-row
  // blocks each, one 16-byte copy per lane per block.
  TileCopy<kLmhKC> tc;
  tc.init(w & 3, lane, K);
  const bool copies_w = w < 4;
  const bf16* src = copies_w ? W : X;
  const int src_rows = copies_w ? N : M;
  auto dma = [&](int tile, int c, int slot) {
    const int v0 = (tile >> 16) * kLmhTileV, m0 = (tile & 0xffff) * kLmhTileM;
    const int row0 = copies_w ? v0 : m0;
    char* b = smem + slot * SLOT + (copies_w ? 0 : 8 * TILE);
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (row0 + 32 * i < src_rows) tc.copy_full(src + c * kLmhKC, row0 + 32 * i, b + i * TILE);
  };

  int tile = lmh_xcd_tile(x, l, n_vt, n_mt);
  int slot = 0;
  dma(tile, 0, 0);
  while (true) {
    const int v0 = (tile >> 16) * kLmhTileV, m0 = (tile & 0xffff) * kLmhTileM;
    const int vrow = v0 + 128 * vw, tok0 = m0 + 64 * tw;
    const bool active = vrow < N && tok0 < M;  // uniform per wave
    const int l_next = l + per_xcd;
    const int tile_next = l_next < n_tiles ? lmh_xcd_tile(x, l_next, n_vt, n_mt) : -1;

    f32x16 acc[4][2];  // [vocabulary block][token block] of Z^T
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int t = 0; t < 2; ++t) acc[a][t] = f32x16{};

    for (int c = 0; c < n_chunks; ++c) {
      // chunk c landed in `slot` (the only copy in flight); every wave is done
      // reading the other slot, which the next copy overwrites
      tile_barrier(0);
      if (c + 1 < n_chunks) {
        dma(tile, c + 1, slot ^ 1);
      } else if (tile_next >= 0) {
        dma(tile_next, 0, slot ^ 1);
      }
      if (active) {
        // Operand fragments are double-buffered across k-steps: the reads of
        // step ks + 1 are issued before the contractions of step ks, so each
        // group of eight contractions runs while the next group's operands
        // arrive instead of waiting on LDS every two contractions.
        const char* b = smem + slot * SLOT;
        MB::frag wf[2][4], xf[2][2];
        auto read_step = [&](int ks, int buf) {
#pragma unroll
          for (int a = 0; a < 4; ++a) wf[buf][a] = read_row_frag<bf16, kLmhKC>(b + (4 * vw + a) * TILE, r, ks, h);
#pragma unroll
          for (int t = 0; t < 2; ++t) xf[buf][t] = read_row_frag<bf16, kLmhKC>(b + (8 + 2 * tw + t) * TILE, r, ks, h);
        };
        read_step(0, 0);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          if (ks + 1 < KS) read_step(ks + 1, (ks + 1) & 1);
#pragma unroll
          for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int t = 0; t < 2; ++t) acc[a][t] = MB::run(wf[ks & 1][a], xf[ks & 1][t], acc[a][t]);
        }
        // issue order: steps 0 and 1's reads, then per step its eight
        // contractions followed by the reads two steps ahead
        static_assert(KS == 4, "the issue order below is written for four k-steps");
        __builtin_amdgcn_sched_group_barrier(0x100, 12, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 16, 0);
      }
      slot ^= 1;
    }

    // Epilogue.  acc[a][t][e]: Z[token tok0 + 32 t + r][vocab vrow + 32 a + acc_row(e, h)]
    if (active) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int tok = tok0 + 32 * t + r;
        float* zrow = Z + (int64_t)tok * N + vrow;
#pragma unroll
        for (int p = 0; p < 2; ++p) {  // two partials of 64 entries: blocks 2p, 2p + 1
          float mx = acc[2 * p][t][0];
#pragma unroll
          for (int a = 2 * p; a < 2 * p + 2; ++a)
#pragma unroll
            for (int e = 0; e < 16; ++e) mx = fmaxf(mx, acc[a][t][e]);
          mx = halves_max(mx);
          float s = 0.f;
#pragma unroll
          for (int a = 2 * p; a < 2 * p + 2; ++a)
#pragma unroll
            for (int e = 0; e < 16; ++e) s += exp2_hw((acc[a][t][e] - mx) * kLog2e);
          s = halves_sum(s);
          if (h == 0) {
            float2* pp = (float2*)(part + ((int64_t)tok * n_part + (vrow + 64 * p) / kLmhPartW) * 2);
            *pp = make_float2(mx, s);
          }
        }
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int g = 0; g < 4; ++g)
            *(f32x4*)(zrow + 32 * a + 8 * g + 4 * h) =
                f32x4{acc[a][t][4 * g], acc[a][t][4 * g + 1], acc[a][t][4 * g + 2], acc[a][t][4 * g + 3]};
      }
    }
    if (tile_next < 0) break;
    l = l_next;
    tile = tile_next;
  }
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

// Work groups per chiplet of the persistent projection grid: one per compute
// unit (the kernel's 128 KB of LDS allows no more).
static int lmh_per_xcd() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 32;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = imax(1, n / kXcdGroup);
  }
  return cached[dev];
}

hipError_t launch_lmhead(const LmheadArgs& a, hipStream_t st) {
  const int per_xcd = lmh_per_xcd();
  hipLaunchKernelGGL(lmhead_logits_stats_kernel, dim3((unsigned)lmh_grid(per_xcd)), dim3(512), 0, st,
                     (const bf16*)a.x, (const bf16*)a.w, a.logits, a.part, a.M, a.N, a.K, per_xcd);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lmhead_merge_kernel, dim3((unsigned)((a.M + 3) / 4)), dim3(256), 0, st, (const float*)a.part,
                     (const float*)a.logits, a.targets, a.lse, a.row_loss, a.M, a.N);
  e = hipGetLastError();
  if (e != hipSuccess || !a.targets || !a.loss) return e;
  return launch_row_mean(a.row_loss, a.loss, a.M, st);
}

}  // namespace cattn
