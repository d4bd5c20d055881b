// bf16 attention kernels for gfx950: forward, dQ and dK/dV (section 4.2 of the
// Nova paper), organised around memory latency on CDNA4.
//
// Differences from the generic kernels (attn_fwd.hip, attn_bwd.hip, used for
// float32):
//  * Streamed operands move in tiles of 32 rows, HBM -> LDS with
//    global_load_lds_dwordx4 (no staging registers, no ds_write), through a
//    ring of Ring<D>::NBUF buffers.  The copy of tile t + AHEAD is issued at
//    the top of tile t, so about AHEAD tiles of compute cover the latency of
//    each copy; the wait at the top of tile t asks only for tile t+1 (newer
//    copies stay in flight), then one barrier publishes it.  Rows past the
//    end of the sequence are loaded from the last valid row (finite values)
//    and masked in the kernel.
//  * A 32-row tile is one sub-block of the matrix-core contractions.  Each
//    wave walks its own range of sub-blocks; operands of sub-block j+1 are
//    read from LDS (tile j+1 is always resident) while sub-block j computes.
//  * The forward is software pipelined: iteration j runs O += P(j-1) V(j-1)
//    and S(j+1) = K(j+1) Q^T on the matrix cores while the vector ALUs do the
//    softmax of S(j).
//  * Only the sub-block of a wave that straddles the causal diagonal (and the
//    ragged last one) is masked; every other sub-block is branch-free.
#include "attn_device.h"
#include "attn_launch.h"

namespace cattn {

typedef __bf16 bf16;
typedef Mma<bf16> MB;

#ifndef CATTN_TRACE
#define CATTN_TRACE(slot)
#endif

// Ring geometry for 32-row tiles of D bf16 columns.
template <int D> struct Ring {
  static constexpr int NBUF = D == 64 ? 6 : 4;
  static constexpr int AHEAD = NBUF - 1;                  // copy distance, in tiles
  static constexpr int TILE = 32 * D * 2;                 // bytes of one tensor's tile
  static constexpr int DMA_PER_TENSOR = TILE / 16 / 256;  // copy instructions per thread
};

// s_waitcnt vmcnt(n) for a wave-uniform n in [0, 30] (expcnt and lgkmcnt left
// at their maxima), through the builtin so that the compiler's own wait
// bookkeeping sees it.
__device__ __forceinline__ void wait_vm(int n) {
#define CATTN_VMW(k) \
  case k:            \
    __builtin_amdgcn_s_waitcnt(0x0F70 | ((k) & 15) | (((k) >> 4) << 14)); \
    break;
  switch (n) {
    CATTN_VMW(0) CATTN_VMW(1) CATTN_VMW(2) CATTN_VMW(3) CATTN_VMW(4) CATTN_VMW(5) CATTN_VMW(6) CATTN_VMW(7)
    CATTN_VMW(8) CATTN_VMW(9) CATTN_VMW(10) CATTN_VMW(11) CATTN_VMW(12) CATTN_VMW(13) CATTN_VMW(14)
    CATTN_VMW(15) CATTN_VMW(16) CATTN_VMW(17) CATTN_VMW(18) CATTN_VMW(19) CATTN_VMW(20) CATTN_VMW(21)
    CATTN_VMW(22) CATTN_VMW(23) CATTN_VMW(24) CATTN_VMW(25) CATTN_VMW(26) CATTN_VMW(27) CATTN_VMW(28)
    CATTN_VMW(29) CATTN_VMW(30)
    default: __builtin_amdgcn_s_waitcnt(0x0F70); break;
  }
#undef CATTN_VMW
}

// Publish a tile: wait until at most n of this wave's copies are in flight
// (the newest ones, which target later tiles) and all of its LDS reads have
// returned, then meet the other waves at the barrier.  A plain s_barrier: the
// release fence of __syncthreads() would wait for every copy in flight and
// undo the prefetch distance.  The asm memory clobber keeps the compiler from
// moving LDS accesses across the barrier.
__device__ __forceinline__ void tile_barrier(int n) {
#define CATTN_TBW(k) \
  case k:            \
    __builtin_amdgcn_s_waitcnt(0x0070 | ((k) & 15) | (((k) >> 4) << 14)); \
    break;
  switch (n) {
    CATTN_TBW(0) CATTN_TBW(1) CATTN_TBW(2) CATTN_TBW(3) CATTN_TBW(4) CATTN_TBW(5) CATTN_TBW(6) CATTN_TBW(7)
    CATTN_TBW(8) CATTN_TBW(9) CATTN_TBW(10) CATTN_TBW(11) CATTN_TBW(12) CATTN_TBW(13) CATTN_TBW(14)
    CATTN_TBW(15) CATTN_TBW(16) CATTN_TBW(17) CATTN_TBW(18) CATTN_TBW(19) CATTN_TBW(20) CATTN_TBW(21)
    CATTN_TBW(22) CATTN_TBW(23) CATTN_TBW(24) CATTN_TBW(25) CATTN_TBW(26) CATTN_TBW(27) CATTN_TBW(28)
    CATTN_TBW(29) CATTN_TBW(30)
    default: __builtin_amdgcn_s_waitcnt(0x0070); break;
  }
#undef CATTN_TBW
  asm volatile("s_barrier" ::: "memory");
}

// One 16-byte HBM -> LDS copy per active lane.  The LDS destination (M0) is
// wave-uniform; lane i's bytes land at M0 + 16 * i.  Issued as inline assembly
// so that the compiler does not treat every later LDS read as aliasing the
// copy in flight (it would then wait for the copy before each read);
// completion is awaited explicitly (wait_vm) before the barrier that
// publishes a tile.
__device__ __forceinline__ void dma16(const void* src, const char* lds_wave_base) {
  const unsigned dst = __builtin_amdgcn_readfirstlane((unsigned)(uintptr_t)lds_wave_base);
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(dst), "v"(src) : "memory", "m0");
}

// HBM -> LDS copy of a 32 x D bf16 tile (rows row0.. of g, row stride D).  The
// chunk a lane deposits at physical position p of the tile is logical chunk
// p ^ swz(row), so the LDS image has the swizzled layout Tile<> reads.  Rows
// >= nrows are clamped to nrows - 1.
template <int D>
__device__ __forceinline__ void dma_tile(const bf16* g, int row0, int nrows, char* lds, int tid) {
  constexpr int CPR = D * 2 / 16;  // 16-byte chunks per row
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
#pragma unroll
  for (int i = 0; i < Ring<D>::DMA_PER_TENSOR; ++i) {
    const int p = i * 256 + w * 64 + lane;
    const int row = p / CPR, lc = (p % CPR) ^ swz(row);
    const int grow = min(row0 + row, nrows - 1);
    dma16(g + (int64_t)grow * D + lc * 8, lds + (i * 256 + w * 64) * 16);
  }
}

// Row-major A-operand fragments of the 32 rows of a tile.
template <int D>
__device__ __forceinline__ void read_rows(const char* lds, int r, int h, MB::frag (&f)[D / 16]) {
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) f[ks] = read_row_frag<bf16, D>(lds, r, ks, h);
}

// Transposed A-operand fragments (columns 32*dt..) of the 32 rows of a tile.
template <int D>
__device__ __forceinline__ void read_trans(const char* lds, int lane, MB::frag (&f)[2][D / 32]) {
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) f[s][dt] = TransRead<bf16, D>::read(lds, 0, s, dt * 32, lane);
}

// Copies issued after tile t+1 and still allowed in flight at the top of
// tile t, for a ring running AHEAD tiles ahead over n tiles.
__device__ __forceinline__ int later_tiles(int t, int n, int ahead) {
  const int k = min(ahead - 2, n - 2 - t);
  return k > 0 ? k : 0;
}

// ---------------------------------------------------------------------------
// Forward
// ---------------------------------------------------------------------------
template <int D, bool CAUSAL>
__global__ __launch_bounds__(256) void attn_fwd_bf16_kernel(const bf16* __restrict__ Q, const bf16* __restrict__ K,
                                                            const bf16* __restrict__ V, bf16* __restrict__ O,
                                                            float* __restrict__ LSE, int S, int BH, int n_qtiles,
                                                            float c) {
  typedef Ring<D> RG;
  constexpr int BQ = 128, NB = RG::NBUF, AH = RG::AHEAD, TILE = RG::TILE;
  constexpr int KS_D = D / 16, DT = D / 32;
  constexpr int PER_TILE = 2 * RG::DMA_PER_TENSOR;
  __shared__ __attribute__((aligned(16))) char smem[NB * 2 * TILE];  // [buffer][K, V]

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index: uniform, kept in an SGPR
  int bh, qt;
  tile_of_block(blockIdx.x, BH, n_qtiles, CAUSAL, bh, qt);
  const int64_t base = (int64_t)bh * S * D;
  const bf16* Kb = K + base;
  const bf16* Vb = V + base;

  const int q0 = qt * BQ, qw = q0 + 32 * w, my_q = qw + r;
  const int kend = CAUSAL ? min(S, q0 + BQ) : S;  // causal loop clamping (workgroup)
  const int n = (kend + 31) / 32;                  // 32-key tiles the workgroup visits
  const int kend_w = qw >= S ? 0 : (CAUSAL ? min(S, qw + 32) : S);
  const int nsb = (kend_w + 31) / 32;              // of which this wave uses the first nsb

  auto buf = [&](int t) { return smem + (t % NB) * 2 * TILE; };
  auto dma = [&](int t) {
    dma_tile<D>(Kb, t * 32, S, buf(t), tid);
    dma_tile<D>(Vb, t * 32, S, buf(t) + TILE, tid);
  };
  CATTN_TRACE(0);
  for (int t = 0; t < AH && t < n; ++t) dma(t);
  MB::frag qf[KS_D];
  load_row_frags<bf16, D>(Q + base, my_q, S, h, qf);
  wait_vm(0);
  __syncthreads();
  CATTN_TRACE(1);

  float m = kMasked, lsum = 0.f;
  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x16{};
  // Pipeline state: sa = S(j); pp, vf = P(j-1) and V(j-1) for O += P V.
  f32x16 sa = f32x16{};
  MB::frag pp[2], vf[2][DT];
  pp[0] = MB::frag{};
  pp[1] = MB::frag{};
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) vf[ks][dt] = MB::frag{};
  {
    MB::frag k0f[KS_D];
    read_rows<D>(buf(0), r, h, k0f);
#pragma unroll
    for (int ks = 0; ks < KS_D; ++ks) sa = MB::run(k0f[ks], qf[ks], sa);
  }

  for (int j = 0; j < n; ++j) {
    if (j > 0) {
      tile_barrier(later_tiles(j, n, AH) * PER_TILE);  // tile j+1 landed; tile j-1 is free
    }
    CATTN_TRACE(2 + j);
    if (j + AH < n) dma(j + AH);
    if (j >= nsb) continue;  // wave-uniform: this wave is done, it only keeps the barriers
    const int k0 = j * 32;
    // causal diagonal / ragged end: only the wave's last sub-block
    if (j == nsb - 1 && ((CAUSAL && k0 + 31 > qw) || k0 + 32 > S)) {
#pragma unroll
      for (int a = 0; a < 16; ++a) {
        const int key = k0 + acc_row(a, h);
        if (key >= S || (CAUSAL && key > my_q)) sa[a] = kMasked;
      }
    }
    MB::frag kf[KS_D];  // K of sub-block j+1 (clamped to the last one)
    read_rows<D>(buf(j + 1 < nsb ? j + 1 : j), r, h, kf);
    __builtin_amdgcn_sched_barrier(0);  // issue the K reads before anything below
    // Softmax of S(j).  The offset moves (per lane, without a branch) only when
    // the block max exceeds it by more than 2^kRescaleLog2 in probability
    // units; alpha rescales the running sum here and O below.
    float mx = sa[0];
#pragma unroll
    for (int a = 1; a < 16; ++a) mx = fmaxf(mx, sa[a]);
    mx = halves_max(mx);
    const float m_use = (j == 0 || (mx - m) * c > kRescaleLog2) ? mx : m;
    const float alpha = exp2_hw((m - m_use) * c);  // 0 on the first block, 1 when unchanged
    m = m_use;
    const float mc = m * c;
    float pv[16];
    float psum = 0.f;
#pragma unroll
    for (int a = 0; a < 16; ++a) {
      pv[a] = exp2_hw(fmaf(sa[a], c, -mc));
      psum += pv[a];
    }
    lsum = fmaf(lsum, alpha, psum);
    // matrix cores, independent of the softmax: O += P(j-1) V(j-1), S(j+1) = K Q^T
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[dt] = MB::run(vf[ks][dt], pp[ks], oacc[dt]);
    f32x16 sn = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KS_D; ++ks) sn = MB::run(kf[ks], qf[ks], sn);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int i = 0; i < 8; ++i) pp[ks][i] = (bf16)pv[8 * ks + i];
#pragma unroll
    for (int i = 0; i < 2 * DT + KS_D; ++i) {  // interleave matrix-core and vector work
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
    }
    // The new P and the running sum are finished here, above the branch, so
    // that the exponentials stay in the same block as the contractions.
    asm volatile("" ::"v"(lsum), "v"(pp[0]), "v"(pp[1]));
    read_trans<D>(buf(j) + TILE, lane, vf);  // V(j), for the next iteration
    if (__builtin_amdgcn_ballot_w64(alpha != 1.0f)) {  // rare: rescale O (after P(j-1) V(j-1))
      // keeps this block a real branch: executed speculatively it would make
      // every iteration wait for the matrix-core accumulation above
      asm volatile("" ::: "memory");
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
    }
    sa = sn;
  }
  if (nsb > 0) {  // drain: O += P(last) V(last)
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[dt] = MB::run(vf[ks][dt], pp[ks], oacc[dt]);
  }

  CATTN_TRACE(60);
  const float l = halves_sum(lsum);
  if (my_q < S) {
    const float inv = 1.0f / l;
    bf16* orow = O + base + (int64_t)my_q * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        store4<bf16>(orow + dt * 32 + 8 * g + 4 * h, oacc[dt][4 * g] * inv, oacc[dt][4 * g + 1] * inv,
                     oacc[dt][4 * g + 2] * inv, oacc[dt][4 * g + 3] * inv);
    if (h == 0) LSE[(int64_t)bh * S + my_q] = (m * c + log2f(l)) * kLn2;
  }
  CATTN_TRACE(61);
}

// ---------------------------------------------------------------------------
// Backward, kernel 1: dQ (reduces over keys).  Also writes, per (batch, head),
// D = rowsum(dO * O) and LSE * log2(e) into the workspace (rows padded to a
// multiple of 32 with zeros) for the dK/dV kernel to copy by DMA.
// ---------------------------------------------------------------------------
template <int D, bool CAUSAL>
__global__ __launch_bounds__(256) void attn_bwd_dq_bf16_kernel(const bf16* __restrict__ Q, const bf16* __restrict__ K,
                                                               const bf16* __restrict__ V, const bf16* __restrict__ O,
                                                               const bf16* __restrict__ dO,
                                                               const float* __restrict__ LSE, bf16* __restrict__ dQ,
                                                               float* __restrict__ ws, int S, int BH, int n_qtiles,
                                                               float c, float scale) {
  typedef Ring<D> RG;
  constexpr int BQ = 128, NB = RG::NBUF, AH = RG::AHEAD, TILE = RG::TILE;
  constexpr int KS_D = D / 16, DT = D / 32;
  constexpr int PER_TILE = 2 * RG::DMA_PER_TENSOR;
  __shared__ __attribute__((aligned(16))) char smem[NB * 2 * TILE];  // [buffer][K, V]

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index: uniform, kept in an SGPR
  int bh, qt;
  tile_of_block(blockIdx.x, BH, n_qtiles, CAUSAL, bh, qt);
  const int64_t base = (int64_t)bh * S * D;
  const bf16* Kb = K + base;
  const bf16* Vb = V + base;
  const int Sp = ws_rows(S);

  const int q0 = qt * BQ, qw = q0 + 32 * w, my_q = qw + r;
  const int kend = CAUSAL ? min(S, q0 + BQ) : S;
  const int n = (kend + 31) / 32;
  const int kend_w = qw >= S ? 0 : (CAUSAL ? min(S, qw + 32) : S);
  const int nsb = (kend_w + 31) / 32;

  auto buf = [&](int t) { return smem + (t % NB) * 2 * TILE; };
  auto dma = [&](int t) {
    dma_tile<D>(Kb, t * 32, S, buf(t), tid);
    dma_tile<D>(Vb, t * 32, S, buf(t) + TILE, tid);
  };
  for (int t = 0; t < AH && t < n; ++t) dma(t);
  MB::frag qf[KS_D], dof[KS_D], of[KS_D];
  load_row_frags<bf16, D>(Q + base, my_q, S, h, qf);
  load_row_frags<bf16, D>(dO + base, my_q, S, h, dof);
  load_row_frags<bf16, D>(O + base, my_q, S, h, of);
  const float lse = my_q < S ? LSE[(int64_t)bh * S + my_q] : 0.f;
  wait_vm(0);
  __syncthreads();

  // D = rowsum(dO * O) in float, from the O the forward produced.
  float dpart = 0.f;
#pragma unroll
  for (int ks = 0; ks < KS_D; ++ks)
#pragma unroll
    for (int i = 0; i < 8; ++i) dpart = fmaf((float)dof[ks][i], (float)of[ks][i], dpart);
  const float Dq = halves_sum(dpart);
  const float lse2 = lse * kLog2e;
  if (h == 0 && my_q < Sp) {
    ws[(int64_t)bh * Sp + my_q] = my_q < S ? Dq : 0.f;
    ws[((int64_t)BH + bh) * Sp + my_q] = lse2;
  }

  f32x16 dqacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) dqacc[dt] = f32x16{};
  MB::frag kf[KS_D], vfr[KS_D];  // row fragments of the current sub-block
  read_rows<D>(buf(0), r, h, kf);
  read_rows<D>(buf(0) + TILE, r, h, vfr);

  for (int j = 0; j < n; ++j) {
    if (j > 0) {
      tile_barrier(later_tiles(j, n, AH) * PER_TILE);
    }
    if (j + AH < n) dma(j + AH);
    if (j >= nsb) continue;
    MB::frag ktr[2][DT];
    read_trans<D>(buf(j), lane, ktr);
    MB::frag kn[KS_D], vn[KS_D];
    const int jn = j + 1 < nsb ? j + 1 : j;
    read_rows<D>(buf(jn), r, h, kn);
    read_rows<D>(buf(jn) + TILE, r, h, vn);
    f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KS_D; ++ks) {
      s = MB::run(kf[ks], qf[ks], s);
      dp = MB::run(vfr[ks], dof[ks], dp);
    }
    const int k0 = j * 32;
    if (j == nsb - 1 && ((CAUSAL && k0 + 31 > qw) || k0 + 32 > S)) {
#pragma unroll
      for (int a = 0; a < 16; ++a) {
        const int key = k0 + acc_row(a, h);
        if (key >= S || (CAUSAL && key > my_q)) s[a] = kMasked;
      }
    }
#pragma unroll
    for (int a = 0; a < 16; ++a) {
      const float p = exp2_hw(fmaf(s[a], c, -lse2));
      dp[a] = p * (dp[a] - Dq);  // dS^T
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const MB::frag db = MB::pack(dp, ks);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) dqacc[dt] = MB::run(ktr[ks][dt], db, dqacc[dt]);
    }
#pragma unroll
    for (int ks = 0; ks < KS_D; ++ks) {
      kf[ks] = kn[ks];
      vfr[ks] = vn[ks];
    }
  }

  if (my_q < S) {
    bf16* row = dQ + base + (int64_t)my_q * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        store4<bf16>(row + dt * 32 + 8 * g + 4 * h, dqacc[dt][4 * g] * scale, dqacc[dt][4 * g + 1] * scale,
                     dqacc[dt][4 * g + 2] * scale, dqacc[dt][4 * g + 3] * scale);
  }
}

// ---------------------------------------------------------------------------
// Backward, kernel 2: dK, dV (reduces over queries)
// ---------------------------------------------------------------------------
template <int D, bool CAUSAL>
__global__ __launch_bounds__(256) void attn_bwd_dkdv_bf16_kernel(const bf16* __restrict__ Q,
                                                                 const bf16* __restrict__ K,
                                                                 const bf16* __restrict__ V,
                                                                 const bf16* __restrict__ dO,
                                                                 const float* __restrict__ ws,
                                                                 bf16* __restrict__ dK, bf16* __restrict__ dV, int S,
                                                                 int BH, int n_ktiles, float c, float scale) {
  typedef Ring<D> RG;
  constexpr int BKV = 128, NB = RG::NBUF, AH = RG::AHEAD, TILE = RG::TILE;
  constexpr int KS_D = D / 16, DT = D / 32;
  constexpr int BUF = 2 * TILE + 2 * 32 * 4;  // Q, dO, then 32 floats LSE*log2e, 32 floats D
  __shared__ __attribute__((aligned(16))) char smem[NB * BUF];

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index: uniform, kept in an SGPR
  int bh, kt;
  tile_of_block(blockIdx.x, BH, n_ktiles, false, bh, kt);
  const int64_t base = (int64_t)bh * S * D;
  const bf16* Qb = Q + base;
  const bf16* dOb = dO + base;
  const int Sp = ws_rows(S);
  const float* Db = ws + (int64_t)bh * Sp;
  const float* Lb = ws + ((int64_t)BH + bh) * Sp;
  // copies per tile issued by this wave: Q and dO, plus the LSE/D copy on wave 0
  const int per_tile = 2 * RG::DMA_PER_TENSOR + (w == 0 ? 1 : 0);

  const int k0 = kt * BKV, kw = k0 + 32 * w, my_k = kw + r;
  // 32-query tiles of the workgroup: from the one holding k0 (causal: the loop's
  // lower bound is raised to the diagonal) to the end of the sequence.
  const int jt0 = CAUSAL ? k0 / 32 : 0;
  const int n = (S + 31) / 32 - jt0;
  const int jb = CAUSAL ? kw / 32 : 0;          // this wave's first sub-block
  const int je = kw >= S ? jb : (S + 31) / 32;  // ... and one past its last

  auto buf = [&](int t) { return smem + (t % NB) * BUF; };
  auto dma = [&](int t) {
    const int row0 = (jt0 + t) * 32;
    char* b = buf(t);
    dma_tile<D>(Qb, row0, S, b, tid);
    dma_tile<D>(dOb, row0, S, b + TILE, tid);
    if (w == 0 && lane < 16)  // 8 chunks of LSE*log2e, then 8 of D (rows < Sp: in bounds)
      dma16((lane < 8 ? Lb : Db) + row0 + 4 * (lane & 7), b + 2 * TILE);
  };
  for (int t = 0; t < AH && t < n; ++t) dma(t);
  MB::frag kf[KS_D], vf[KS_D];
  load_row_frags<bf16, D>(K + base, my_k, S, h, kf);
  load_row_frags<bf16, D>(V + base, my_k, S, h, vf);
  wait_vm(0);
  __syncthreads();

  f32x16 dkacc[DT], dvacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) {
    dkacc[dt] = f32x16{};
    dvacc[dt] = f32x16{};
  }
  MB::frag qf[KS_D], dof[KS_D];  // row fragments of the current sub-block

  for (int t = 0; t < n; ++t) {
    if (t > 0) {
      tile_barrier(later_tiles(t, n, AH) * per_tile);
    }
    if (t + AH < n) dma(t + AH);
    const int j = jt0 + t;            // global sub-block index
    if (j < jb || j >= je) continue;  // wave-uniform
    const char* lq = buf(t);
    const char* ldo = lq + TILE;
    const float* llse = (const float*)(lq + 2 * TILE);
    const float* ld = llse + 32;
    if (j == jb) {  // a wave's first sub-block can be any tile: read it here
      read_rows<D>(lq, r, h, qf);
      read_rows<D>(ldo, r, h, dof);
    }
    MB::frag dotr[2][DT], qtr[2][DT];
    read_trans<D>(ldo, lane, dotr);
    read_trans<D>(lq, lane, qtr);
    MB::frag qn[KS_D], don[KS_D];
    const int tn = j + 1 < je ? t + 1 : t;
    read_rows<D>(buf(tn), r, h, qn);
    read_rows<D>(buf(tn) + TILE, r, h, don);
    f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KS_D; ++ks) {
      s = MB::run(qf[ks], kf[ks], s);
      dp = MB::run(dof[ks], vf[ks], dp);
    }
    // s[a], dp[a]: query 32j + acc_row(a, h), key my_k
    const int qs = j * 32;
    if ((CAUSAL && j == jb) || qs + 32 > S) {
#pragma unroll
      for (int a = 0; a < 16; ++a) {
        const int qry = qs + acc_row(a, h);
        if (qry >= S || (CAUSAL && my_k > qry)) s[a] = kMasked;
      }
    }
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 l4 = *(const f32x4*)(llse + 8 * g + 4 * h);
      const f32x4 d4 = *(const f32x4*)(ld + 8 * g + 4 * h);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int a = 4 * g + i;
        const float p = exp2_hw(fmaf(s[a], c, -l4[i]));
        s[a] = p;
        dp[a] = p * (dp[a] - d4[i]);  // dS
      }
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const MB::frag pb = MB::pack(s, ks);
      const MB::frag db = MB::pack(dp, ks);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        dvacc[dt] = MB::run(dotr[ks][dt], pb, dvacc[dt]);
        dkacc[dt] = MB::run(qtr[ks][dt], db, dkacc[dt]);
      }
    }
#pragma unroll
    for (int ks = 0; ks < KS_D; ++ks) {
      qf[ks] = qn[ks];
      dof[ks] = don[ks];
    }
  }

  if (my_k < S) {
    bf16* krow = dK + base + (int64_t)my_k * D;
    bf16* vrow = dV + base + (int64_t)my_k * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int col = dt * 32 + 8 * g + 4 * h;
        store4<bf16>(krow + col, dkacc[dt][4 * g] * scale, dkacc[dt][4 * g + 1] * scale,
                     dkacc[dt][4 * g + 2] * scale, dkacc[dt][4 * g + 3] * scale);
        store4<bf16>(vrow + col, dvacc[dt][4 * g], dvacc[dt][4 * g + 1], dvacc[dt][4 * g + 2], dvacc[dt][4 * g + 3]);
      }
  }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
template <int D, bool CAUSAL>
static hipError_t fwd_bf16_t(const FwdArgs& a, hipStream_t st) {
  const int n_qtiles = (a.S + 127) / 128;
  hipLaunchKernelGGL((attn_fwd_bf16_kernel<D, CAUSAL>), dim3((unsigned)((int64_t)a.BH * n_qtiles)), dim3(256), 0,
                     st, (const bf16*)a.q, (const bf16*)a.k, (const bf16*)a.v, (bf16*)a.o, a.lse, a.S, a.BH,
                     n_qtiles, a.scale * kLog2e);
  return hipGetLastError();
}

hipError_t launch_fwd_bf16(const FwdArgs& a, hipStream_t st) {
  if (a.D == 64) return a.causal ? fwd_bf16_t<64, true>(a, st) : fwd_bf16_t<64, false>(a, st);
  return a.causal ? fwd_bf16_t<128, true>(a, st) : fwd_bf16_t<128, false>(a, st);
}

template <int D, bool CAUSAL>
static hipError_t bwd_bf16_t(const BwdArgs& a, int phase, hipStream_t st) {
  const float c = a.scale * kLog2e;
  if (phase != 2) {
    const int n_qtiles = (a.S + 127) / 128;
    hipLaunchKernelGGL((attn_bwd_dq_bf16_kernel<D, CAUSAL>), dim3((unsigned)((int64_t)a.BH * n_qtiles)), dim3(256),
                       0, st, (const bf16*)a.q, (const bf16*)a.k, (const bf16*)a.v, (const bf16*)a.o,
                       (const bf16*)a.dout, a.lse, (bf16*)a.dq, a.ws, a.S, a.BH, n_qtiles, c, a.scale);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || phase == 1) return e;
  }
  const int n_ktiles = (a.S + 127) / 128;
  hipLaunchKernelGGL((attn_bwd_dkdv_bf16_kernel<D, CAUSAL>), dim3((unsigned)((int64_t)a.BH * n_ktiles)), dim3(256),
                     0, st, (const bf16*)a.q, (const bf16*)a.k, (const bf16*)a.v, (const bf16*)a.dout,
                     (const float*)a.ws, (bf16*)a.dk, (bf16*)a.dv, a.S, a.BH, n_ktiles, c, a.scale);
  return hipGetLastError();
}

hipError_t launch_bwd_bf16(const BwdArgs& a, int phase, hipStream_t st) {
  if (a.D == 64) return a.causal ? bwd_bf16_t<64, true>(a, phase, st) : bwd_bf16_t<64, false>(a, phase, st);
  return a.causal ? bwd_bf16_t<128, true>(a, phase, st) : bwd_bf16_t<128, false>(a, phase, st);
}

}  // namespace cattn
