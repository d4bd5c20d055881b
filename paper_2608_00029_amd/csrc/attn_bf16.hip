// bf16 attention kernels for gfx950: forward, dQ and dK/dV (section 4.2 of the
// Nova paper), organised around memory latency and vector-ALU issue on CDNA4.
//
// Differences from the generic kernels (attn_fwd.hip, attn_bwd.hip, used for
// float32):
//  * Streamed operands move in tiles of 32 rows, HBM -> LDS with
//    global_load_lds_dwordx4 (no staging registers, no ds_write), through a
//    ring of NB buffers.  The copy of tile t + NB - 1 is issued at the top of
//    tile t, so several tiles of compute cover the latency of each copy; the
//    wait at the top of tile t asks only for the tiles it is about to read
//    (newer copies stay in flight), then one barrier publishes them.  Rows
//    past the end of the sequence are loaded from the last valid row (finite
//    values) and masked in the kernel.
//  * The copies take a wave-uniform base address in scalar registers plus a
//    per-lane 32-bit offset fixed for the whole kernel, and every loop is
//    unrolled by the ring depth so that each LDS read names its buffer with an
//    immediate offset: no per-iteration vector address arithmetic.
//  * A 32-row tile is one sub-block of the matrix-core contractions.  Each
//    wave walks its own range of sub-blocks; operands of sub-block j+1 are
//    read from LDS (tile j+1 is always resident) while sub-block j computes.
//  * The forward is software pipelined: iteration j runs O += P(j-1) V(j-1)
//    and S(j+1) = K(j+1) Q^T on the matrix cores while the vector ALUs do the
//    softmax of S(j).
//  * Only the sub-block of a wave that straddles the causal diagonal (and the
//    ragged last one) is masked; every other sub-block is branch-free.
#include <utility>

#include "attn_device.h"
#include "attn_launch.h"
#include "bf16_stream.h"

namespace cattn {

// Ring depths (LDS slots of 32-row tiles) and iterations per ring barrier, as
// measured best on the MI355X.  The unsplit rings at head dimension 64 hold 4
// tiles, copies 3 tiles ahead (the forward, at four work groups per CU, uses
// 128 of the CU's 160 KB of LDS; 6-tile backward rings measured 2-5% slower).
constexpr int kFwdNb64 = 4;      // forward at head dimension 64
constexpr int kBwdNb64 = 4;      // dQ and dK/dV at head dimension 64
constexpr int kFwdNb128 = 3;     // forward at head dimension 128 (three work groups per CU)
constexpr int kBwdNb128 = 4;     // dQ and dK/dV at head dimension 128
constexpr int kFwdNbSplit = 3;   // forward at D = 64 with the key range in two parts (one ring each)
constexpr int kBwdNbSplit = 4;   // dQ and dK/dV at D = 64 with the loop range in two parts
constexpr int kFwdGroup = 2;     // iterations per barrier, where the ring is deep enough (ring_group)
constexpr int kDqGroup = 2;
constexpr int kDkdvGroup = 2;
// The backward at D = 64 splits each tile's loop range in two when the unsplit
// grid would fill fewer than this many work-group slots per CU.
constexpr int kBwdSplitWgPerCu = 2;

// Causal loop clamping (section 4.2): the loops visit only the tiles that hold
// visible (query, key) pairs -- the forward and dQ loops stop at the diagonal,
// the dK/dV loop starts there.  A test build (CATTN_TEST_NOCLAMP=1, never the
// product library) visits every tile instead, masking the ones past the
// diagonal entirely, to show that clamping changes no result: a fully masked
// tile has P = exp2(-1e30 c - m c) = 0 exactly, adds 0 to every sum and never
// moves the softmax offset.
#ifndef CATTN_TEST_NOCLAMP
#define CATTN_TEST_NOCLAMP 0
#endif
constexpr bool kNoClamp = CATTN_TEST_NOCLAMP != 0;

// The forward keeps a softmax offset that moves only when a block's partial
// probability sum exceeds this bound (or is not finite).  Probabilities are
// then at most 2^32 (offset at most 32 below the running max, base 2), far
// inside float and bf16 range even summed over 2^24 keys; O/l and LSE are
// exact for any offset.
constexpr float kSumMax = 4294967296.0f;

// ---------------------------------------------------------------------------
// Forward
//
// A workgroup owns 32*QG queries of one (batch, head), QG = 4/SPLIT query
// groups of 32 (one per wave), and splits the keys it must visit into SPLIT
// consecutive parts: wave w takes query group w % QG and key part w / QG.
// Each part streams its own ring of K/V tiles, so the sequential chain of a
// wave is 1/SPLIT of the key range (the critical path of the causal grid is
// its heaviest query tile).  With SPLIT = 2 the two partial results of a
// query group -- (O, running offset, running sum) -- merge lane to lane
// through LDS at the end with the usual rescale-by-offset-difference rule.
//
// Online softmax in base 2 with a lazily moved offset: the exponentials of a
// block are taken against the current offset m and summed in float; only
// when some lane's sum leaves [0, kSumMax] (a score far above m, or the first
// block, where m is the mask value) does the wave take the rare path that
// computes the block max, moves m, rescales O and the running sum, and redoes
// the block.  No per-block max is computed on the common path.
// ---------------------------------------------------------------------------
template <int D, bool CAUSAL, int SPLIT, int NB, bool RAG>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(SPLIT == 1 ? (D == 128 ? 3 : 4) : 1, 10)))
void attn_fwd_bf16_kernel(const bf16* __restrict__ Q, const bf16* __restrict__ K,
                                                            const bf16* __restrict__ V, bf16* __restrict__ O,
                                                            float* __restrict__ LSE, int S, int BH, int n_qtiles,
                                                            float c, int band, int H, int seq_major) {
  typedef TileGeom<D> G;
  constexpr int QG = 4 / SPLIT, BQ = 32 * QG;
  constexpr int TILE = G::TILE, SET = 2 * TILE;
  constexpr int KS_D = D / 16, DT = D / 32;
  constexpr int PER_TILE = 2 * G::DMA_PER_TENSOR;
  __shared__ __attribute__((aligned(16))) char smem[SPLIT * NB * SET];  // [part][slot][K, V]
  static_assert(SPLIT == 1 || 2 * 64 * (2 * DT * 16 + 2) * 4 <= SPLIT * NB * SET, "merge area");

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index: uniform, kept in an SGPR
  const int qg = w % QG, part = w / QG;
  int bh, qt;
  tile_of_block_banded(blockIdx.x, BH, n_qtiles, CAUSAL, CAUSAL ? band : 0, bh, qt);
  const Rows rw = rows_of(bh, H, S, D, seq_major);
  const int64_t base = rw.base;
  const int rs = rw.rs;
  const bf16* Kb = K + base;
  const bf16* Vb = V + base;

  const int q0 = qt * BQ, qw = q0 + 32 * qg, my_q = qw + r;
  const int kend = CAUSAL && !kNoClamp ? min(S, q0 + BQ) : S;   // causal loop clamping (workgroup)
  const int n = (kend + 31) / 32;                   // 32-key tiles of the workgroup
  const int L = (n + SPLIT - 1) / SPLIT;            // tiles per part (the last may be short)
  const int kend_w = qw >= S ? 0 : (CAUSAL && !kNoClamp ? min(S, qw + 32) : S);
  const int nsb = (kend_w + 31) / 32;               // tiles this wave's queries need
  const int tb = part * L;                          // this wave's tiles: [tb, te)
  const int te = min(nsb, min(n, tb + L));
  const int cnt = te > tb ? te - tb : 0;

  const int n_last = n - (SPLIT - 1) * L;  // tiles of the last part (<= L)
  // the key tile that holds the ragged end of the sequence, if this workgroup copies one
  const int t_rag = RAG && (S - 1) / 32 < n ? (S - 1) / 32 : -1;
  // the iteration (in this wave's part) whose tile must be masked: the wave's
  // last tile when it straddles the causal diagonal or the end of the sequence
  // (without the clamp, every tile from the one holding the diagonal on: i >= i_mask)
  const int i_mask = CAUSAL && kNoClamp ? qw / 32 - tb
                     : nsb > 0 && ((CAUSAL && (nsb - 1) * 32 + 31 > qw) || nsb * 32 > S) ? nsb - 1 - tb : -1;

  TileCopy<D> tc;
  tc.init(w, lane, rs);
  const char* ring = smem + part * NB * SET;  // this wave's part
  auto dma = [&](int x, auto slc) {  // iteration x's tile of every part, into ring slot slc
#pragma unroll
    for (int p = 0; p < SPLIT; ++p) {
      if (p < SPLIT - 1 || x < n_last) {
        const int t = p * L + x;
        char* dst = smem + (p * NB + decltype(slc)::value) * SET;
        if (!RAG || t != t_rag) {
          tc.copy_full(Kb, t * 32, dst);
          tc.copy_full(Vb, t * 32, dst + TILE);
        } else {
          tc.copy(Kb, t * 32, S, dst);
          tc.copy(Vb, t * 32, S, dst + TILE);
        }
      }
    }
  };
  // Unsplit grids: each block runs start to end in its iteration (no score
  // block computed ahead) with every K and V fragment read from LDS one
  // contraction step before its use, which leaves room for four waves per SIMD
  // at D = 64 (110 registers) and three at D = 128.  Split grids compute
  // S(j+1) while the softmax of S(j) runs.
  constexpr bool LEANF = SPLIT == 1;
  constexpr int NEED = LEANF ? 0 : 1;  // iteration i reads the tiles of iterations i .. i+NEED
  constexpr int GROUP = ring_group(SPLIT, NB, NEED, kFwdGroup);  // iterations per barrier
  static_assert(!LEANF || SPLIT * NB * SET <= 65536, "tile reads reach every slot by immediate offset");
  ring_prologue<NB, GROUP>(L, dma);
  Frag128 fo;
  if constexpr (LEANF && D == 128) fo.init(r, h, lane);
  auto rowf = [&](const char* t, int ks) -> MB::frag {  // K row fragment ks of tile t
    if constexpr (D == 128) return fo.row_frag(t, ks);
    else return read_row_frag<bf16, D>(t, r, ks, h);
  };
  auto trf = [&](const char* t, int ks, int dt) -> MB::frag {  // transposed V fragment
    if constexpr (D == 128) return fo.trans(t, ks, dt);
    else return TransRead<bf16, D>::read(t, 0, ks, dt * 32, lane);
  };
  MB::frag qf[KS_D];
  load_row_frags<bf16, D>(Q + base, my_q, S, h, rs, qf);
  wait_vm(0);
  __syncthreads();

  float m = kMasked, lsum = 0.f;
  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x16{};
  // Pipeline state of iteration j: sa = S(j); pp, vf = P(j-1) and V(j-1) for O += P V.
  // With an even ring depth the two copies alternate by ring slot parity (every
  // index a constant, no register moves); otherwise index 1 is copied to 0.
  constexpr bool PAR = NB % 2 == 0;
  f32x16 sa[2];
  MB::frag pp[2][2], vf[2][DT];  // V(j-1) is read into the same registers once O += P V has issued
#pragma unroll
  for (int x = 0; x < 2; ++x) {
    sa[x] = f32x16{};
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) pp[x][ks] = MB::frag{};
  }
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) vf[ks][dt] = MB::frag{};
  if constexpr (!LEANF) {
    MB::frag k0f[KS_D];
    read_rows<D>(ring, r, h, k0f);
#pragma unroll
    for (int ks = 0; ks < KS_D; ++ks) sa[0] = MB::run(k0f[ks], qf[ks], sa[0]);
  }

  auto softmax = [&](const f32x16& s, float mc, f32x16& pv) {
#pragma unroll
    for (int a = 0; a < 16; ++a) pv[a] = exp2_hw(fmaf(s[a], c, -mc));
    float ps[8];  // pairwise sum: a short dependency chain
#pragma unroll
    for (int a = 0; a < 8; ++a) ps[a] = pv[2 * a] + pv[2 * a + 1];
#pragma unroll
    for (int a = 0; a < 4; ++a) ps[a] = ps[2 * a] + ps[2 * a + 1];
    return (ps[0] + ps[1]) + (ps[2] + ps[3]);
  };

  for (int i0 = 0; i0 < L; i0 += NB) {
    unroll<NB>([&](auto slc) {
      constexpr int sl = decltype(slc)::value;
      constexpr int pc = PAR ? (sl & 1) : 0, pn = PAR ? (pc ^ 1) : 1;
      const int i = i0 + sl;
      if (i >= L) return;
      ring_step<NB, GROUP, NEED, SPLIT, PER_TILE, sl>(i, L, n_last, dma);
      if (i >= cnt) return;  // wave-uniform: this wave is done, it only keeps the barriers
      if constexpr (LEANF) {
        const char* kt = ring + sl * SET;
        f32x16 s = f32x16{};
        MB::frag ka[2];
        ka[0] = rowf(kt, 0);
#pragma unroll
        for (int ks = 0; ks < KS_D; ++ks) {
          if (ks + 1 < KS_D) ka[(ks + 1) & 1] = rowf(kt, ks + 1);
          s = MB::run(ka[ks & 1], qf[ks], s);
        }
        if (CAUSAL && kNoClamp ? i >= i_mask : i == i_mask) {
          const int k0 = (tb + i) * 32;
#pragma unroll
          for (int a = 0; a < 16; ++a) {
            const int key = k0 + acc_row(a, h);
            if ((RAG && key >= S) || (CAUSAL && key > my_q)) s[a] = kMasked;
          }
        }
        f32x16 pv;
        float psum = softmax(s, m * c, pv);
        if (__builtin_amdgcn_ballot_w64(!(psum <= kSumMax))) {  // rare: move the offset
          asm volatile("" ::: "memory");
          float mx = s[0];
#pragma unroll
          for (int a = 1; a < 16; ++a) mx = fmaxf(mx, s[a]);
          const float mnew = fmaxf(m, halves_max(mx));
          const float alpha = exp2_hw((m - mnew) * c);  // 0 on the first block
          m = mnew;
          psum = softmax(s, m * c, pv);
          lsum *= alpha;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
        }
        lsum += psum;
        const MB::frag pb[2] = {MB::pack(pv, 0), MB::pack(pv, 1)};
        MB::frag va[2];
        va[0] = trf(kt + TILE, 0, 0);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            const int x = ks * DT + dt;
            if (x + 1 < 2 * DT) va[(x + 1) & 1] = trf(kt + TILE, (x + 1) / DT, (x + 1) % DT);
            oacc[dt] = MB::run(va[x & 1], pb[ks], oacc[dt]);
          }
        return;
      }
      f32x16& sa_ = sa[pc];
      // causal diagonal / ragged end: only the last tile of the wave's queries
      if (CAUSAL && kNoClamp ? i >= i_mask : i == i_mask) {
        const int k0 = (tb + i) * 32;
#pragma unroll
        for (int a = 0; a < 16; ++a) {
          const int key = k0 + acc_row(a, h);
          if ((RAG && key >= S) || (CAUSAL && key > my_q)) sa_[a] = kMasked;
        }
      }
      // K of the next tile.  On a wave's last iteration this slot holds another
      // tile (or nothing yet); the product is computed and discarded.
      MB::frag kf[KS_D];
      read_rows<D>(ring + ((sl + 1) % NB) * SET, r, h, kf);
      __builtin_amdgcn_sched_barrier(0);  // issue the K reads before anything below
      f32x16 pv;
      float psum = softmax(sa_, m * c, pv);
      // matrix cores, independent of the softmax: O += P(j-1) V(j-1), S(j+1) = K Q^T
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) oacc[dt] = MB::run(vf[ks][dt], pp[pc][ks], oacc[dt]);
      f32x16& sn = sa[pn];
      sn = f32x16{};
#pragma unroll
      for (int ks = 0; ks < KS_D; ++ks) sn = MB::run(kf[ks], qf[ks], sn);
      MB::frag (&pn_)[2] = pp[pn];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) pn_[ks] = MB::pack(pv, ks);
#pragma unroll
      for (int e = 0; e < 2 * DT + KS_D; ++e) {  // interleave matrix-core and vector work
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
      }
      // The new P and its sum are finished here, above the branch, so that
      // the exponentials stay in the same block as the contractions.
      asm volatile("" ::"v"(psum), "v"(pn_[0]), "v"(pn_[1]));
      read_trans<D>(ring + sl * SET + TILE, lane, vf);  // V(j), for the next iteration
      if (__builtin_amdgcn_ballot_w64(!(psum <= kSumMax))) {  // rare: move the offset
        // keeps this block a real branch: executed speculatively it would make
        // every iteration wait for the matrix-core accumulation above
        asm volatile("" ::: "memory");
        float mx = sa_[0];
#pragma unroll
        for (int a = 1; a < 16; ++a) mx = fmaxf(mx, sa_[a]);
        const float mnew = fmaxf(m, halves_max(mx));  // same in both halves of a query
        const float alpha = exp2_hw((m - mnew) * c);  // 0 on the first block
        m = mnew;
        psum = softmax(sa_, m * c, pv);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) pn_[ks] = MB::pack(pv, ks);
        lsum *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;  // after O += P(j-1) V(j-1)
      }
      lsum += psum;
      if constexpr (!PAR) {
        sa[0] = sa[1];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) pp[0][ks] = pp[1][ks];
      }
    });
  }
  // drain: O += P(last) V(last), held at index (cnt & 1) by parity (index 0 otherwise)
  auto drain = [&](const MB::frag (&pl)[2]) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[dt] = MB::run(vf[ks][dt], pl[ks], oacc[dt]);
  };
  if (!LEANF && cnt > 0) {
    if (PAR && (cnt & 1)) {
      drain(pp[1]);
    } else {
      drain(pp[0]);
    }
  }

  if constexpr (SPLIT == 2) {
    // Merge the two key parts of each query group: part 1 hands (O, m, l) to
    // part 0 through LDS, lane to lane (both waves share the same lane layout).
    wait_vm(0);
    __syncthreads();  // every wave is done with the rings
    float* xb = (float*)smem + (size_t)qg * 64 * (2 * DT * 16 + 2);
    if (part == 1) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int a = 0; a < 16; ++a) xb[(dt * 16 + a) * 64 + lane] = oacc[dt][a];
      xb[(DT * 16) * 64 + lane] = m;
      xb[(DT * 16 + 1) * 64 + lane] = lsum;
    }
    __syncthreads();
    if (part == 1) return;
    const float m1 = xb[(DT * 16) * 64 + lane], l1 = xb[(DT * 16 + 1) * 64 + lane];
    const float mn = fmaxf(m, m1);
    const float s0 = exp2_hw((m - mn) * c), s1 = exp2_hw((m1 - mn) * c);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int a = 0; a < 16; ++a) oacc[dt][a] = oacc[dt][a] * s0 + xb[(dt * 16 + a) * 64 + lane] * s1;
    lsum = lsum * s0 + l1 * s1;
    m = mn;
  }

  const float l = halves_sum(lsum);
  if (my_q < S) {
    const float inv = 1.0f / l;
    bf16* orow = O + base + (int64_t)my_q * rs;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        store4<bf16>(orow + dt * 32 + 8 * g + 4 * h, oacc[dt][4 * g] * inv, oacc[dt][4 * g + 1] * inv,
                     oacc[dt][4 * g + 2] * inv, oacc[dt][4 * g + 3] * inv);
    if (h == 0) LSE[(int64_t)bh * S + my_q] = (m * c + log2f(l)) * kLn2;
  }
}

// ---------------------------------------------------------------------------
// Backward, kernel 1: dQ (reduces over keys).  Also writes, per (batch, head),
// D = rowsum(dO * O) and -LSE/scale into the workspace (rows padded to a
// multiple of 32 with zeros) for the dK/dV kernel to copy by DMA.
//
// Like the forward, a workgroup owns 32*QG queries (QG = 4/SPLIT query groups
// of 32, one per wave) and splits the keys it must visit into SPLIT parts,
// each streaming its own ring of K/V tiles; with SPLIT = 2 the two partial
// dQ are added through LDS at the end.
//
// dS = P (dP - D) takes one multiply per element: the dP contraction starts
// from an accumulator holding D and multiplies by -dO, so it yields D - dP.
// ---------------------------------------------------------------------------
template <int D, bool CAUSAL, int SPLIT, int NB, bool RAG, bool STR>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(STR ? 4 : 1, 10)))
void attn_bwd_dq_bf16_kernel(const bf16* __restrict__ Q, const bf16* __restrict__ K,
                                                               const bf16* __restrict__ V, const bf16* __restrict__ O,
                                                               const bf16* __restrict__ dO,
                                                               const float* __restrict__ LSE, bf16* __restrict__ dQ,
                                                               float* __restrict__ ws, int S, int BH, int n_qtiles,
                                                               float c, float scale, int band, int H, int seq_major) {
  typedef TileGeom<D> G;
  constexpr int QG = 4 / SPLIT, BQ = 32 * QG;
  constexpr int TILE = G::TILE, SET = 2 * TILE;
  constexpr int KS_D = D / 16, DT = D / 32;
  constexpr int PER_TILE = 2 * G::DMA_PER_TENSOR;
  __shared__ __attribute__((aligned(16))) char smem[SPLIT * NB * SET];  // [part][slot][K, V]
  static_assert(SPLIT == 1 || QG * 64 * (DT * 16) * 4 <= SPLIT * NB * SET, "merge area");

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index: uniform, kept in an SGPR
  const int qg = w % QG, part = w / QG;
  int bh, qt;
  tile_of_block_banded(blockIdx.x, BH, n_qtiles, CAUSAL, CAUSAL ? band : 0, bh, qt);
  const Rows rw = rows_of(bh, H, S, D, seq_major);
  const int64_t base = rw.base;
  const int rs = rw.rs;
  const bf16* Kb = K + base;
  const bf16* Vb = V + base;
  const int Sp = ws_rows(S);

  const int q0 = qt * BQ, qw = q0 + 32 * qg, my_q = qw + r;
  const int kend = CAUSAL && !kNoClamp ? min(S, q0 + BQ) : S;
  const int n = (kend + 31) / 32;          // 32-key tiles of the workgroup
  const int L = (n + SPLIT - 1) / SPLIT;   // tiles per part (the last may be short)
  const int kend_w = qw >= S ? 0 : (CAUSAL && !kNoClamp ? min(S, qw + 32) : S);
  const int nsb = (kend_w + 31) / 32;      // tiles this wave's queries need
  const int tb = part * L;                 // this wave's tiles: [tb, te)
  const int te = min(nsb, min(n, tb + L));
  const int cnt = te > tb ? te - tb : 0;

  const int n_last = n - (SPLIT - 1) * L;  // tiles of the last part (<= L)
  // the key tile that holds the ragged end of the sequence, if this workgroup copies one
  const int t_rag = RAG && (S - 1) / 32 < n ? (S - 1) / 32 : -1;
  // the iteration (in this wave's part) whose tile must be masked: the wave's
  // last tile when it straddles the causal diagonal or the end of the sequence
  // (without the clamp, every tile from the one holding the diagonal on: i >= i_mask)
  const int i_mask = CAUSAL && kNoClamp ? qw / 32 - tb
                     : nsb > 0 && ((CAUSAL && (nsb - 1) * 32 + 31 > qw) || nsb * 32 > S) ? nsb - 1 - tb : -1;

  TileCopy<D> tc;
  tc.init(w, lane, rs);
  auto dma = [&](int x, auto slc) {  // iteration x's tile of every part, into ring slot slc
#pragma unroll
    for (int p = 0; p < SPLIT; ++p) {
      if (p < SPLIT - 1 || x < n_last) {
        const int t = p * L + x;
        char* dst = smem + (p * NB + decltype(slc)::value) * SET;
        if (!RAG || t != t_rag) {
          tc.copy_full(Kb, t * 32, dst);
          tc.copy_full(Vb, t * 32, dst + TILE);
        } else {
          tc.copy(Kb, t * 32, S, dst);
          tc.copy(Vb, t * 32, S, dst + TILE);
        }
      }
    }
  };
  constexpr int NEED = 0;  // iteration i reads the tiles of iterations i .. i+NEED
  constexpr int GROUP = ring_group(SPLIT, NB, NEED, kDqGroup);  // iterations per barrier
  ring_prologue<NB, GROUP>(L, dma);
  MB::frag qf[KS_D], dof[KS_D], of[KS_D];
  load_row_frags<bf16, D>(Q + base, my_q, S, h, rs, qf);
  load_row_frags<bf16, D>(dO + base, my_q, S, h, rs, dof);
  load_row_frags<bf16, D>(O + base, my_q, S, h, rs, of);
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
  if (part == 0 && h == 0 && my_q < Sp) {  // workspace of this head: D row, then -LSE/scale row
    float* wsh = ws + (int64_t)bh * 2 * Sp;
    wsh[my_q] = my_q < S ? Dq : 0.f;
    wsh[Sp + my_q] = my_q < S ? -lse / scale : 0.f;
  }
#pragma unroll
  for (int ks = 0; ks < KS_D; ++ks) dof[ks] = negated(dof[ks]);
  f32x16 dinit;
#pragma unroll
  for (int a = 0; a < 16; ++a) dinit[a] = Dq;

  f32x16 dqacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) dqacc[dt] = f32x16{};
  const char* ring = smem + part * NB * SET;  // this wave's part
  // STR (unsplit grids at D = 64 with at least four work groups per CU):
  // every K, V and K^T fragment is read one contraction step before its use
  // instead of a whole tile's at once, and D is broadcast into the dP
  // accumulator in each iteration; the registers that saves give four waves
  // per SIMD (124 registers).  Grids of up to about three work groups per CU
  // run faster with the whole-tile reads at three waves per SIMD.
  static_assert(!STR || (SPLIT == 1 && D == 64), "streamed form: unsplit, D = 64");
  auto rowf = [&](const char* t, int ks) { return read_row_frag<bf16, D>(t, r, ks, h); };
  auto trf = [&](const char* t, int ks, int dt) { return TransRead<bf16, D>::read(t, 0, ks, dt * 32, lane); };

  for (int i0 = 0; i0 < L; i0 += NB) {
    unroll<NB>([&](auto slc) {
      constexpr int sl = decltype(slc)::value;
      const int i = i0 + sl;
      if (i >= L) return;
      ring_step<NB, GROUP, NEED, SPLIT, PER_TILE, sl>(i, L, n_last, dma);
      if (i >= cnt) return;  // wave-uniform: this wave is done, it only keeps the barriers
      const int j = tb + i;  // key tile of this iteration
      const char* cur = ring + sl * SET;
      if constexpr (STR) {
        // D broadcast into the dP accumulator here, not kept in 16 registers
        // across the loop (the empty asm stops the compiler from hoisting it)
        float dq_ = Dq;
        asm volatile("" : "+v"(dq_));
        f32x16 s = f32x16{}, dx;
#pragma unroll
        for (int a = 0; a < 16; ++a) dx[a] = dq_;
        MB::frag ka[2], va[2];
        ka[0] = rowf(cur, 0);
        va[0] = rowf(cur + TILE, 0);
#pragma unroll
        for (int ks = 0; ks < KS_D; ++ks) {
          if (ks + 1 < KS_D) {
            ka[(ks + 1) & 1] = rowf(cur, ks + 1);
            va[(ks + 1) & 1] = rowf(cur + TILE, ks + 1);
          }
          s = MB::run(ka[ks & 1], qf[ks], s);
          dx = MB::run(va[ks & 1], dof[ks], dx);  // D - dP^T
        }
        if (CAUSAL && kNoClamp ? i >= i_mask : i == i_mask) {
          const int k0 = j * 32;
#pragma unroll
          for (int a = 0; a < 16; ++a) {
            const int key = k0 + acc_row(a, h);
            if ((RAG && key >= S) || (CAUSAL && key > my_q)) s[a] = kMasked;
          }
        }
#pragma unroll
        for (int a = 0; a < 16; ++a) {
          const float p = exp2_hw(fmaf(s[a], c, -lse2));
          dx[a] = -p * dx[a];  // dS^T = P (dP - D)
        }
        const MB::frag db[2] = {MB::pack(dx, 0), MB::pack(dx, 1)};
        MB::frag ta[2];
        ta[0] = trf(cur, 0, 0);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            const int x = ks * DT + dt;
            if (x + 1 < 2 * DT) ta[(x + 1) & 1] = trf(cur, (x + 1) / DT, (x + 1) % DT);
            dqacc[dt] = MB::run(ta[x & 1], db[ks], dqacc[dt]);
          }
        return;
      }
      // split grids read the whole tile's fragments here
      MB::frag kf[KS_D], vfr[KS_D];
      read_rows<D>(cur, r, h, kf);
      read_rows<D>(cur + TILE, r, h, vfr);
      MB::frag ktr[2][DT];
      read_trans<D>(cur, lane, ktr);
      f32x16 s = f32x16{}, dx = dinit;
#pragma unroll
      for (int ks = 0; ks < KS_D; ++ks) {
        s = MB::run(kf[ks], qf[ks], s);
        dx = MB::run(vfr[ks], dof[ks], dx);  // D - dP^T
      }
      if (CAUSAL && kNoClamp ? i >= i_mask : i == i_mask) {
        const int k0 = j * 32;
#pragma unroll
        for (int a = 0; a < 16; ++a) {
          const int key = k0 + acc_row(a, h);
          if ((RAG && key >= S) || (CAUSAL && key > my_q)) s[a] = kMasked;
        }
      }
#pragma unroll
      for (int a = 0; a < 16; ++a) {
        const float p = exp2_hw(fmaf(s[a], c, -lse2));
        dx[a] = -p * dx[a];  // dS^T = P (dP - D)
      }
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const MB::frag db = MB::pack(dx, ks);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) dqacc[dt] = MB::run(ktr[ks][dt], db, dqacc[dt]);
      }
    });
  }

  if constexpr (SPLIT == 2) {
    // Add the two key parts of each query group: part 1 hands dQ to part 0
    // through LDS, lane to lane (both waves share the same lane layout).
    wait_vm(0);
    __syncthreads();  // every wave is done with the rings
    float* xb = (float*)smem + (size_t)qg * 64 * (DT * 16);
    if (part == 1) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int a = 0; a < 16; ++a) xb[(dt * 16 + a) * 64 + lane] = dqacc[dt][a];
    }
    __syncthreads();
    if (part == 1) return;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int a = 0; a < 16; ++a) dqacc[dt][a] += xb[(dt * 16 + a) * 64 + lane];
  }

  if (my_q < S) {
    bf16* row = dQ + base + (int64_t)my_q * rs;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        store4<bf16>(row + dt * 32 + 8 * g + 4 * h, dqacc[dt][4 * g] * scale, dqacc[dt][4 * g + 1] * scale,
                     dqacc[dt][4 * g + 2] * scale, dqacc[dt][4 * g + 3] * scale);
  }
}

// ---------------------------------------------------------------------------
// Backward, kernel 2: dK, dV (reduces over queries).  Both score contractions
// start from per-query values copied to LDS with the tile: S from -LSE/scale
// (so P = exp2(scale*log2e * acc)) and dP, multiplied by -V, from D (so the
// contraction yields D - dP).
//
// A workgroup owns 32*KG keys of one (batch, head), KG = 4/SPLIT key groups of
// 32 (one per wave), and splits the query tiles it must visit into SPLIT
// consecutive parts: wave w takes key group w % KG and query part w / KG.
// Each part streams its own ring of Q/dO tiles, so the sequential chain of a
// wave is 1/SPLIT of the query range (the heaviest causal key tile sees every
// query tile).  With SPLIT = 2 the partial dK, dV of the two parts are added
// lane to lane through LDS at the end (fixed order: deterministic, no atomics).
//
// Every per-iteration decision is a compare against an index computed once
// per wave (the first and last active iteration, the one holding the causal
// diagonal, the ragged tile), and every wave issues the same copies per tile,
// so that the common wait at the barrier is a compile-time count.
// ---------------------------------------------------------------------------
// dK/dV at D = 64, unsplit: operands read where they are used instead of one
// tile ahead, which gives three waves per SIMD.  At D = 128 (STREAM below) each
// operand fragment is read one contraction step before its use, which gives
// two; split grids at D = 64 read the next tile's rows one tile ahead.
template <int D, bool CAUSAL, int SPLIT, int NB>
constexpr bool dkdv_lean() {
  return D == 64 && SPLIT == 1;
}
template <int D, bool CAUSAL, int SPLIT, int NB, bool RAG>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(dkdv_lean<D, CAUSAL, SPLIT, NB>() ? 3 : (D == 128 ? 2 : 1), 10)))
void attn_bwd_dkdv_bf16_kernel(const bf16* __restrict__ Q,
                                                                 const bf16* __restrict__ K,
                                                                 const bf16* __restrict__ V,
                                                                 const bf16* __restrict__ dO,
                                                                 const float* __restrict__ ws,
                                                                 bf16* __restrict__ dK, bf16* __restrict__ dV, int S,
                                                                 int BH, int n_ktiles, float c, float scale, int band,
                                                                 int H, int seq_major) {
  typedef TileGeom<D> G;
  constexpr bool LEAN = dkdv_lean<D, CAUSAL, SPLIT, NB>();
  // D = 128: every operand fragment read from LDS one contraction step before
  // its use, so that the K, V, dK and dV fragments (192 registers) and the two
  // score blocks leave room for two waves per SIMD
  constexpr bool STREAM = D == 128 && SPLIT == 1;
  constexpr int KG = 4 / SPLIT, BKV = 32 * KG;
  constexpr int TILE = G::TILE;
  constexpr int KS_D = D / 16, DT = D / 32;
  // LDS: the Q and dO tiles of every slot first, then the 32 floats of
  // -LSE/scale and the 32 of D of every slot, so that every tile read of the
  // ring lies within the 64 KB an LDS instruction's immediate offset reaches
  // from one per-lane base address (one address register per fragment for
  // all slots: at D = 128 this keeps the kernel at two waves per SIMD).
  constexpr int SETB = 2 * TILE, AUX = 2 * 32 * 4, AUX0 = SPLIT * NB * SETB;
  constexpr int BUF = SETB + AUX;
  // copies per part tile issued by every wave: its share of Q and dO, and 4 of the 16 LSE/D chunks
  constexpr int PER_TILE = 2 * G::DMA_PER_TENSOR + 1;
  // [part][slot] Q, dO tiles, then [part][slot] -LSE/scale and D rows
  __shared__ __attribute__((aligned(16))) char smem[SPLIT * NB * BUF];
  static_assert(SPLIT == 1 || KG * 64 * (4 * DT * 16) * 4 <= SPLIT * NB * BUF, "merge area");
  static_assert(!STREAM || AUX0 <= 65536, "tile reads reach every slot by immediate offset");

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index: uniform, kept in an SGPR
  const int kg = w % KG, part = w / KG;
  int bh, kt;
  tile_of_block_banded(blockIdx.x, BH, n_ktiles, false, CAUSAL ? band : 0, bh, kt);
  const Rows rw = rows_of(bh, H, S, D, seq_major);
  const int64_t base = rw.base;
  const int rs = rw.rs;
  const bf16* Qb = Q + base;
  const bf16* dOb = dO + base;
  const int Sp = ws_rows(S);
  const float* wsh = ws + (int64_t)bh * 2 * Sp;  // D row, then -LSE/scale row
  // The 16 chunks of 4 floats that follow a Q/dO tile in LDS -- 8 of
  // -LSE/scale, then 8 of D -- are copied by lanes 0..3 of every wave: chunk
  // q = 4w + lane (rows < Sp: in bounds).
  const int ldq = 4 * w + (lane & 3);
  const unsigned ld_voff = (unsigned)((ldq < 8 ? Sp + 4 * ldq : 4 * (ldq - 8)) * 4);

  const int k0 = kt * BKV, kw = k0 + 32 * kg, my_k = kw + r;
  // 32-query tiles of the workgroup: from the one holding k0 (causal: the loop's
  // lower bound is raised to the diagonal) to the end of the sequence, walked
  // from the LAST tile down (walk position t holds query tile nt - 1 - t).  The
  // work groups of one head then start on the same tile and stream the same
  // Q/dO tiles at about the same time, so that one HBM fetch of a tile serves
  // all of them from L2; the masked diagonal tile comes last.
  const int nt = (S + 31) / 32;                 // query tiles of the sequence
  const int jt0 = CAUSAL && !kNoClamp ? k0 / 32 : 0;
  const int n = nt - jt0;
  const int L = (n + SPLIT - 1) / SPLIT;        // iterations; part p owns walk positions [p*L, min(n, p*L + L))
  const int n_last = n - (SPLIT - 1) * L;       // tiles of the last part (<= L)
  const int jb = CAUSAL && !kNoClamp ? kw / 32 : 0;  // this wave's first query tile
  const int je = kw >= S ? jb : nt;             // ... and one past its last
  const int tb = part * L;                      // this wave's part starts at walk position tb
  // iteration indices, relative to this wave's part: the wave's tiles jb .. je-1
  // sit at walk positions nt - je .. nt - 1 - jb
  const int i_lo = max(0, nt - je - tb);                                             // first active
  const int i_span = max(0, min(part == SPLIT - 1 ? n_last : L, nt - jb - tb) - i_lo);  // active count
  // causal diagonal (without the clamp, the tiles before it come after it in the walk: i >= i_diag)
  const int i_diag = CAUSAL ? nt - 1 - kw / 32 - tb : -1;
  const int t_rag = RAG ? 0 : -1;               // walk position of the ragged (last) tile
  const int i_rag = t_rag - tb;                  // ... in this part
  // copies: iteration x of the ring holds walk position p*L + x of every part p with x < L (x < n_last for the last)

  TileCopy<D> tc;
  tc.init(w, lane, rs);
  auto dma = [&](int x, auto slc) {  // iteration x's tile of every part, into ring slot slc
#pragma unroll
    for (int p = 0; p < SPLIT; ++p) {
      if (p < SPLIT - 1 || x < n_last) {
        const int t = p * L + x;
        const int row0 = (nt - 1 - t) * 32;
        char* b = smem + (p * NB + decltype(slc)::value) * SETB;
        if (!RAG || t != t_rag) {
          tc.copy_full(Qb, row0, b);
          tc.copy_full(dOb, row0, b + TILE);
        } else {
          tc.copy(Qb, row0, S, b);
          tc.copy(dOb, row0, S, b + TILE);
        }
        if (lane < 4) dma16(wsh + row0, ld_voff, lds_addr(smem + AUX0 + (p * NB + decltype(slc)::value) * AUX) + 64 * w);
      }
    }
  };
  constexpr int NEED = LEAN || STREAM ? 0 : 1;  // iteration i reads the tiles of iterations i .. i+NEED
  // With one part, the waves meet at a barrier every GROUP iterations: a wave
  // that runs late on its SIMD then holds the others back less often.
  constexpr int GROUP = ring_group(SPLIT, NB, NEED, kDkdvGroup);
  ring_prologue<NB, GROUP>(L, dma);
  MB::frag kf[KS_D], vf[KS_D];
  load_row_frags<bf16, D>(K + base, my_k, S, h, rs, kf);
  load_row_frags<bf16, D>(V + base, my_k, S, h, rs, vf);
  wait_vm(0);
  __syncthreads();
#pragma unroll
  for (int ks = 0; ks < KS_D; ++ks) vf[ks] = negated(vf[ks]);

  f32x16 dkacc[DT], dvacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) {
    dkacc[dt] = f32x16{};
    dvacc[dt] = f32x16{};
  }
  MB::frag qf[KS_D], dof[KS_D];  // row fragments of the current sub-block
  Frag128 fo;
  if constexpr (STREAM) fo.init(r, h, lane);
  const char* ring = smem + part * NB * SETB;
  const char* aux = smem + AUX0 + part * NB * AUX;

  for (int i0 = 0; i0 < L; i0 += NB) {
    unroll<NB>([&](auto slc) {
      constexpr int sl = decltype(slc)::value, sn = (sl + 1) % NB;
      const int i = i0 + sl;
      if (i >= L) return;
      ring_step<NB, GROUP, NEED, SPLIT, PER_TILE, sl>(i, L, n_last, dma);
      if ((unsigned)(i - i_lo) >= (unsigned)i_span) return;  // wave-uniform: not an active sub-block
      const char* lq = ring + sl * SETB;
      const char* ldo = lq + TILE;
      const float* llse = (const float*)(aux + sl * AUX);
      const float* ld = llse + 32;
      MB::frag dotr[2][DT], qtr[2][DT];
      MB::frag qn[KS_D], don[KS_D];  // next tile of the part (on a wave's last tile: discarded)
      if constexpr (LEAN) {
        read_rows<D>(lq, r, h, qf);
        read_rows<D>(ldo, r, h, dof);
      } else if constexpr (!STREAM) {
        if (i == i_lo) {  // a wave's first sub-block: read it here
          read_rows<D>(lq, r, h, qf);
          read_rows<D>(ldo, r, h, dof);
        }
        read_trans<D>(ldo, lane, dotr);
        read_trans<D>(lq, lane, qtr);
        read_rows<D>(ring + sn * SETB, r, h, qn);
        read_rows<D>(ring + sn * SETB + TILE, r, h, don);
      }
      f32x16 s, dx;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 l4 = *(const f32x4*)(llse + 8 * g + 4 * h);
        const f32x4 d4 = *(const f32x4*)(ld + 8 * g + 4 * h);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          s[4 * g + e] = l4[e];
          dx[4 * g + e] = d4[e];
        }
      }
      if constexpr (STREAM) {
        MB::frag qa[2], da[2];
        qa[0] = fo.row_frag(lq, 0);
        da[0] = fo.row_frag(ldo, 0);
#pragma unroll
        for (int ks = 0; ks < KS_D; ++ks) {
          if (ks + 1 < KS_D) {
            qa[(ks + 1) & 1] = fo.row_frag(lq, ks + 1);
            da[(ks + 1) & 1] = fo.row_frag(ldo, ks + 1);
          }
          s = MB::run(qa[ks & 1], kf[ks], s);
          dx = MB::run(da[ks & 1], vf[ks], dx);  // D - dP
        }
      } else {
#pragma unroll
        for (int ks = 0; ks < KS_D; ++ks) {
          s = MB::run(qf[ks], kf[ks], s);
          dx = MB::run(dof[ks], vf[ks], dx);  // D - dP
        }
      }
      // s[a], dx[a]: S - LSE/scale and D - dP of query 32j + acc_row(a, h), key my_k
      if ((CAUSAL && kNoClamp ? i >= i_diag : i == i_diag) || (RAG && i == i_rag)) {  // diagonal or ragged end
        const int qs = (nt - 1 - tb - i) * 32;
#pragma unroll
        for (int a = 0; a < 16; ++a) {
          const int qry = qs + acc_row(a, h);
          if ((RAG && qry >= S) || (CAUSAL && my_k > qry)) s[a] = kMasked;
        }
      }
#pragma unroll
      for (int a = 0; a < 16; ++a) {
        const float p = exp2_hw(s[a] * c);
        s[a] = p;
        dx[a] = -p * dx[a];  // dS = P (dP - D)
      }
      if constexpr (LEAN) {
        read_trans<D>(ldo, lane, dotr);
        read_trans<D>(lq, lane, qtr);
      }
      if constexpr (STREAM) {
        // P and dS packed first, so that their float forms are dead before the
        // transposed fragments are read
        const MB::frag pb[2] = {MB::pack(s, 0), MB::pack(s, 1)};
        const MB::frag db[2] = {MB::pack(dx, 0), MB::pack(dx, 1)};
        MB::frag ta[2], tq[2];
        ta[0] = fo.trans(ldo, 0, 0);
        tq[0] = fo.trans(lq, 0, 0);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            const int x = ks * DT + dt;
            if (x + 1 < 2 * DT) {
              const int ks1 = (x + 1) / DT, dt1 = (x + 1) % DT;
              ta[(x + 1) & 1] = fo.trans(ldo, ks1, dt1);
              tq[(x + 1) & 1] = fo.trans(lq, ks1, dt1);
            }
            dvacc[dt] = MB::run(ta[x & 1], pb[ks], dvacc[dt]);
            dkacc[dt] = MB::run(tq[x & 1], db[ks], dkacc[dt]);
          }
        }
      } else {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const MB::frag pb = MB::pack(s, ks);
          const MB::frag db = MB::pack(dx, ks);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            dvacc[dt] = MB::run(dotr[ks][dt], pb, dvacc[dt]);
            dkacc[dt] = MB::run(qtr[ks][dt], db, dkacc[dt]);
          }
        }
      }
      if constexpr (!LEAN && !STREAM) {
#pragma unroll
        for (int ks = 0; ks < KS_D; ++ks) {
          qf[ks] = qn[ks];
          dof[ks] = don[ks];
        }
      }
    });
  }

  if constexpr (SPLIT == 2) {
    // Add the two query parts of each key group: part 1 hands (dK, dV) to
    // part 0 through LDS, lane to lane (both waves share the same lane layout).
    wait_vm(0);
    __syncthreads();  // every wave is done with the rings
    float* xb = (float*)smem + (size_t)kg * 64 * (4 * DT * 16);
    if (part == 1) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int a = 0; a < 16; ++a) {
          xb[(dt * 16 + a) * 64 + lane] = dkacc[dt][a];
          xb[((DT + dt) * 16 + a) * 64 + lane] = dvacc[dt][a];
        }
    }
    __syncthreads();
    if (part == 1) return;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int a = 0; a < 16; ++a) {
        dkacc[dt][a] += xb[(dt * 16 + a) * 64 + lane];
        dvacc[dt][a] += xb[((DT + dt) * 16 + a) * 64 + lane];
      }
  }

  if (my_k < S) {
    bf16* krow = dK + base + (int64_t)my_k * rs;
    bf16* vrow = dV + base + (int64_t)my_k * rs;
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
// Compute units of the current device (queried once per device).
static int cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

// Forward ring depths: per key part when the key range is split in two (two
// rings of 3 fit the LDS budget of three workgroups per CU), and unsplit.
template <int D> struct FwdCfg {
  static constexpr int NB_SPLIT = kFwdNbSplit;
  static constexpr int NB = D == 64 ? kFwdNb64 : kFwdNb128;
};
template <int D> struct BwdCfg {
  static constexpr int NB = D == 64 ? kBwdNb64 : kBwdNb128;
};

template <int D, bool CAUSAL, int SPLIT, int NB, bool RAG, bool STR>
static hipError_t launch_dq_t(const BwdArgs& a, float c, int n_qtiles, hipStream_t st) {
  hipLaunchKernelGGL((attn_bwd_dq_bf16_kernel<D, CAUSAL, SPLIT, NB, RAG, STR>),
                     dim3((unsigned)((int64_t)a.BH * n_qtiles)), dim3(256), 0, st, (const bf16*)a.q,
                     (const bf16*)a.k, (const bf16*)a.v, (const bf16*)a.o, (const bf16*)a.dout, a.lse, (bf16*)a.dq,
                     a.ws, a.S, a.BH, n_qtiles, c, a.scale, cu_count(), a.H, (int)a.seq_major);
  return hipGetLastError();
}

template <int D, bool CAUSAL, int SPLIT, int NB, bool RAG>
static hipError_t launch_dq(const BwdArgs& a, float c, hipStream_t st) {
  constexpr int BQ = 128 / SPLIT;
  const int n_qtiles = (a.S + BQ - 1) / BQ;
  if constexpr (D == 64 && SPLIT == 1) {
    if ((int64_t)a.BH * n_qtiles >= 4 * (int64_t)cu_count())
      return launch_dq_t<D, CAUSAL, SPLIT, NB, RAG, true>(a, c, n_qtiles, st);
  }
  return launch_dq_t<D, CAUSAL, SPLIT, NB, RAG, false>(a, c, n_qtiles, st);
}

template <int D, bool CAUSAL, int SPLIT, int NB, bool RAG>
static hipError_t launch_dkdv(const BwdArgs& a, float c, hipStream_t st) {
  constexpr int BKV = 128 / SPLIT;
  const int n_ktiles = (a.S + BKV - 1) / BKV;
  // dealt in alternating directions only when every work group is resident
  // from the start (three per CU)
  const int band = dkdv_lean<D, CAUSAL, SPLIT, NB>() && (int64_t)a.BH * n_ktiles <= 3 * (int64_t)cu_count()
                       ? cu_count() : 0;
  hipLaunchKernelGGL((attn_bwd_dkdv_bf16_kernel<D, CAUSAL, SPLIT, NB, RAG>), dim3((unsigned)((int64_t)a.BH * n_ktiles)),
                     dim3(256), 0, st, (const bf16*)a.q, (const bf16*)a.k, (const bf16*)a.v, (const bf16*)a.dout,
                     (const float*)a.ws, (bf16*)a.dk, (bf16*)a.dv, a.S, a.BH, n_ktiles, c, a.scale,
                     band, a.H, (int)a.seq_major);
  return hipGetLastError();
}

template <int D, bool CAUSAL, int SPLIT, int NB, bool RAG>
static hipError_t launch_fwd_split(const FwdArgs& a, hipStream_t st) {
  constexpr int BQ = 128 / SPLIT;
  const int n_qtiles = (a.S + BQ - 1) / BQ;
  hipLaunchKernelGGL((attn_fwd_bf16_kernel<D, CAUSAL, SPLIT, NB, RAG>), dim3((unsigned)((int64_t)a.BH * n_qtiles)),
                     dim3(256), 0, st, (const bf16*)a.q, (const bf16*)a.k, (const bf16*)a.v, (bf16*)a.o, a.lse, a.S,
                     a.BH, n_qtiles, a.scale * kLog2e, cu_count(), a.H, (int)a.seq_major);
  return hipGetLastError();
}

template <int D, bool CAUSAL, bool RAG>
static hipError_t fwd_bf16_t(const FwdArgs& a, hipStream_t st) {
  if constexpr (D == 64) {
    // Split each query tile's key range over two parts when the unsplit grid
    // (128-query tiles) cannot fill the GPU's workgroup slots (three per CU).
    // (The no-clamp test build never splits: a split part would then start on
    // tiles that are fully masked for its queries, with no real score to set
    // the softmax offset from.)
    const bool split = !kNoClamp && (int64_t)a.BH * ((a.S + 127) / 128) < 3 * (int64_t)cu_count();
    if (split) return launch_fwd_split<D, CAUSAL, 2, FwdCfg<D>::NB_SPLIT, RAG>(a, st);
  }
  return launch_fwd_split<D, CAUSAL, 1, FwdCfg<D>::NB, RAG>(a, st);
}

// The kernels come in two builds: with the ragged-end handling (S not a
// multiple of 32: the last tile's rows past S are masked and copied from row
// S - 1) and without it, so that whole tiles carry no per-tile test for it.
template <int D, bool CAUSAL>
static hipError_t fwd_bf16_r(const FwdArgs& a, hipStream_t st) {
  return a.S % 32 ? fwd_bf16_t<D, CAUSAL, true>(a, st) : fwd_bf16_t<D, CAUSAL, false>(a, st);
}

hipError_t launch_fwd_bf16(const FwdArgs& a, hipStream_t st) {
  if (a.D == 64) return a.causal ? fwd_bf16_r<64, true>(a, st) : fwd_bf16_r<64, false>(a, st);
  return a.causal ? fwd_bf16_r<128, true>(a, st) : fwd_bf16_r<128, false>(a, st);
}

template <int D, bool CAUSAL, bool RAG>
static hipError_t bwd_bf16_t(const BwdArgs& a, int phase, hipStream_t st) {
  constexpr int NB = BwdCfg<D>::NB;
  const float c = a.scale * kLog2e;
  // Split the key range of a query tile (dQ), or the query range of a key tile
  // (dK/dV), over two parts when the unsplit grid cannot fill the GPU's
  // workgroup slots (two per CU): the heaviest causal tile's sequential chain
  // then sets the time.  With a full grid the unsplit kernels have less
  // overhead per unit of work.
  bool split = false;
  if constexpr (D == 64)
    split = !kNoClamp && (int64_t)a.BH * ((a.S + 127) / 128) < kBwdSplitWgPerCu * (int64_t)cu_count();
  if (phase != 2) {
    hipError_t e;
    if constexpr (D == 64) {
      e = split ? launch_dq<D, CAUSAL, 2, kBwdNbSplit, RAG>(a, c, st) : launch_dq<D, CAUSAL, 1, NB, RAG>(a, c, st);
    } else {
      e = launch_dq<D, CAUSAL, 1, NB, RAG>(a, c, st);
    }
    if (e != hipSuccess || phase == 1) return e;
  }
  if constexpr (D == 64) {
    if (split) return launch_dkdv<D, CAUSAL, 2, kBwdNbSplit, RAG>(a, c, st);
  }
  return launch_dkdv<D, CAUSAL, 1, BwdCfg<D>::NB, RAG>(a, c, st);
}

template <int D, bool CAUSAL>
static hipError_t bwd_bf16_r(const BwdArgs& a, int phase, hipStream_t st) {
  return a.S % 32 ? bwd_bf16_t<D, CAUSAL, true>(a, phase, st) : bwd_bf16_t<D, CAUSAL, false>(a, phase, st);
}

hipError_t launch_bwd_bf16(const BwdArgs& a, int phase, hipStream_t st) {
  if (a.D == 64) return a.causal ? bwd_bf16_r<64, true>(a, phase, st) : bwd_bf16_r<64, false>(a, phase, st);
  return a.causal ? bwd_bf16_r<128, true>(a, phase, st) : bwd_bf16_r<128, false>(a, phase, st);
}

}  // namespace cattn
