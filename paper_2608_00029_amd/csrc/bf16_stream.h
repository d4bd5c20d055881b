// Streaming building blocks of the bf16 kernels for gfx950: HBM -> LDS tile
// copies (global_load_lds_dwordx4 through a ring of LDS slots, with explicit
// vmcnt waits and plain barriers), row-major and transposed MFMA operand
// fragments read from the swizzled LDS tiles, and compile-time unrolling.
// Shared by the attention kernels (attn_bf16.hip) and the loss-head kernel
// (lmhead_bf16.hip).
#pragma once

#include <stdint.h>

#include <utility>

#include "attn_device.h"

namespace cattn {

typedef __bf16 bf16;
typedef Mma<bf16> MB;
template <int N> using IC = std::integral_constant<int, N>;


// f(IC<0>{}), f(IC<1>{}), ..., f(IC<N-1>{}), in order.
template <typename F, int... I>
__device__ __forceinline__ void unroll_each(F& f, std::integer_sequence<int, I...>) {
  (f(IC<I>{}), ...);
}
template <int N, typename F> __device__ __forceinline__ void unroll(F&& f) {
  unroll_each(f, std::make_integer_sequence<int, N>{});
}

template <int D> struct TileGeom {
  static constexpr int TILE = 32 * D * 2;                 // bytes of one tensor's 32-row tile
  static constexpr int CPR = D * 2 / 16;                  // 16-byte chunks per row
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

// tile_barrier(N) for a compile-time N: a single s_waitcnt.
template <int N> __device__ __forceinline__ void tile_barrier_c() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0070 | (N & 15) | ((N >> 4) << 14));
  asm volatile("s_barrier" ::: "memory");
}

// The ring protocol at the top of iteration i (ring slot SL = i % NB, every
// part's tile x in slot x % NB): wait for the tiles this iteration (or group
// of GROUP iterations) reads, meet the other waves, then copy the tiles the
// slots freed by the barrier take next.  GROUP == 1: every iteration, tile
// i + NB - 1 (ring_in_flight counts what may stay in flight); GROUP > 1: at
// the first iteration of each group, tiles i + NB - GROUP .. i + NB - 1
// (ring_group_in_flight).  dma(x, IC<slot>) copies iteration x's tiles;
// every wave issues PER_TILE copies per tile and part.  The tiles before the
// loop come from ring_prologue.
template <int NB, int GROUP, int NEED, int SPLIT, int PER_TILE, int SL, typename Dma>
__device__ __forceinline__ void ring_step(int i, int L, int n_last, Dma& dma) {
  constexpr int AH = NB - 1;
  if constexpr (GROUP == 1) {
    if (i > 0) {
      if (i + AH - 1 < n_last) {
        tile_barrier_c<ring_in_flight_full(SPLIT, AH, NEED) * PER_TILE>();
      } else {
        tile_barrier(ring_in_flight(i, L, n_last, SPLIT, AH, NEED) * PER_TILE);
      }
    }
    if (i + AH < L) dma(i + AH, IC<(SL + AH) % NB>{});
  } else if constexpr (SL % GROUP == 0) {
    static_assert(SPLIT == 1 && NB % GROUP == 0 && NB >= 2 * GROUP + NEED, "grouped ring");
    if (i > 0) {
      if (i + NB - 1 < L) {
        tile_barrier_c<ring_group_in_flight(0, 1 << 20, NB, GROUP, NEED) * PER_TILE>();
      } else {
        tile_barrier(ring_group_in_flight(i, L, NB, GROUP, NEED) * PER_TILE);
      }
    }
    unroll<GROUP>([&](auto g) {
      constexpr int x = NB - GROUP + decltype(g)::value;
      if (i + x < L) dma(i + x, IC<(SL + x) % NB>{});
    });
  }
}
template <int NB, int GROUP, typename Dma> __device__ __forceinline__ void ring_prologue(int L, Dma& dma) {
  unroll<NB - GROUP>([&](auto I) {
    if (decltype(I)::value < L) dma(decltype(I)::value, I);
  });
}

// Byte address of an LDS location (the value M0 takes).
__device__ __forceinline__ unsigned lds_addr(const char* p) {
  return (unsigned)(uintptr_t)(__attribute__((address_space(3))) const char*)p;
}

// One 16-byte HBM -> LDS copy per active lane: lane i copies the 16 bytes at
// sbase + voff (sbase wave-uniform, in scalar registers) to LDS byte address
// lds + 16 * i.  Issued as inline assembly so that the compiler does not treat
// every later LDS read as aliasing the copy in flight (it would then wait for
// the copy before each read); completion is awaited explicitly (wait_vm /
// tile_barrier) before the barrier that publishes a tile.
// M0 is a reserved register to the compiler, which warns about the clobber;
// the clobber is what keeps it from assuming M0 survives the statement.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void* sbase, unsigned voff, unsigned lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds), "v"(voff), "s"(sbase)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// HBM -> LDS copy of 32-row tiles of an [S][D] bf16 matrix whose rows are rs elements apart.  The
// chunk a lane deposits at physical position p of the tile is logical chunk
// p ^ swz(row), so the LDS image has the swizzled layout Tile<> reads.  The
// per-lane source offsets inside a tile are fixed for the kernel; only the
// ragged last tile (rows >= nrows are read from row nrows - 1) recomputes them.
template <int D> struct TileCopy {
  typedef TileGeom<D> G;
  unsigned voff[G::DMA_PER_TENSOR];
  int w, lane, rs;
  __device__ __forceinline__ void init(int w_, int lane_, int rs_) {
    w = w_;
    lane = lane_;
    rs = rs_;
#pragma unroll
    for (int i = 0; i < G::DMA_PER_TENSOR; ++i) {
      const int p = i * 256 + w * 64 + lane;
      const int row = p / G::CPR;
      voff[i] = (unsigned)(row * rs * 2 + (((p % G::CPR) ^ swz(row)) << 4));
    }
  }
  // a tile known to lie inside the sequence (row0 + 32 <= nrows)
  __device__ __forceinline__ void copy_full(const bf16* g, int row0, char* lds) const {
    const bf16* src = g + (int64_t)row0 * rs;
    const unsigned dst = lds_addr(lds) + w * 64 * 16;
#pragma unroll
    for (int i = 0; i < G::DMA_PER_TENSOR; ++i) dma16(src, voff[i], dst + i * 256 * 16);
  }
  __device__ __forceinline__ void copy(const bf16* g, int row0, int nrows, char* lds) const {
    const bf16* src = g + (int64_t)row0 * rs;
    const unsigned dst = lds_addr(lds) + w * 64 * 16;
    if (row0 + 32 <= nrows) {
#pragma unroll
      for (int i = 0; i < G::DMA_PER_TENSOR; ++i) dma16(src, voff[i], dst + i * 256 * 16);
    } else {
#pragma unroll
      for (int i = 0; i < G::DMA_PER_TENSOR; ++i) {
        const int p = i * 256 + w * 64 + lane;
        const int row = p / G::CPR, lc = (p % G::CPR) ^ swz(row);
        const int src_row = min(row, nrows - 1 - row0);
        dma16(src, (unsigned)(src_row * rs * 2 + lc * 16), dst + i * 256 * 16);
      }
    }
  }
};

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

// Fragment reads of a D = 128 tile from per-lane offsets computed once.  The
// swizzle permutes only bits 0-2 of a row's 16-byte chunk index, so chunk bit 3
// -- row fragments ks >= 4, transposed fragments of columns 64.. -- is a fixed
// 128-byte step: 4 offsets serve the 8 row fragments and 8 the 16 transposed
// halves, each read an offset register plus an immediate (the compiler would
// otherwise keep one address register per fragment and per ring slot).
struct Frag128 {
  typedef Tile<__bf16, 128> T;
  static_assert(T::kChunks == 16, "row of 16 chunks");
  unsigned row[4];       // row fragment ks & 3 of row r
  unsigned tr[2][2][2];  // transposed: [k-step s][rows +8][column block dt & 1]
  __device__ __forceinline__ void init(int r, int h, int lane) {
#pragma unroll
    for (int k = 0; k < 4; ++k) row[k] = (unsigned)T::off(r, k * 16 + h * 8);
    const int g = lane >> 4, hh = g >> 1, m = lane & 15;
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int d = 0; d < 2; ++d)
          tr[s][e][d] = (unsigned)T::off(16 * s + 4 * hh + (m >> 2) + 8 * e, 32 * d + 16 * (g & 1) + 4 * (m & 3));
  }
  __device__ __forceinline__ MB::frag row_frag(const char* tile, int ks) const {
    return *(const MB::frag*)(tile + row[ks & 3] + (ks >> 2) * 128);
  }
  __device__ __forceinline__ MB::frag trans(const char* tile, int s, int dt) const {
    const int step = (dt >> 1) * 128;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(tile + tr[s][0][dt & 1] + step));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(tile + tr[s][1][dt & 1] + step));
    const bf16x4 l4 = __builtin_bit_cast(bf16x4, lo), h4 = __builtin_bit_cast(bf16x4, hi);
    MB::frag f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[i] = l4[i];
      f[4 + i] = h4[i];
    }
    return f;
  }
};

// Flip the sign of every element of a bf16 fragment.
__device__ __forceinline__ MB::frag negated(MB::frag f) {
  u32x4 u = __builtin_bit_cast(u32x4, f);
  u ^= 0x80008000u;
  return __builtin_bit_cast(MB::frag, u);
}

}  // namespace cattn
