// Device-side building blocks shared by the forward and backward attention
// kernels for gfx950 (CDNA4): matrix-core operand fragments, the swizzled LDS
// tile layout, global->LDS tile staging and cross-half wave reductions.
//
// Matrix-core shape.  Every contraction is issued as 32x32 output blocks:
//   bf16: v_mfma_f32_32x32x16_bf16  (A 32x16, B 16x32, C 32x32 float)
//   f32 : v_mfma_f32_32x32x2_f32    (A 32x2,  B 2x32,  C 32x32 float)
// A lane L = 32*h + r (h = half of the wave, r = L % 32) supplies row r of A
// and column r of B, each holding KL consecutive contraction elements starting
// at h*KL (KL = 8 for bf16, 1 for f32).  It receives the C entries
//   C[8*(a/4) + 4*h + a%4][r]   for accumulator index a = 0..15.
// Only the C layout matters for correctness: any permutation of the
// contraction index applied to A and B alike leaves the result unchanged.
// The kernels rely on that to feed a C-layout accumulator (scores, P, dS)
// straight back into a second contraction as its B operand without any
// register shuffle: accumulator indices a in [s*KL, (s+1)*KL) form k-step s,
// and the matching A operand rows are read from LDS in the same order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn_sched.h"

namespace cattn {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr float kLog2e = 1.44269504088896340736f;
constexpr float kLn2 = 0.69314718055994530942f;
// Finite mask sentinel (section 4.2): masked scores get a large negative
// finite value rather than -inf; the base-2 exponential maps it to exactly 0.
constexpr float kMasked = -1.0e30f;
// Largest base-2 exponent a probability may reach before the float32 forward
// moves its softmax offset (P <= 2^8 = 256, far inside float range).  The bf16
// forward uses a bound on the block's probability sum instead (2^32, see
// kSumMax there).
constexpr float kRescaleLog2 = 8.0f;

// ---------------------------------------------------------------------------
// Matrix-core traits
// ---------------------------------------------------------------------------
template <typename T> struct Mma;

template <> struct Mma<__bf16> {
  static constexpr int K = 16;   // contraction length of one instruction
  static constexpr int KL = 8;   // contraction elements held per lane
  typedef bf16x8 frag;
  static __device__ __forceinline__ f32x16 run(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  // B operand of k-step s built from a C-layout accumulator (round to nearest even).
  static __device__ __forceinline__ frag pack(const f32x16& acc, int s) {
    frag f;
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = (__bf16)acc[8 * s + i];
    return f;
  }
};

template <> struct Mma<float> {
  static constexpr int K = 2;
  static constexpr int KL = 1;
  typedef float frag;
  static __device__ __forceinline__ f32x16 run(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag pack(const f32x16& acc, int s) { return acc[s]; }
};

// Row (within a 32-row block) that accumulator index a of half h refers to.
__device__ __forceinline__ int acc_row(int a, int h) { return 8 * (a >> 2) + 4 * h + (a & 3); }

// ---------------------------------------------------------------------------
// LDS tile: row-major [rows][D] of T, with 16-byte chunks XOR-swizzled by row.
// ---------------------------------------------------------------------------
// Physical 16-byte chunk of logical chunk c in row r is c ^ swz(r), swz linear
// over GF(2) in the row bits (per-bit masks 2, 7, 6, 5, 7 for bits 0..4).
// Chosen by timing every such map on MI355X against the two access patterns a
// tile sees -- 16-byte row reads by 32 consecutive rows and transposed 8-byte
// reads of 4 consecutive rows x 2 chunks: it makes the transposed reads run at
// the rate of conflict-free linear reads (about twice as fast as keying by
// row pairs) and is among the fastest maps for the row reads.
__device__ __forceinline__ int swz(int row) {
  return ((row & 1) ? 2 : 0) ^ ((row & 2) ? 7 : 0) ^ ((row & 4) ? 6 : 0) ^ ((row & 8) ? 5 : 0) ^
         ((row & 16) ? 7 : 0);
}

template <typename T, int D> struct Tile {
  static constexpr int kRowBytes = D * (int)sizeof(T);
  static constexpr int kChunks = kRowBytes / 16;
  static_assert(kChunks >= 8, "swizzle needs at least 8 chunks per row");
  __device__ __forceinline__ static int off(int row, int col) {
    const int byte = col * (int)sizeof(T);
    return row * kRowBytes + ((((byte >> 4) ^ swz(row))) << 4) + (byte & 15);
  }
};

// Contiguous-K operand (rows of a row-major tile): lane (h, r) reads row `row`
// at columns [ks*K + h*KL, +KL).
template <typename T, int D>
__device__ __forceinline__ typename Mma<T>::frag read_row_frag(const char* lds, int row, int ks, int h) {
  typedef Mma<T> M;
  return *(const typename M::frag*)(lds + Tile<T, D>::off(row, ks * M::K + h * M::KL));
}

// Transposed operand: the A operand of a contraction over the tile's ROW index
// (keys for V and K, queries for Q and dO), i.e. A[m][k] = tile[row(k)][n0 + m].
// Rows follow the accumulator order of k-step s inside the 32-row block at rb,
// so the B operand can be Mma<T>::pack(acc, s).
template <typename T, int D> struct TransRead;

template <int D> struct TransRead<__bf16, D> {
  // ds_read_b64_tr_b16: within each group of 16 lanes, lane 4j+c supplies the
  // address of 4 consecutive elements of row j (columns 4c..4c+3 of a 16-wide
  // strip); lane n of the group receives column n of rows 0..3 of the strip.
  static __device__ __forceinline__ bf16x8 read(const char* lds, int rb, int s, int n0, int lane) {
    const int g = lane >> 4, h = g >> 1, m = lane & 15;
    const int col = n0 + 16 * (g & 1) + 4 * (m & 3);
    const int row = rb + 16 * s + 4 * h + (m >> 2);
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(lds + Tile<__bf16, D>::off(row, col)));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(lds + Tile<__bf16, D>::off(row + 8, col)));
    bf16x8 f;
    const bf16x4 l4 = __builtin_bit_cast(bf16x4, lo), h4 = __builtin_bit_cast(bf16x4, hi);
#pragma unroll
    for (int i = 0; i < 4; ++i) { f[i] = l4[i]; f[4 + i] = h4[i]; }
    return f;
  }
};

template <int D> struct TransRead<float, D> {
  static __device__ __forceinline__ float read(const char* lds, int rb, int s, int n0, int lane) {
    const int h = lane >> 5;
    return *(const float*)(lds + Tile<float, D>::off(rb + acc_row(s, h), n0 + (lane & 31)));
  }
};

// ---------------------------------------------------------------------------
// Global -> registers -> LDS staging of an R x D tile (rows >= nrows are zero).
// Consecutive threads take consecutive 16-byte chunks of a row, so each row is
// one fully coalesced 128/256-byte segment.
// ---------------------------------------------------------------------------
template <typename T, int D, int R, int NT> struct TileStage {
  static constexpr int kChunksPerRow = Tile<T, D>::kChunks;
  static constexpr int kPerThread = R * kChunksPerRow / NT;
  static_assert(R * kChunksPerRow % NT == 0, "tile must split evenly over the threads");
  u32x4 reg[kPerThread];

  // rows of g are rs elements apart
  __device__ __forceinline__ void load(const T* g, int row0, int nrows, int tid, int rs) {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int c = tid + i * NT;
      const int row = c / kChunksPerRow, ch = c % kChunksPerRow;
      if (row0 + row < nrows) {
        reg[i] = *(const u32x4*)((const char*)g + ((int64_t)(row0 + row) * rs) * (int64_t)sizeof(T) + ch * 16);
      } else {
        reg[i] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  }
  __device__ __forceinline__ void store(char* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int c = tid + i * NT;
      const int row = c / kChunksPerRow, ch = c % kChunksPerRow;
      *(u32x4*)(lds + row * Tile<T, D>::kRowBytes + ((ch ^ swz(row)) << 4)) = reg[i];
    }
  }
};

// ---------------------------------------------------------------------------
// Cross-half reductions: combine lane r with lane r + 32 (v_permlane32_swap
// exchanges the upper half of its first operand with the lower half of its
// second; passing x twice gives every lane both halves' values, lower first,
// so both halves compute the identical result).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void halves(float x, float& lo, float& hi) {
  const unsigned u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  lo = __uint_as_float(r[0]);
  hi = __uint_as_float(r[1]);
}
__device__ __forceinline__ float halves_max(float x) { float a, b; halves(x, a, b); return fmaxf(a, b); }
__device__ __forceinline__ float halves_sum(float x) { float a, b; halves(x, a, b); return a + b; }

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

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

// Store 4 consecutive row elements (one accumulator run) converted to T.
template <typename T> __device__ __forceinline__ void store4(T* dst, float a, float b, float c, float d);
template <> __device__ __forceinline__ void store4<float>(float* dst, float a, float b, float c, float d) {
  *(f32x4*)dst = f32x4{a, b, c, d};
}
template <> __device__ __forceinline__ void store4<__bf16>(__bf16* dst, float a, float b, float c, float d) {
  bf16x4 v;
  v[0] = (__bf16)a; v[1] = (__bf16)b; v[2] = (__bf16)c; v[3] = (__bf16)d;
  *(bf16x4*)dst = v;
}

// Load the contiguous-K B-operand fragments of one row straight from global
// memory (zero when row >= S); rows of g are rs elements apart.
template <typename T, int D>
__device__ __forceinline__ void load_row_frags(const T* g, int row, int S, int h, int rs,
                                               typename Mma<T>::frag (&f)[D / Mma<T>::K]) {
  typedef Mma<T> M;
#pragma unroll
  for (int ks = 0; ks < D / M::K; ++ks) {
    if (row < S) {
      f[ks] = *(const typename M::frag*)(g + (int64_t)row * rs + ks * M::K + h * M::KL);
    } else {
      f[ks] = typename M::frag{};
    }
  }
}

// Where the S x D matrix of (batch, head) bh starts, in elements, and how far
// apart its rows are: [B, H, S, D] storage (heads-major: rows D apart) or
// [B, S, H, D] storage (sequence-major, the layout a fused QKV projection
// produces: rows H*D apart, heads D apart).  Batch stride H*S*D in both.
struct Rows {
  int64_t base;
  int rs;
};
__device__ __forceinline__ Rows rows_of(int bh, int H, int S, int D, bool seq_major) {
  if (!seq_major) return Rows{(int64_t)bh * S * D, D};
  const int b = bh / H, hh = bh - b * H;
  return Rows{(int64_t)b * H * S * D + (int64_t)hh * D, H * D};
}

// Map a block index to (head, tile) so that the heaviest causal tiles start
// first and every tile of a head lands on the same XCD when B*H % 8 == 0
// (blocks are dealt to the 8 XCDs round-robin).  `heavy_last` = true when the
// highest tile index carries the most work (forward / dQ: queries late in the
// sequence see the most keys); false for dK/dV (early keys see most queries).
__device__ __forceinline__ void tile_of_block(int bid, int BH, int ntiles, bool heavy_last, int& bh, int& tile) {
  bh = bid % BH;
  const int t = bid / BH;
  tile = heavy_last ? (ntiles - 1 - t) : t;
}
// The same, with the heaviest-first ranks dealt to rounds of `band` work groups
// in alternating directions (banded_rank), so that the work groups sharing a
// compute unit carry complementary amounts of causal work.
__device__ __forceinline__ void tile_of_block_banded(int bid, int BH, int ntiles, bool heavy_last, int band, int& bh,
                                                     int& tile) {
  tile_of_block(banded_rank(bid, BH * ntiles, band), BH, ntiles, heavy_last, bh, tile);
}

}  // namespace cattn
