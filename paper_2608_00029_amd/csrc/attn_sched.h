// Tile-schedule arithmetic shared by the kernels and their launchers: plain
// constexpr integer functions (no HIP types), so that the same definitions
// compile for the GPU and, in the tests, with the host C++ compiler.
#pragma once

namespace cattn {

constexpr int imin(int a, int b) { return a < b ? a : b; }
constexpr int imax(int a, int b) { return a > b ? a : b; }

// Rows per (batch, head) of each backward workspace row: S padded to a
// multiple of 32 (padding entries hold zeros), so that 32-row tiles of it can
// be copied whole.
constexpr int ws_rows(int S) { return (S + 31) / 32 * 32; }

// Ring of LDS buffers streamed over iterations 0 .. L-1 by `split` parts: at
// iteration x every part owns one tile, except that the last part owns tiles
// only while x < n_last (n_last <= L).  The tiles of iteration x are copied at
// the top of iteration x - ahead (iterations 0 .. ahead-1 before the loop),
// each wave issuing the same number of copies per part tile, and a wave's
// copies complete in issue order.  Iteration i reads the tiles of iterations
// i .. i+need.  At the top of iteration i a wave may therefore leave in flight
// the part tiles of iterations i+need+1 .. i+ahead-1; this is their number.
constexpr int ring_in_flight(int i, int L, int n_last, int split, int ahead, int need) {
  int k = 0;
  for (int x = i + need + 1; x <= i + ahead - 1; ++x) k += (x < L ? split - 1 : 0) + (x < n_last ? 1 : 0);
  return k;
}
// The common case, when every part owns a tile at each of those iterations
// (i + ahead - 1 < n_last): a compile-time count.
constexpr int ring_in_flight_full(int split, int ahead, int need) { return (ahead - 1 - need) * split; }

// Order in which a grid of n work groups takes the work items, when items are
// ranked heaviest first (rank 0 = most work).  Work groups are placed on the
// GPU in rounds of `band` (one per compute unit): group b shares its compute
// unit with groups b +- band, b +- 2 band, ...  Every other round walks the
// ranks backwards, so that a compute unit that receives one of the heaviest
// items in one round receives one of the lightest of the next.  The walk is
// backwards in steps of kXcdGroup, keeping each rank's position within its
// group of kXcdGroup: work groups are dealt to the GPU's kXcdGroup chiplets
// (each with its own L2) round-robin by index, and a rank keeps the chiplet of
// the same-numbered group, so the tiles of one head, which share K/V or
// Q/dO, stay in one L2.  band <= 0 keeps the plain heaviest-first order.  A
// permutation of [0, n).
constexpr int kXcdGroup = 8;
constexpr int banded_rank(int bid, int n, int band) {
  if (band <= 0) return bid;
  const int r = bid / band, p = bid % band;
  if ((r & 1) == 0) return bid;
  const int size = n - r * band < band ? n - r * band : band;
  if (size % kXcdGroup != 0 || band % kXcdGroup != 0) return r * band + size - 1 - p;
  return r * band + (size / kXcdGroup - 1 - p / kXcdGroup) * kXcdGroup + p % kXcdGroup;
}

// Ring with one barrier per group of G iterations (one part; G divides the
// ring depth NB): the prologue copies tiles 0 .. NB-G-1, and at the top of
// iteration i (i % G == 0) the copies of tiles i+NB-G .. i+NB-1 are issued
// into the slots of tiles i-G .. i-1, which every wave finished at the
// barrier.  Iterations i .. i+G-1 read tiles up to i+G-1+need, so the wait at
// the top of i (i > 0) may leave in flight the tiles issued before that lie
// beyond it: this is their number.  Needs NB >= 2 G + need (the tiles a
// group reads are then copied before its top).
// Iterations per barrier a ring of NB slots can take with `split` parts and
// `need` tiles of look-ahead: the largest g <= want that groups the ring (one
// part, NB a multiple of g, NB >= 2 g + need), else 1.
constexpr int ring_group(int split, int NB, int need, int want) {
  for (int g = want; g > 1; --g)
    if (split == 1 && NB % g == 0 && NB >= 2 * g + need) return g;
  return 1;
}
constexpr int ring_group_in_flight(int i, int L, int NB, int G, int need) {
  const int last_issued = imin(L - 1, i + NB - G - 1);
  const int d = last_issued - (i + G - 1 + need);
  return d > 0 ? d : 0;
}

}  // namespace cattn

