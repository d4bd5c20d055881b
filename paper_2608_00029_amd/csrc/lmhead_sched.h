// Tile schedule of the fused loss-head projection: plain constexpr integer
// functions (no HIP types), so that the same definitions compile for the GPU
// and, in the tests, with the host C++ compiler.
#pragma once

#include "attn_sched.h"

namespace cattn {

constexpr int kLmhTileV = 256;  // vocabulary rows per output tile
constexpr int kLmhTileM = 256;  // tokens per output tile
constexpr int kLmhKC = 64;      // K chunk per ring slot
constexpr int kLmhPartW = 64;   // vocabulary entries per partial statistic

constexpr int lmh_vtiles(int N) { return (N + kLmhTileV - 1) / kLmhTileV; }
constexpr int lmh_mtiles(int M) { return (M + kLmhTileM - 1) / kLmhTileM; }

// Output tiles whose vocabulary tile index is congruent to x modulo kXcdGroup:
// the tiles of chiplet x (work groups are dealt to the chiplets round-robin).
constexpr int lmh_xcd_vtiles(int x, int n_vt) { return x < n_vt ? (n_vt - x + kXcdGroup - 1) / kXcdGroup : 0; }
constexpr int lmh_xcd_tiles(int x, int n_vt, int n_mt) { return lmh_xcd_vtiles(x, n_vt) * n_mt; }

// The l-th tile (0 <= l < lmh_xcd_tiles) of chiplet x, as (vocabulary tile,
// token tile) packed into vt * 65536 + mt.  A chiplet walks its vocabulary
// tiles in bands of 8 with the token tiles inside and the vocabulary index
// fastest, so that the tiles it runs at once share a few W and X row blocks
// (its L2 holds them).
constexpr int lmh_xcd_tile(int x, int l, int n_vt, int n_mt) {
  const int nv = lmh_xcd_vtiles(x, n_vt);
  const int vb = l / (8 * n_mt);
  const int g = imin(8, nv - 8 * vb);
  const int rem = l - vb * 8 * n_mt;
  const int mt = rem / g;
  const int vt = x + kXcdGroup * (8 * vb + rem % g);
  return vt * 65536 + mt;
}

// Persistent grid: work group b runs on chiplet b % kXcdGroup and takes that
// chiplet's tiles b / kXcdGroup, b / kXcdGroup + per_xcd, ... where per_xcd is
// the number of work groups per chiplet (the grid has kXcdGroup * per_xcd).
constexpr int lmh_grid(int n_wg_per_xcd) { return kXcdGroup * n_wg_per_xcd; }

}  // namespace cattn
