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

// Copies issued after tile t+1 and still allowed in flight at the top of
// tile t, in tiles, for a ring that runs `ahead` tiles ahead over n tiles
// (tile t+k is copied at the top of tile t+k-ahead).
constexpr int later_tiles(int t, int n, int ahead) { return imax(0, imin(ahead - 2, n - 2 - t)); }

}  // namespace cattn
