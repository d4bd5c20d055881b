// Exhaustive check of the ring-schedule arithmetic of attn_sched.h against an
// explicit simulation of the copies, for every ring depth, split and read
// depth the kernels use and every tile count up to 300.
#include <cstdio>
#include <initializer_list>

#include "attn_sched.h"
#include "lmhead_sched.h"
#include <vector>

using namespace cattn;

int main() {
  long bad = 0, checks = 0;
  for (int NB : {3, 4, 6, 8}) {
    const int AH = NB - 1;
    for (int split : {1, 2}) {
      for (int need : {0, 1}) {
        if (need >= AH) continue;
        for (int n = 1; n <= 300; ++n) {
          const int L = (n + split - 1) / split, n_last = n - (split - 1) * L;
          auto tiles = [&](int x) { return (x < L ? split - 1 : 0) + (x < n_last ? 1 : 0); };
          for (int i = 1; i < L; ++i) {
            ++checks;
            // copies issued before the wait at the top of iteration i, in iteration order:
            // iterations 0 .. AH-1 before the loop, iteration i'+AH at the top of iteration i' < i
            int issued = 0;
            for (int x = 0; x < L && x <= i - 1 + AH; ++x) issued += tiles(x);
            const int f = ring_in_flight(i, L, n_last, split, AH, need);
            int required = 0;  // every part tile this iteration reads
            for (int x = 0; x <= i + need && x < L; ++x) required += tiles(x);
            if (f < 0 || issued - f < required) ++bad;
            if (i + AH - 1 < n_last && f != ring_in_flight_full(split, AH, need)) ++bad;
            // the copy issued at the top of iteration i (iteration i+AH) reuses the buffer
            // of iteration i-1, finished before the barrier, never one read at i .. i+need
            if (i + AH < L) {
              const int b = (i + AH) % NB;
              if (b != (i - 1) % NB) ++bad;
              for (int k = 0; k <= need; ++k)
                if (b == (i + k) % NB) ++bad;
            }
          }
        }
      }
    }
  }
  // banded_rank is a permutation of [0, n) for every grid size and band
  for (int n = 1; n <= 1200; n += 7) {
    for (int band : {0, 1, 3, 80, 256, 304}) {
      static unsigned char seen[1200];
      for (int i = 0; i < n; ++i) seen[i] = 0;
      for (int b = 0; b < n; ++b) {
        ++checks;
        const int r = banded_rank(b, n, band);
        if (r < 0 || r >= n || seen[r]) ++bad;
        else seen[r] = 1;
      }
    }
  }
  for (int S = 1; S <= 5000; ++S) {
    const int p = ws_rows(S);
    if (p % 32 != 0 || p < S || p >= S + 32) ++bad;
  }
  // loss-head persistent grid: every (vocabulary tile, token tile) is taken by
  // exactly one work group, on the chiplet of its vocabulary tile, in bounds
  for (int N : {128, 256, 384, 1152, 2304, 50304, 65536 + 128}) {
    for (int M : {128, 256, 384, 8192}) {
      const int n_vt = lmh_vtiles(N), n_mt = lmh_mtiles(M);
      for (int per_xcd : {1, 3, 32}) {
        std::vector<int> seen((size_t)n_vt * n_mt, 0);
        for (int b = 0; b < lmh_grid(per_xcd); ++b) {
          const int x = b % kXcdGroup;
          for (int l = b / kXcdGroup; l < lmh_xcd_tiles(x, n_vt, n_mt); l += per_xcd) {
            ++checks;
            const int t = lmh_xcd_tile(x, l, n_vt, n_mt), vt = t >> 16, mt = t & 0xffff;
            if (vt < 0 || vt >= n_vt || mt < 0 || mt >= n_mt || vt % kXcdGroup != x) {
              ++bad;
              continue;
            }
            ++seen[(size_t)vt * n_mt + mt];
          }
        }
        for (int c : seen)
          if (c != 1) ++bad;
      }
    }
  }
  // grouped ring (one barrier per G iterations): every tile an iteration reads has landed at the
  // group's wait (copies complete in issue order), and no copy overwrites a tile still to be read
  for (int NB : {3, 4, 6, 8, 9, 12}) {
    for (int G : {1, 2, 3, 4})
    for (int need : {0, 1}) {
      const int pro = NB - G;
      if (NB % G || NB < 2 * G + need) continue;
      ++checks;
      if (ring_group(1, NB, need, G) != G || ring_group(2, NB, need, G) != 1) ++bad;
      for (int L = 1; L <= 70; ++L) {
        std::vector<int> order;  // tiles in issue order
        for (int t = 0; t < pro && t < L; ++t) order.push_back(t);
        std::vector<char> landed(L, 0);
        for (int t : order) landed[t] = 1;  // the prologue waits for everything
        for (int i = 0; i < L; i += G) {
          if (i > 0) {
            const int k = ring_group_in_flight(i, L, NB, G, need);
            ++checks;
            if (k < 0 || k > (int)order.size()) {
              ++bad;
              continue;
            }
            for (size_t x = 0; x + k < order.size(); ++x) landed[order[x]] = 1;
          }
          for (int g = 0; g < G; ++g) {
            const int t = i + pro + g;
            if (t >= L) continue;
            ++checks;
            const int prev = t - NB;  // the slot's previous tile: read by iterations prev - 1 and prev
            if (prev >= 0 && prev >= i) ++bad;
            order.push_back(t);
          }
          for (int j = i; j < i + G && j < L; ++j)
            for (int t = j; t <= j + need && t < L; ++t) {
              ++checks;
              if (!landed[t]) ++bad;
            }
        }
      }
    }
  }
  std::printf("checks=%ld bad=%ld\n", checks, bad);
  return bad != 0 || checks == 0;
}
