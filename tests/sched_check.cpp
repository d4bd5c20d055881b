// Exhaustive check of the tile-schedule arithmetic of attn_sched.h against the
// conditions the streaming loops of the bf16 kernels rely on.
//
// A loop over n tiles with a ring of NB buffers copies tile k into buffer
// k % NB at the top of tile k - AHEAD (AHEAD = NB - 1; tiles 0..AHEAD-1 before
// the loop), each wave issuing a fixed number of copies per tile, and the
// copies of one wave complete in issue order.  At the top of tile t (t >= 1)
// the wave waits until at most later_tiles(t, n, AHEAD) tiles of its copies
// are in flight, then meets the other waves at a barrier; during tile t it
// reads tiles t and t+1.
#include <cstdio>
#include <initializer_list>

#include "attn_sched.h"

using namespace cattn;

int main() {
  long bad = 0, checks = 0;
  for (int NB : {3, 4, 6, 8}) {
    const int AH = NB - 1;
    for (int n = 1; n <= 300; ++n) {
      for (int t = 1; t < n; ++t) {
        ++checks;
        // copies issued before the wait at the top of tile t: tiles 0 .. min(t + AH - 1, n - 1)
        const int issued = imin(t + AH, n);
        const int done = issued - later_tiles(t, n, AH);  // tiles 0 .. done-1 have landed
        if (done < imin(t + 2, n)) ++bad;                  // tiles t and t+1 are resident
        if (later_tiles(t, n, AH) < 0) ++bad;
        // the copy issued at the top of tile t (tile t + AH) goes to the buffer of tile
        // t - 1, which every wave finished before the barrier; never to tile t or t + 1
        if (t + AH < n) {
          const int b = (t + AH) % NB;
          if (b == t % NB || b == (t + 1) % NB || b != (t - 1) % NB) ++bad;
        }
      }
    }
  }
  for (int S = 1; S <= 5000; ++S) {
    const int p = ws_rows(S);
    if (p % 32 != 0 || p < S || p >= S + 32) ++bad;
  }
  std::printf("checks=%ld bad=%ld\n", checks, bad);
  return bad != 0 || checks == 0;
}
