// Host check of K1's tile order: the device functions xcd_tile and tile_coords, compiled for
// the host from the library's own header, must map every launch onto its tiles one to one.
// Exit status 0 and "ok <count>" when every case holds; the first failing case otherwise.
#include <cstdio>
#include <vector>

#include "k_lmhead.h"

int main() {
  // block id -> tile is a permutation of [0, G) for every grid size
  for (int G = 1; G <= 4096; ++G) {
    std::vector<char> hit(G, 0);
    for (int b = 0; b < G; ++b) {
      const int t = asv::xcd_tile(b, G);
      if (t < 0 || t >= G || hit[t]++) {
        std::printf("xcd_tile G=%d block %d -> tile %d\n", G, b, t);
        return 1;
      }
    }
  }
  // tile -> (slab, row tile) covers every pair once, slab-major (blk_rows 0 or >= RT) or in
  // blocks of bs slabs x br row tiles with ragged last blocks and groups
  long cases = 0;
  for (int RT = 1; RT <= 24; ++RT)
    for (int n = 1; n <= 70; ++n)
      for (int bs = 1; bs <= 10; ++bs)
        for (int br = 0; br <= RT + 1; ++br) {
          std::vector<char> hit((size_t)n * RT, 0);
          for (int t = 0; t < n * RT; ++t) {
            int slab = -1, rt = -1;
            asv::tile_coords(t, n, RT, bs, br, slab, rt);
            if (slab < 0 || slab >= n || rt < 0 || rt >= RT || hit[(size_t)slab * RT + rt]++) {
              std::printf("tile_coords RT=%d slabs=%d block %dx%d: tile %d -> (%d, %d)\n", RT, n,
                          bs, br, t, slab, rt);
              return 1;
            }
          }
          ++cases;
        }
  std::printf("ok %ld\n", cases);
  return 0;
}
