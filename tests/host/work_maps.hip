// Host-side check that the kernels' workgroup -> work maps are bijections
// (every work item is taken by exactly one workgroup).  Built and run by
// tests/test_work_maps.py on the CPU; no GPU call is made.
#include <cstdio>
#include <vector>

#include "kernels.h"

int main() {
  long checked = 0;
  // xcd_contiguous: a permutation of [0, G) whose XCD x = b % 8 takes a
  // contiguous range of work indices, in increasing order.
  for (int G = 1; G <= 4200; ++G) {
    std::vector<int> seen(G, 0);
    std::vector<int> last(8, -1);
    for (int b = 0; b < G; ++b) {
      const int w = sdq::xcd_contiguous(b, G);
      if (w < 0 || w >= G || seen[w]++) {
        std::printf("xcd_contiguous(%d, %d) = %d: out of range or repeated\n", b, G, w);
        return 1;
      }
      const int x = b & 7;
      if (last[x] >= 0 && w != last[x] + 1) {
        std::printf("xcd_contiguous: XCD %d of G = %d is not contiguous (%d after %d)\n", x, G, w, last[x]);
        return 1;
      }
      last[x] = w;
      ++checked;
    }
  }
  // tile_work: a bijection from [0, G * MB) onto the pairs (group, token block).
  for (int G = 1; G <= 180; ++G) {
    for (int MB = 1; MB <= 40; ++MB) {
      std::vector<int> seen(G * MB, 0);
      for (int b = 0; b < G * MB; ++b) {
        int g = -1, mb = -1;
        sdq::tile_work(b, G, MB, g, mb);
        if (g < 0 || g >= G || mb < 0 || mb >= MB || seen[g * MB + mb]++) {
          std::printf("tile_work(%d, G=%d, MB=%d) = (%d, %d): out of range or repeated\n", b, G, MB, g, mb);
          return 1;
        }
        ++checked;
      }
    }
  }
  std::printf("work maps ok: %ld workgroups checked\n", checked);
  return 0;
}
