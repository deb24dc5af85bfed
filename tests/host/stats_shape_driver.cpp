// Prints the statistics block shape for each "blocks n_cu n_bins grid" line
// of stdin (stats_shape.h, the same source the library compiles).
#include <cstdio>

#include "stats_shape.h"

int main() {
  long blocks;
  int n_cu, n_bins, grid;
  while (std::scanf("%ld %d %d %d", &blocks, &n_cu, &n_bins, &grid) == 4)
    std::printf("%d\n", starkv::stats_shape_for(blocks, n_cu, n_bins, grid));
  return 0;
}
