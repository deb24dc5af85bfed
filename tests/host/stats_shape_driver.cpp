// Prints the statistics block shape for each "blocks n_cu n_bins grid" line
// of stdin (stats_shape.h, the same source the library compiles).  With the
// argument "layer" it instead prints "stability_blocks layer_blocks" for
// each subspace count read.
#include <cstdio>
#include <cstring>

#include "stats_shape.h"

int main(int argc, char** argv) {
  if (argc > 1 && std::strcmp(argv[1], "layer") == 0) {
    int n_sub;
    while (std::scanf("%d", &n_sub) == 1)
      std::printf("%d %d\n", starkv::stats_stab_blocks(n_sub), starkv::stats_layer_blocks(n_sub));
    return 0;
  }
  long blocks;
  int n_cu, n_bins, grid;
  while (std::scanf("%ld %d %d %d", &blocks, &n_cu, &n_bins, &grid) == 4)
    std::printf("%d\n", starkv::stats_shape_for(blocks, n_cu, n_bins, grid));
  return 0;
}
