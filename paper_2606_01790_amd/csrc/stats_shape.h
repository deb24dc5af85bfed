// Block shape of the statistics kernel (threads per block) for a call, from
// its block count, the GPU's CU count and the binning parameters.  Host and
// tests share this code; the kernel's LDS partitions per shape live in
// state.hip (StatsShape).
//   1024  the wide shape, one block per CU: when every block fits on the GPU
//         at once, or the bins need its LDS;
//   512   the narrow shape, two blocks per CU (n_bins <= kNarrowMaxBins);
//   256   the small shape, four blocks per CU, when even two per CU leave
//         blocks for a second round (n_bins <= kSmallMaxBins and
//         grid^2 <= kSmallMaxCells).
// A layer's blocks: one per subspace (MI), one for the AEB statistic and
// stats_stab_blocks for the stability means, kStabSubspaces subspaces each.
#pragma once

namespace starkv {

constexpr int kNarrowMaxBins = 17;
constexpr int kSmallMaxBins = 9;
constexpr int kSmallMaxCells = 64;
constexpr int kStabSubspaces = 8;

inline int stats_stab_blocks(int n_sub) { return (n_sub + kStabSubspaces - 1) / kStabSubspaces; }
inline int stats_layer_blocks(int n_sub) { return n_sub + 1 + stats_stab_blocks(n_sub); }

inline int stats_shape_for(long blocks, int n_cu, int n_bins, int grid) {
  if (blocks <= n_cu || n_bins > kNarrowMaxBins) return 1024;
  if (blocks > 2L * n_cu && n_bins <= kSmallMaxBins && grid * grid <= kSmallMaxCells)
    return 256;
  return 512;
}

}  // namespace starkv
