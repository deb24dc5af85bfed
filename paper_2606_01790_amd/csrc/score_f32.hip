// float32 instantiations of the scoring passes (v_mfma_f32_32x32x2f32), for
// up to four 32-row blocks of window rows per group.
#include "score_kernels.h"

namespace starkv {

int run_score_f32(const ScoreArgs& a, int d, int n_layers, hipStream_t st) {
  return d == 128 ? run_nrb_small<float, 128>(a, n_layers, st)
                  : run_nrb_small<float, 64>(a, n_layers, st);
}

}  // namespace starkv
