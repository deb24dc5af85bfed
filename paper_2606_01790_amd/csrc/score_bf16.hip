// bf16 instantiations of the scoring passes (v_mfma_f32_32x32x16_bf16).
#include "score_kernels.h"

namespace starkv {

int run_score_bf16(const ScoreArgs& a, int d, int n_layers, hipStream_t st) {
  return d == 128 ? run_nrb<__bf16, 128>(a, n_layers, st) : run_nrb<__bf16, 64>(a, n_layers, st);
}

}  // namespace starkv
