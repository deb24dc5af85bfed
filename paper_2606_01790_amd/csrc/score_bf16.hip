// bf16 instantiations of the scoring passes (v_mfma_f32_32x32x16_bf16).
// With d = 128 and one subspace per KV group, or per-head subspaces whose
// heads are whole 32-row blocks, pass 2 runs on the persistent slab kernel
// of score_slab.h; other shapes use the tile kernels of both passes.
#include <algorithm>

#include "score_slab.h"

namespace starkv {
namespace {

template <int NRB>
int slab_passes(const ScoreArgs& a, int n_layers, int n_cu, hipStream_t st) {
  using KS = KStage<__bf16, 128, NRB * 64>;
  const int items = a.n_chunks * a.G * n_layers;
  const size_t lds1 = 2 * (size_t)KS::kElems * sizeof(__bf16);
  score_pass1<__bf16, 128, NRB><<<items, NRB * 64, lds1, st>>>(a);
  SlabGrid sg;
  sg.S = (a.Lp + 63) / 64;
  sg.nlg = a.G * n_layers;
  // one block per CU (the kernel holds two 256-VGPR waves per SIMD), never
  // more blocks than slabs
  const int nb = (int)std::min<long>(n_cu, (long)sg.S * sg.nlg);
  if (a.n_out > 1)
    score_pass2_slab<NRB, true><<<nb, 512, SlabLds<NRB>::kBytes, st>>>(a, sg);
  else
    score_pass2_slab<NRB, false><<<nb, 512, SlabLds<NRB>::kBytes, st>>>(a, sg);
  return (int)hipGetLastError();
}

}  // namespace

int run_pass2_slab(const ScoreArgs& a, int n_layers, int n_cu, hipStream_t st) {
  switch (a.Rpad / 32) {
#define STARKV_SLAB(n) \
  case n: return slab_passes<n>(a, n_layers, n_cu, st);
    STARKV_SLAB(1) STARKV_SLAB(2) STARKV_SLAB(3) STARKV_SLAB(4) STARKV_SLAB(5) STARKV_SLAB(6)
    STARKV_SLAB(7) STARKV_SLAB(8) STARKV_SLAB(9) STARKV_SLAB(10) STARKV_SLAB(11)
    STARKV_SLAB(12) STARKV_SLAB(13) STARKV_SLAB(14)
#undef STARKV_SLAB
  }
  return (int)hipErrorInvalidValue;
}

int run_score_bf16(const ScoreArgs& a, int d, int n_layers, hipStream_t st) {
  if (d == 128 && a.Rpad / 32 <= kSlabMaxNrb && (a.n_out == 1 || a.n_part == 1)) {
    int dev = 0, n_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n_cu <= 0)
      return (int)hipErrorInvalidDevice;
    return run_pass2_slab(a, n_layers, n_cu, st);
  }
  return d == 128 ? run_nrb<__bf16, 128>(a, n_layers, st) : run_nrb<__bf16, 64>(a, n_layers, st);
}

}  // namespace starkv
