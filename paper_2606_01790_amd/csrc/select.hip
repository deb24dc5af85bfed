// The selection kernel: one workgroup per layer runs select_body
// (select_body.h) with its fixed LDS static and the key cache dynamic.
#include "select_body.h"

namespace starkv {

void fill_sel_args(SelArgs& a, const Geometry& g, const starkv_params& p, const float* sbar,
                   const uint8_t* gstar, const float* scalars, const starkv_span* spans,
                   int32_t n_spans, int32_t frame, int32_t B, float* s, int32_t* idx,
                   int cache) {
  a.sbar = sbar;
  a.gstar = gstar;
  a.scal = scalars;
  a.s = s;
  a.idx = idx;
  a.G = g.Ns;   // g* indexes the scoring subspaces
  a.Lp = g.Lp;
  a.B = B;
  a.sc = (int)scalars_count(g.Ns);
  a.frame = frame;
  a.cache = cache;
  a.delta = p.delta;
  a.d_min = p.d_min;
  a.tem = p.tem_decay;
  a.n_spans = n_spans;
  for (int i = 0; i < n_spans; ++i) {
    a.start[i] = spans[i].start;
    a.end[i] = spans[i].start + spans[i].rows * spans[i].cols;
    a.sframe[i] = spans[i].frame;
  }
}

namespace {

__global__ __launch_bounds__(kSelThreads) void select_kernel(SelArgs a) {
  __shared__ SelShared sh;
  extern __shared__ __align__(16) uint32_t keys[];
  select_body(a, blockIdx.x, sh, keys);
}

}  // namespace

int launch_select(const Geometry& g, const starkv_params& p, const float* sbar,
                  const uint8_t* gstar, const float* scalars,
                  const starkv_span* spans, int32_t n_spans, int32_t frame,
                  int32_t B, float* s, int32_t* idx, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  SelArgs a;
  fill_sel_args(a, g, p, sbar, gstar, scalars, spans, n_spans, frame, B, s, idx,
                g.Lp < kSelLdsKeys ? g.Lp : kSelLdsKeys);
  const size_t lds = (size_t)a.cache * sizeof(uint32_t);
  // once per process; function-local static initialisation is thread-safe
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&select_kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
      (int)(kSelLdsKeys * sizeof(uint32_t)));
  (void)attr;
  select_kernel<<<g.n_layers, kSelThreads, lds, st>>>(a);
  return (int)hipGetLastError();
}

}  // namespace starkv
