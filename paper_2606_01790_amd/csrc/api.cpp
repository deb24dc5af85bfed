// extern "C" entry points of libstarkv.so: argument validation on the host,
// then the launch functions of the kernels.  Nothing here allocates memory or
// synchronises a stream.
#include <cstring>

#include "internal.h"

using namespace starkv;

namespace {

starkv_status hip_status(int err) { return err ? STARKV_E_HIP : STARKV_OK; }

// Rows of the current frame (0 without spans).
int frame_tokens(const starkv_span* spans, int32_t n_spans, int32_t frame) {
  const int i = current_span(spans, n_spans, frame);
  return i < 0 ? 0 : spans[i].rows * spans[i].cols;
}

}  // namespace

extern "C" {

int32_t starkv_abi_version(void) { return STARKV_ABI_VERSION; }

const char* starkv_status_str(starkv_status s) {
  switch (s) {
    case STARKV_OK: return "ok";
    case STARKV_E_NULL: return "a required pointer is NULL";
    case STARKV_E_SHAPE: return "inconsistent or unsupported dimensions";
    case STARKV_E_BUDGET: return "budget B outside [0, L_p]";
    case STARKV_E_SPANS: return "malformed visual spans";
    case STARKV_E_PARAM: return "hyper-parameter out of range";
    case STARKV_E_DTYPE: return "unknown element type";
    case STARKV_E_ALIGN: return "pointer or stride not 16-byte aligned";
    case STARKV_E_WORKSPACE: return "workspace missing or too small";
    case STARKV_E_STATE: return "state capacity too small for the frame";
    case STARKV_E_HIP: return "HIP launch error";
  }
  return "unknown status";
}

void starkv_params_default(starkv_params* p) {
  if (!p) return;
  std::memset(p, 0, sizeof(*p));
  p->lam = 0.5f;
  p->n_warmup = 5;
  p->n_ramp = 10;
  p->rho_mi = 0.9f;
  p->tau = 1.0f;
  p->rho_t = 0.9f;
  p->delta = 0.2f;
  p->d_min = 0.1f;
  p->t_min = 0.75f;
  p->t_max = 1.25f;
  p->n_bins = 8;
  p->grid = 8;
  p->pool_kernel = 5;
  p->eps = 1e-8f;
  p->tem_decay = STARKV_TEM_EXP;
  p->aeb_mode = STARKV_AEB_ENTROPY;
}

size_t starkv_workspace_bytes(const starkv_dims* dims) {
  Geometry g;
  if (check_dims(dims, &g) != STARKV_OK) return 0;
  return ws_layout(g).total;
}

size_t starkv_scalars_count(const starkv_dims* dims) {
  Geometry g;
  if (check_dims(dims, &g) != STARKV_OK) return 0;
  return scalars_count(g.Ns);
}

size_t starkv_state_bytes(const starkv_dims* dims, int32_t frame_cap) {
  Geometry g;
  if (check_dims(dims, &g) != STARKV_OK || frame_cap < 0) return 0;
  return state_stride(g.Ns, frame_cap) * (size_t)g.n_layers;
}

starkv_status starkv_state_init(const starkv_dims* dims, void* state,
                                int32_t frame_cap, void* stream) {
  Geometry g;
  starkv_status st = check_dims(dims, &g);
  if (st != STARKV_OK) return st;
  if (!state) return STARKV_E_NULL;
  if (frame_cap < 0) return STARKV_E_STATE;
  if (!aligned(state, 16)) return STARKV_E_ALIGN;
  return hip_status(launch_state_init(g, state, frame_cap, stream));
}

starkv_status starkv_score(const starkv_dims* dims, const starkv_params* params,
                           const void* q, const void* k,
                           const starkv_kv_layout* k_layout, float* S,
                           float* sbar, uint8_t* gstar, void* ws,
                           size_t ws_bytes, void* stream) {
  Geometry g;
  starkv_status st = check_dims(dims, &g);
  if (st != STARKV_OK) return st;
  if ((st = check_pool(params)) != STARKV_OK) return st;
  if (!q || !k || !k_layout || !S || !sbar || !gstar) return STARKV_E_NULL;
  if ((st = check_layout(k_layout, g)) != STARKV_OK) return st;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(S, 4) || !aligned(sbar, 4))
    return STARKV_E_ALIGN;
  if (!ws || ws_bytes < ws_layout(g).total) return STARKV_E_WORKSPACE;
  if (!aligned(ws, 16)) return STARKV_E_ALIGN;
  return hip_status(launch_score(g, *params, q, k, *k_layout, S, sbar, gstar, ws, stream));
}

starkv_status starkv_update_state(const starkv_dims* dims,
                                  const starkv_params* params, const float* S,
                                  const float* sbar, const starkv_span* spans,
                                  int32_t n_spans, int32_t frame, void* state,
                                  int32_t frame_cap, float* scalars, void* ws,
                                  size_t ws_bytes, void* stream) {
  (void)ws;
  (void)ws_bytes;
  Geometry g;
  starkv_status st = check_dims(dims, &g);
  if (st != STARKV_OK) return st;
  if ((st = check_params(params)) != STARKV_OK) return st;
  if (!S || !sbar || !state || !scalars) return STARKV_E_NULL;
  if ((st = check_spans(spans, n_spans, frame, g.Lp)) != STARKV_OK) return st;
  if (frame_cap < 0 || frame_tokens(spans, n_spans, frame) > frame_cap)
    return STARKV_E_STATE;
  if (!aligned(S, 4) || !aligned(sbar, 4) || !aligned(scalars, 4) ||
      !aligned(state, 16))
    return STARKV_E_ALIGN;
  return hip_status(launch_update_state(g, *params, S, sbar, spans, n_spans, frame,
                                        state, frame_cap, scalars, stream));
}

starkv_status starkv_select(const starkv_dims* dims, const starkv_params* params,
                            const float* sbar, const uint8_t* gstar,
                            const float* scalars, const starkv_span* spans,
                            int32_t n_spans, int32_t frame, int32_t B, float* s,
                            int32_t* idx, void* ws, size_t ws_bytes,
                            void* stream) {
  (void)ws;
  (void)ws_bytes;
  Geometry g;
  starkv_status st = check_dims(dims, &g);
  if (st != STARKV_OK) return st;
  if ((st = check_params(params)) != STARKV_OK) return st;
  if (!sbar || !gstar || !scalars || !s) return STARKV_E_NULL;
  if (B < 0 || B > g.Lp) return STARKV_E_BUDGET;
  if (B > 0 && !idx) return STARKV_E_NULL;
  if ((st = check_spans(spans, n_spans, frame, g.Lp)) != STARKV_OK) return st;
  if (!aligned(sbar, 4) || !aligned(scalars, 4) || !aligned(s, 4) ||
      (idx && !aligned(idx, 4)))
    return STARKV_E_ALIGN;
  return hip_status(launch_select(g, *params, sbar, gstar, scalars, spans, n_spans,
                                  frame, B, s, idx, stream));
}

starkv_status starkv_update_state_select(const starkv_dims* dims,
                                         const starkv_params* params, const float* S,
                                         const float* sbar, const uint8_t* gstar,
                                         const starkv_span* spans, int32_t n_spans,
                                         int32_t frame, void* state, int32_t frame_cap,
                                         float* scalars, int32_t B, float* s, int32_t* idx,
                                         void* ws, size_t ws_bytes, void* stream) {
  (void)ws;
  (void)ws_bytes;
  Geometry g;
  starkv_status st = check_dims(dims, &g);
  if (st != STARKV_OK) return st;
  if ((st = check_params(params)) != STARKV_OK) return st;
  if (!S || !sbar || !gstar || !state || !scalars || !s) return STARKV_E_NULL;
  if (B < 0 || B > g.Lp) return STARKV_E_BUDGET;
  if (B > 0 && !idx) return STARKV_E_NULL;
  if ((st = check_spans(spans, n_spans, frame, g.Lp)) != STARKV_OK) return st;
  if (frame_cap < 0 || frame_tokens(spans, n_spans, frame) > frame_cap)
    return STARKV_E_STATE;
  if (!aligned(S, 4) || !aligned(sbar, 4) || !aligned(scalars, 4) || !aligned(state, 16) ||
      !aligned(s, 4) || (idx && !aligned(idx, 4)))
    return STARKV_E_ALIGN;
  return hip_status(launch_update_state_select(g, *params, S, sbar, gstar, spans, n_spans,
                                               frame, state, frame_cap, scalars, B, s, idx,
                                               stream));
}

starkv_status starkv_compact(const starkv_dims* dims, const void* k,
                             const void* v, const starkv_kv_layout* kv_layout,
                             const int32_t* idx, int32_t B, void* k_out,
                             void* v_out, void* stream) {
  Geometry g;
  starkv_status st = check_dims(dims, &g);
  if (st != STARKV_OK) return st;
  if (!k || !v || !kv_layout || !k_out || !v_out) return STARKV_E_NULL;
  if (B < 0 || B > g.Lp) return STARKV_E_BUDGET;
  if (B > 0 && !idx) return STARKV_E_NULL;
  if ((st = check_layout(kv_layout, g)) != STARKV_OK) return st;
  if (!aligned(k, 16) || !aligned(v, 16) || !aligned(k_out, 16) ||
      !aligned(v_out, 16) || (idx && !aligned(idx, 4)))
    return STARKV_E_ALIGN;
  return hip_status(launch_compact(g, k, v, *kv_layout, idx, B, k_out, v_out, stream));
}

size_t starkv_decode_workspace_bytes(const starkv_dims* dims, int32_t n_tokens) {
  DecodeGeometry g;
  if (check_decode(dims, n_tokens, &g) != STARKV_OK) return 0;
  return decode_ws_bytes(g);
}

starkv_status starkv_decode(const starkv_dims* dims, const void* q, const void* k,
                            const void* v, const starkv_kv_layout* kv_layout,
                            int32_t n_tokens, float* out, void* ws, size_t ws_bytes,
                            void* stream) {
  DecodeGeometry g;
  starkv_status st = check_decode(dims, n_tokens, &g);
  if (st != STARKV_OK) return st;
  if (!q || !k || !v || !kv_layout || !out) return STARKV_E_NULL;
  const int64_t esz = 2;
  if (kv_layout->layer_stride < 0 || kv_layout->group_stride < 0 ||
      kv_layout->token_stride < g.d)
    return STARKV_E_SHAPE;
  if ((kv_layout->layer_stride * esz) % 16 || (kv_layout->group_stride * esz) % 16 ||
      (kv_layout->token_stride * esz) % 16)
    return STARKV_E_ALIGN;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 4))
    return STARKV_E_ALIGN;
  if (!ws || ws_bytes < decode_ws_bytes(g)) return STARKV_E_WORKSPACE;
  if (!aligned(ws, 16)) return STARKV_E_ALIGN;
  return hip_status(launch_decode(g, q, k, v, *kv_layout, out, ws, stream));
}

}  // extern "C"
