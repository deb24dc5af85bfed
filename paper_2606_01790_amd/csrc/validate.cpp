// Host-side argument validation and buffer geometry.  No HIP: this unit is
// also built with the host compiler for the sanitizer tests.
#include <algorithm>
#include <cmath>
#include <cstdint>

#include "internal.h"

namespace starkv {

bool aligned(const void* p, size_t a) {
  return (reinterpret_cast<uintptr_t>(p) % a) == 0;
}

starkv_status check_dims(const starkv_dims* dims, Geometry* g) {
  if (!dims) return STARKV_E_NULL;
  if (dims->dtype != STARKV_F32 && dims->dtype != STARKV_BF16)
    return STARKV_E_DTYPE;
  const int64_t H = dims->H, G = dims->G, d = dims->d, L = dims->L,
                W = dims->W, nl = dims->n_layers;
  if (nl < 1 || nl > 4096) return STARKV_E_SHAPE;
  if (G < 1 || G > STARKV_MAX_GROUPS || H < G || H % G != 0 || H > 4096)
    return STARKV_E_SHAPE;
  if (d != 64 && d != 128) return STARKV_E_SHAPE;
  if (W < 1 || L > kMaxL || W >= L) return STARKV_E_SHAPE;
  const int64_t esz = dims->dtype == STARKV_F32 ? 4 : 2;
  const int64_t R = W * (H / G);
  const int64_t Rpad = (R + 31) / 32 * 32;
  if (Rpad > 512 || Rpad * (d * esz + 16) > kMaxQBytes) return STARKV_E_SHAPE;
  if (esz == 4 && Rpad > 128) return STARKV_E_SHAPE;   // float32: up to 4 row blocks
  // per-head subspaces: a head's window rows must be whole 8-row groups of
  // the MFMA output, and the subspaces must fit the statistics kernels
  if (dims->per_head != 0 && dims->per_head != 1) return STARKV_E_SHAPE;
  if (dims->per_head && (H > STARKV_MAX_GROUPS || W % 8 != 0)) return STARKV_E_SHAPE;
  if (g) {
    g->n_layers = (int)nl;
    g->H = (int)H;
    g->G = (int)G;
    g->d = (int)d;
    g->L = (int)L;
    g->W = (int)W;
    g->Lp = (int)(L - W);
    g->R = (int)R;
    g->Rpad = (int)Rpad;
    g->esz = (int)esz;
    g->dtype = dims->dtype;
    g->Ns = dims->per_head ? (int)H : (int)G;
    g->hps = (int)(H / g->Ns);
  }
  return STARKV_OK;
}

static bool finite(float x) { return std::isfinite(x); }

starkv_status check_pool(const starkv_params* p) {
  if (!p) return STARKV_E_NULL;
  if (p->pool_kernel < 1 || p->pool_kernel > 63 || p->pool_kernel % 2 == 0)
    return STARKV_E_PARAM;
  return STARKV_OK;
}

starkv_status check_params(const starkv_params* p) {
  if (!p) return STARKV_E_NULL;
  if (!finite(p->lam) || p->lam < 0.f || p->lam > 1.f) return STARKV_E_PARAM;
  if (p->n_warmup < 0 || p->n_ramp < 0) return STARKV_E_PARAM;
  if (!finite(p->rho_mi) || p->rho_mi < 0.f || p->rho_mi >= 1.f)
    return STARKV_E_PARAM;
  if (!finite(p->rho_t) || p->rho_t < 0.f || p->rho_t >= 1.f)
    return STARKV_E_PARAM;
  if (!finite(p->tau) || p->tau <= 0.f) return STARKV_E_PARAM;
  if (!finite(p->delta) || p->delta < 0.f) return STARKV_E_PARAM;
  if (!finite(p->d_min) || p->d_min < 0.f || p->d_min > 1.f)
    return STARKV_E_PARAM;
  if (!finite(p->t_min) || !finite(p->t_max) || p->t_min <= 0.f ||
      p->t_max < p->t_min)
    return STARKV_E_PARAM;
  if (p->n_bins < 1 || p->n_bins > 64) return STARKV_E_PARAM;
  if (p->grid < 1 || p->grid > 16) return STARKV_E_PARAM;
  if (!finite(p->eps) || p->eps < 0.f) return STARKV_E_PARAM;
  if (p->tem_decay < STARKV_TEM_EXP || p->tem_decay > STARKV_TEM_GAMMA) return STARKV_E_PARAM;
  if (p->aeb_mode < STARKV_AEB_ENTROPY || p->aeb_mode > STARKV_AEB_CONFIDENCE)
    return STARKV_E_PARAM;
  return check_pool(p);
}

starkv_status check_spans(const starkv_span* spans, int32_t n_spans,
                          int32_t frame, int Lp) {
  if (n_spans < 0 || n_spans > STARKV_MAX_SPANS) return STARKV_E_SPANS;
  if (n_spans == 0) return STARKV_OK;
  if (!spans) return STARKV_E_NULL;
  int64_t prev_end = 0;
  bool has_frame = false;
  for (int i = 0; i < n_spans; ++i) {
    const starkv_span& s = spans[i];
    if (s.rows < 1 || s.cols < 1 || s.start < 0) return STARKV_E_SPANS;
    const int64_t n = (int64_t)s.rows * s.cols;
    if (s.start < prev_end) return STARKV_E_SPANS;  // unsorted or overlapping
    if ((int64_t)s.start + n > Lp) return STARKV_E_SPANS;
    if (s.frame > frame) return STARKV_E_SPANS;
    for (int j = 0; j < i; ++j)
      if (spans[j].frame == s.frame) return STARKV_E_SPANS;
    if (s.frame == frame) has_frame = true;
    prev_end = (int64_t)s.start + n;
  }
  if (!has_frame) return STARKV_E_SPANS;
  return STARKV_OK;
}

starkv_status check_layout(const starkv_kv_layout* lay, const Geometry& g) {
  if (!lay) return STARKV_E_NULL;
  if (lay->layer_stride < 0 || lay->group_stride < 0 || lay->token_stride < g.d)
    return STARKV_E_SHAPE;
  if ((lay->layer_stride * g.esz) % 16 || (lay->group_stride * g.esz) % 16 ||
      (lay->token_stride * g.esz) % 16)
    return STARKV_E_ALIGN;
  return STARKV_OK;
}

int current_span(const starkv_span* spans, int32_t n_spans, int32_t frame) {
  for (int i = 0; i < n_spans; ++i)
    if (spans[i].frame == frame) return i;
  return -1;
}

int max_chunks(const Geometry& g) { return (g.Lp + kMinChunk - 1) / kMinChunk; }

static size_t up256(size_t x) { return (x + 255) / 256 * 256; }

WsLayout ws_layout(const Geometry& g) {
  WsLayout w;
  const size_t lg = (size_t)g.n_layers * g.G;
  w.part_off = 0;
  w.sraw_off = up256(lg * max_chunks(g) * g.Rpad * 2 * sizeof(float));
  w.total = w.sraw_off + up256((size_t)g.n_layers * g.Ns * g.Lp * sizeof(float));
  return w;
}

size_t scalars_count(int G) { return 4 * (size_t)G + 4; }

starkv_status check_decode(const starkv_dims* dims, int32_t n_tokens, DecodeGeometry* g) {
  if (!dims) return STARKV_E_NULL;
  if (dims->dtype != STARKV_F32 && dims->dtype != STARKV_BF16) return STARKV_E_DTYPE;
  if (dims->dtype != STARKV_BF16) return STARKV_E_DTYPE;   // bf16 caches only
  const int64_t H = dims->H, G = dims->G, d = dims->d, nl = dims->n_layers;
  if (nl < 1 || nl > 4096) return STARKV_E_SHAPE;
  if (G < 1 || G > STARKV_MAX_GROUPS || H < G || H % G != 0 || H / G > 16)
    return STARKV_E_SHAPE;
  if (d != 64 && d != 128) return STARKV_E_SHAPE;
  if (n_tokens < 1 || n_tokens > kMaxL) return STARKV_E_SHAPE;
  if (g) {
    g->n_layers = (int)nl;
    g->H = (int)H;
    g->G = (int)G;
    g->d = (int)d;
    g->n_tok = n_tokens;
    // about 256 tokens (two tiles per wave) per block, at most ~4096 blocks:
    // enough blocks in flight to cover the HBM latency of a short cache
    const int64_t cap = std::max<int64_t>(1, 4096 / (nl * G));
    int64_t ns = std::min<int64_t>((n_tokens + 255) / 256, cap);
    int64_t chunk = (n_tokens + ns - 1) / ns;
    chunk = (chunk + 31) / 32 * 32;
    g->chunk = (int)chunk;
    g->n_split = (int)((n_tokens + chunk - 1) / chunk);
  }
  return STARKV_OK;
}

size_t decode_ws_bytes(const DecodeGeometry& g) {
  return up256((size_t)g.n_layers * g.G * g.n_split * (g.H / g.G) * (g.d + 2) * sizeof(float));
}

size_t state_mibar_off() { return sizeof(StateHeader); }
size_t state_m_off(int G) {
  return sizeof(StateHeader) + ((size_t)G * 4 + 15) / 16 * 16;
}
size_t state_stride(int G, int frame_cap) {
  return up256(state_m_off(G) + (size_t)G * frame_cap * 4);
}

}  // namespace starkv
