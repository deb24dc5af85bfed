// Window attention scoring (sec. 3.3, Eqs. A_raw and base_score): launch
// sequence, pooling and group aggregation.  The two MFMA passes and the
// merge of their row statistics live in score_kernels.h.
#include <algorithm>

#include "score_kernels.h"

namespace starkv {
namespace {

// ---------------------------------------------------------------- pooling
// S[g,t] = (1/(k*hps)) sum_{|j|<=k/2} S_raw[g,t+j] (zero outside [0,L_p))
// for each of the G scoring subspaces (hps heads each), sbar = mean over
// subspaces, g* = first argmax.  The pooled sum adds the k window values in
// token order; the mean and the argmax take the subspaces in order.
constexpr int kAggChunk = 8;   // subspaces per LDS tile
constexpr int kAggMaxRadius = 31;   // pool widths up to 63
// loads per thread that fill one tile: every one is issued before the first
// LDS store, so a tile costs one round trip
constexpr int kAggLoads = (kAggChunk * (256 + 2 * kAggMaxRadius) + 255) / 256;

__global__ __launch_bounds__(256) void score_aggregate(const float* sraw, float* S,
                                                       float* sbar, uint8_t* gstar,
                                                       int G, int Lp, int radius,
                                                       float inv_norm, float inv_g) {
  // the block's 256 tokens plus the pooling halo, for up to kAggChunk
  // subspaces at a time, in LDS (a small tile keeps many blocks per CU when
  // there is a subspace per head)
  extern __shared__ float tile[];
  const int layer = blockIdx.y;
  const int t0 = blockIdx.x * 256;
  const int span = 256 + 2 * radius;
  const int t = t0 + threadIdx.x;
  float best = -INFINITY, total = 0.f;
  int bg = 0;
  for (int g0 = 0; g0 < G; g0 += kAggChunk) {
    const int ng = min(kAggChunk, G - g0);
    float v[kAggLoads];
#pragma unroll
    for (int j = 0; j < kAggLoads; ++j) {
      const int i = threadIdx.x + j * 256;
      const int g = g0 + i / span, u = t0 - radius + i % span;
      v[j] = (i < ng * span && u >= 0 && u < Lp) ? sraw[(size_t)(layer * G + g) * Lp + u] : 0.f;
    }
    if (g0 > 0) __syncthreads();   // the previous subspaces are read
#pragma unroll
    for (int j = 0; j < kAggLoads; ++j) {
      const int i = threadIdx.x + j * 256;
      if (i < ng * span) tile[i] = v[j];
    }
    __syncthreads();
    if (t < Lp) {
      for (int gi = 0; gi < ng; ++gi) {
        const int g = g0 + gi;
        const float* row = tile + gi * span + threadIdx.x;
        float acc = 0.f;
        for (int j = 0; j <= 2 * radius; ++j) acc += row[j];
        const float sv = acc * inv_norm;
        S[(size_t)(layer * G + g) * Lp + t] = sv;
        total += sv;
        if (sv > best) { best = sv; bg = g; }
      }
    }
  }
  if (t >= Lp) return;
  sbar[(size_t)layer * Lp + t] = total * inv_g;
  gstar[(size_t)layer * Lp + t] = (uint8_t)bg;
}

}  // namespace

int launch_score(const Geometry& g, const starkv_params& p, const void* q,
                 const void* k, const starkv_kv_layout& lay, float* S,
                 float* sbar, uint8_t* gstar, void* ws, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const WsLayout wl = ws_layout(g);
  ScoreArgs a;
  a.q = q;
  a.k = k;
  a.ls = lay.layer_stride;
  a.gs = lay.group_stride;
  a.ts = lay.token_stride;
  a.H = g.H;
  a.G = g.G;
  a.W = g.W;
  a.R = g.R;
  a.Rpad = g.Rpad;
  a.Lp = g.Lp;
  a.n_chunks_max = max_chunks(g);
  // Each block scores one contiguous token range of one (layer, group).
  // Up to 1024 blocks: two blocks per CU fit the LDS, so that is two full
  // rounds over the 256 CUs; ranges are at least 256 tokens so that the
  // window-query load stays a small fraction of the K traffic.
  const long nlg = (long)g.n_layers * g.G;
  long per_lg = 1024 / nlg;   // about two rounds of two blocks per CU
  per_lg = std::min<long>(per_lg, (g.Lp + kMinChunk - 1) / kMinChunk);
  per_lg = std::max<long>(per_lg, 1);
  int chunk = (int)((g.Lp + per_lg - 1) / per_lg);
  chunk = (chunk + 127) / 128 * 128;
  a.chunk = chunk;
  a.n_chunks = (g.Lp + chunk - 1) / chunk;
  a.scale = kLog2e / sqrtf((float)g.d);
  // per-head subspaces: head h of group g owns rows [h*W, (h+1)*W) of the
  // group's window rows, i.e. W/32 whole row blocks, or W/8 of the 8-row
  // groups a wave keeps apart
  a.Ns = g.Ns;
  a.n_out = g.Ns / g.G;
  if (a.n_out == 1) {
    a.n_part = 1;
    a.upo = g.Rpad / 32;
  } else {
    a.n_part = g.W % 32 == 0 ? 1 : 4;
    a.upo = g.W / (32 / a.n_part);
  }
  a.part = reinterpret_cast<float2*>(static_cast<char*>(ws) + wl.part_off);
  a.sraw = reinterpret_cast<float*>(static_cast<char*>(ws) + wl.sraw_off);

  const int err = g.dtype == STARKV_BF16 ? run_score_bf16(a, g.d, g.n_layers, st)
                                         : run_score_f32(a, g.d, g.n_layers, st);
  if (err) return err;
  const int radius = p.pool_kernel / 2;
  if (radius > kAggMaxRadius) return (int)hipErrorInvalidValue;   // validated before
  const float inv_norm = 1.0f / ((float)p.pool_kernel * (float)g.hps);
  dim3 ag((g.Lp + 255) / 256, g.n_layers);
  const size_t lds = (size_t)std::min(g.Ns, kAggChunk) * (256 + 2 * radius) * sizeof(float);
  score_aggregate<<<ag, 256, lds, st>>>(a.sraw, S, sbar, gstar, g.Ns, g.Lp, radius,
                                        inv_norm, 1.0f / (float)g.Ns);
  return (int)hipGetLastError();
}

}  // namespace starkv
