// Window attention scoring (sec. 3.3): A_raw summed over the window rows and
// the heads of each KV group, then AvgPool1D, group mean, sbar and g*.
//
// The window softmax of every query row needs that row's max and sum over
// all L_p past keys before any key's normalised mass is known, so scoring
// runs in two passes over K:
//   pass 1  per (layer, group, token chunk): for each window row r, the
//           chunk's max M_r and sum of 2^(y - M_r), y = q.k * log2(e)/sqrt(d);
//   pass 2  merges the chunk statistics into c_r = M_r + log2(l_r) and sums
//           2^(y_rt - c_r) over the group's rows for every token t.
// Both passes run the Q_g x K^T contraction on 32x32 MFMA tiles: the R = W*H/G
// window rows of group g sit in LDS, K rows stream straight from HBM into
// MFMA fragments.  Pass 1 puts tokens on the MFMA M axis, so each lane owns one
// query row and reduces over its tokens in registers.  Pass 2 puts query rows
// on M, so each lane owns one token and reduces over its rows in registers.
#include "device_common.h"
#include "internal.h"

namespace starkv {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegBig = -1e30f;

struct ScoreArgs {
  const void* q;
  const void* k;
  int64_t ls, gs, ts;   // element strides of the K cache
  int H, G, W, R, Rpad, Lp;
  int chunk, n_chunks, n_chunks_max;
  float scale;          // log2(e) / sqrt(d)
  float2* part;         // [n_layers][G][n_chunks_max][Rpad]  (M, l)
  float* sraw;          // [n_layers][G][Lp]
};

template <typename T, int D>
struct QTile {
  static constexpr int kStride = D + 16 / (int)sizeof(T);   // padded LDS row
  static constexpr int kVecPerRow = D * (int)sizeof(T) / 16;
  static constexpr int kElemPerVec = 16 / (int)sizeof(T);
  // Copy the R window rows of one group into LDS, zero rows R..Rpad.
  __device__ static void load(const T* qg, T* qs, int R, int Rpad) {
    const int nvec = Rpad * kVecPerRow;
    for (int v = threadIdx.x; v < nvec; v += blockDim.x) {
      const int row = v / kVecPerRow, part = v % kVecPerRow;
      int4 val = make_int4(0, 0, 0, 0);
      if (row < R)
        val = *reinterpret_cast<const int4*>(qg + (size_t)row * D + part * kElemPerVec);
      *reinterpret_cast<int4*>(qs + row * kStride + part * kElemPerVec) = val;
    }
  }
};

template <typename T, int D>
__device__ inline const T* group_q(const ScoreArgs& a, int layer, int g) {
  return reinterpret_cast<const T*>(a.q) +
         ((size_t)layer * a.H + (size_t)g * (a.H / a.G)) * (size_t)a.W * D;
}

template <typename T>
__device__ inline const T* group_k(const ScoreArgs& a, int layer, int g) {
  return reinterpret_cast<const T*>(a.k) + (int64_t)layer * a.ls + (int64_t)g * a.gs;
}

// 2^((m - mn) * scale) for a running max m <= mn, ms = mn * scale.  Exactly 1
// when the max did not move: with the -1e30 start value the fma would
// otherwise return the rounding residual of the product, not 0.
__device__ inline float rescale(float m, float mn, float ms, float scale) {
  return m == mn ? 1.0f : __builtin_amdgcn_exp2f(fmaf(m, scale, -ms));
}

// ---------------------------------------------------------------- pass 1
template <typename T, int D, int NRBM>
__global__ __launch_bounds__(256) void score_pass1(ScoreArgs a) {
  using M = Mfma<T>;
  using QT = QTile<T, D>;
  constexpr int NK = D / M::kStep;
  extern __shared__ __align__(16) unsigned char smem[];
  T* qs = reinterpret_cast<T*>(smem);
  float2* red = reinterpret_cast<float2*>(smem + (size_t)a.Rpad * QT::kStride * sizeof(T));

  const int chunk = blockIdx.x, g = blockIdx.y, layer = blockIdx.z;
  const int nrb = a.Rpad / 32;
  QT::load(group_q<T, D>(a, layer, g), qs, a.R, a.Rpad);
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const T* kg = group_k<T>(a, layer, g);
  const int t_begin = chunk * a.chunk;
  const int t_end = min(t_begin + a.chunk, a.Lp);

  float m[NRBM], l[NRBM];
#pragma unroll
  for (int rb = 0; rb < NRBM; ++rb) { m[rb] = kNegBig; l[rb] = 0.f; }

  for (int tb = t_begin + wave * 32; tb < t_end; tb += 4 * 32) {
    const int tok = min(tb + l32, a.Lp - 1);
    const T* krow = kg + (int64_t)tok * a.ts;
    typename M::frag kf[NK];
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) kf[kk] = M::load(krow, kk, half);
#pragma unroll
    for (int rb = 0; rb < NRBM; ++rb) {
      if (rb < nrb) {
        const T* qrow = qs + (rb * 32 + l32) * QT::kStride;
        f32x16 acc = {};
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) acc = M::mma(kf[kk], M::load(qrow, kk, half), acc);
        // acc[4i+j]: token tb + 8i + 4*half + j, query row rb*32 + l32
        float mt = -INFINITY;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int t = tb + 8 * (e >> 2) + 4 * half + (e & 3);
          const float v = (t < t_end) ? acc[e] : -INFINITY;
          acc[e] = v;
          mt = fmaxf(mt, v);
        }
        const float mn = fmaxf(m[rb], mt);
        const float ms = mn * a.scale;
        float sum = 0.f;
#pragma unroll
        for (int e = 0; e < 16; ++e) sum += __builtin_amdgcn_exp2f(fmaf(acc[e], a.scale, -ms));
        l[rb] = l[rb] * rescale(m[rb], mn, ms, a.scale) + sum;
        m[rb] = mn;
      }
    }
  }
  // merge the two lane halves (same query row, other tokens), then waves
#pragma unroll
  for (int rb = 0; rb < NRBM; ++rb) {
    if (rb < nrb) {
      const float mo = __shfl_xor(m[rb], 32), lo = __shfl_xor(l[rb], 32);
      const float mn = fmaxf(m[rb], mo);
      const float ms = mn * a.scale;
      l[rb] = l[rb] * rescale(m[rb], mn, ms, a.scale) + lo * rescale(mo, mn, ms, a.scale);
      m[rb] = mn;
      if (half == 0) red[wave * a.Rpad + rb * 32 + l32] = make_float2(mn * a.scale, l[rb]);
    }
  }
  __syncthreads();
  float2* out = a.part + ((size_t)(layer * a.G + g) * a.n_chunks_max + chunk) * a.Rpad;
  for (int r = threadIdx.x; r < a.Rpad; r += blockDim.x) {
    float Mx = kNegBig, lx = 0.f;
    for (int w = 0; w < 4; ++w) {
      const float2 p = red[w * a.Rpad + r];
      const float mn = fmaxf(Mx, p.x);
      lx = lx * __builtin_amdgcn_exp2f(Mx - mn) + p.y * __builtin_amdgcn_exp2f(p.x - mn);
      Mx = mn;
    }
    out[r] = make_float2(Mx, lx);
  }
}

// ---------------------------------------------------------------- pass 2
template <typename T, int D, int NRBM>
__global__ __launch_bounds__(256) void score_pass2(ScoreArgs a) {
  using M = Mfma<T>;
  using QT = QTile<T, D>;
  constexpr int NK = D / M::kStep;
  extern __shared__ __align__(16) unsigned char smem[];
  T* qs = reinterpret_cast<T*>(smem);
  float* cst = reinterpret_cast<float*>(smem + (size_t)a.Rpad * QT::kStride * sizeof(T));

  const int chunk = blockIdx.x, g = blockIdx.y, layer = blockIdx.z;
  const int nrb = a.Rpad / 32;
  QT::load(group_q<T, D>(a, layer, g), qs, a.R, a.Rpad);
  // c_r = M_r + log2(l_r) over all chunks, fixed merge order
  const float2* part = a.part + (size_t)(layer * a.G + g) * a.n_chunks_max * a.Rpad;
  for (int r = threadIdx.x; r < a.Rpad; r += blockDim.x) {
    float Mx = kNegBig, lx = 0.f;
    for (int c = 0; c < a.n_chunks; ++c) {
      const float2 p = part[(size_t)c * a.Rpad + r];
      const float mn = fmaxf(Mx, p.x);
      lx = lx * __builtin_amdgcn_exp2f(Mx - mn) + p.y * __builtin_amdgcn_exp2f(p.x - mn);
      Mx = mn;
    }
    cst[r] = (r < a.R) ? Mx + log2f(lx) : INFINITY;
  }
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const T* kg = group_k<T>(a, layer, g);
  const int t_begin = chunk * a.chunk;
  const int t_end = min(t_begin + a.chunk, a.Lp);
  float* srow = a.sraw + (size_t)(layer * a.G + g) * a.Lp;

  for (int tb = t_begin + wave * 32; tb < t_end; tb += 4 * 32) {
    const int tok = tb + l32;
    const T* krow = kg + (int64_t)min(tok, a.Lp - 1) * a.ts;
    typename M::frag kf[NK];
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) kf[kk] = M::load(krow, kk, half);
    float tsum = 0.f;
#pragma unroll
    for (int rb = 0; rb < NRBM; ++rb) {
      if (rb < nrb) {
        const T* qrow = qs + (rb * 32 + l32) * QT::kStride;
        f32x16 acc = {};
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) acc = M::mma(M::load(qrow, kk, half), kf[kk], acc);
        // acc[4i+j]: query row rb*32 + 8i + 4*half + j, token tb + l32
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const f32x4 c4 = *reinterpret_cast<const f32x4*>(cst + rb * 32 + 8 * i + 4 * half);
#pragma unroll
          for (int j = 0; j < 4; ++j)
            tsum += __builtin_amdgcn_exp2f(fmaf(acc[4 * i + j], a.scale, -c4[j]));
        }
      }
    }
    tsum += __shfl_xor(tsum, 32);
    if (half == 0 && tok < t_end) srow[tok] = tsum;
  }
}

// ---------------------------------------------------------------- pooling
// S[g,t] = (1/(k*H/G)) sum_{|j|<=k/2} S_raw[g,t+j] (zero outside [0,L_p)),
// sbar = mean over groups, g* = first argmax.
__global__ __launch_bounds__(256) void score_aggregate(const float* sraw, float* S,
                                                       float* sbar, uint8_t* gstar,
                                                       int G, int Lp, int radius,
                                                       float inv_norm, float inv_g) {
  const int layer = blockIdx.y;
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= Lp) return;
  float best = -INFINITY, total = 0.f;
  int bg = 0;
  for (int g = 0; g < G; ++g) {
    const float* row = sraw + (size_t)(layer * G + g) * Lp;
    float acc = 0.f;
    for (int j = -radius; j <= radius; ++j) {
      const int u = t + j;
      if (u >= 0 && u < Lp) acc += row[u];
    }
    const float sv = acc * inv_norm;
    S[(size_t)(layer * G + g) * Lp + t] = sv;
    total += sv;
    if (sv > best) { best = sv; bg = g; }
  }
  sbar[(size_t)layer * Lp + t] = total * inv_g;
  gstar[(size_t)layer * Lp + t] = (uint8_t)bg;
}

template <typename T, int D, int NRBM>
int run_passes(const ScoreArgs& a, int n_layers, size_t lds1, size_t lds2,
               hipStream_t st) {
  dim3 grid(a.n_chunks, a.G, n_layers);
  hipFuncSetAttribute(reinterpret_cast<const void*>(&score_pass1<T, D, NRBM>),
                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds1);
  hipFuncSetAttribute(reinterpret_cast<const void*>(&score_pass2<T, D, NRBM>),
                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds2);
  score_pass1<T, D, NRBM><<<grid, 256, lds1, st>>>(a);
  score_pass2<T, D, NRBM><<<grid, 256, lds2, st>>>(a);
  return (int)hipGetLastError();
}

template <typename T, int D>
int run_nrb(const ScoreArgs& a, int n_layers, size_t lds1, size_t lds2, hipStream_t st) {
  const int nrb = a.Rpad / 32;
  if (nrb <= 1) return run_passes<T, D, 1>(a, n_layers, lds1, lds2, st);
  if (nrb <= 2) return run_passes<T, D, 2>(a, n_layers, lds1, lds2, st);
  if (nrb <= 4) return run_passes<T, D, 4>(a, n_layers, lds1, lds2, st);
  if (nrb <= 8) return run_passes<T, D, 8>(a, n_layers, lds1, lds2, st);
  return run_passes<T, D, 16>(a, n_layers, lds1, lds2, st);
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
  int chunk = kMinChunk;
  const long nlg = (long)g.n_layers * g.G;
  while (chunk < 2048 && nlg * ((g.Lp + chunk - 1) / chunk) > 2048) chunk *= 2;
  a.chunk = chunk;
  a.n_chunks = (g.Lp + chunk - 1) / chunk;
  a.scale = kLog2e / sqrtf((float)g.d);
  a.part = reinterpret_cast<float2*>(static_cast<char*>(ws) + wl.part_off);
  a.sraw = reinterpret_cast<float*>(static_cast<char*>(ws) + wl.sraw_off);

  const size_t qbytes = (size_t)g.Rpad * (g.d * g.esz + 16);
  const size_t lds1 = qbytes + (size_t)4 * g.Rpad * sizeof(float2);
  const size_t lds2 = qbytes + (size_t)g.Rpad * sizeof(float);
  int err;
  if (g.dtype == STARKV_BF16)
    err = g.d == 128 ? run_nrb<__bf16, 128>(a, g.n_layers, lds1, lds2, st)
                     : run_nrb<__bf16, 64>(a, g.n_layers, lds1, lds2, st);
  else
    err = g.d == 128 ? run_nrb<float, 128>(a, g.n_layers, lds1, lds2, st)
                     : run_nrb<float, 64>(a, g.n_layers, lds1, lds2, st);
  if (err) return err;
  const int radius = p.pool_kernel / 2;
  const float inv_norm = 1.0f / ((float)p.pool_kernel * (float)(g.H / g.G));
  dim3 ag((g.Lp + 255) / 256, g.n_layers);
  score_aggregate<<<ag, 256, 0, st>>>(a.sraw, S, sbar, gstar, g.G, g.Lp, radius,
                                      inv_norm, 1.0f / (float)g.G);
  return (int)hipGetLastError();
}

}  // namespace starkv
