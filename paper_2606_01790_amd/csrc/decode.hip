// Decode attention over a (compressed) KV cache, the step that follows the
// compression stage (sec. 4.3, decode-time efficiency): one new query token
// per head attends to the n cached tokens of its KV group,
//   o[h] = sum_t softmax_t(q[h] . K[g(h),t] / sqrt(d)) V[g(h),t].
//
// Split-token scheme: a block takes one token range of one (layer, group)
// and all H/G heads of the group, so every K and V row is read from HBM
// once for the whole group.  Its 4 waves take the range's 32-token tiles
// round-robin, each with its own running (max, sum, output) per head:
//   q . K   on v_mfma_f32_16x16x32_bf16, the group's heads as the 16 rows of
//           A (zero past H/G) and 16 tokens as the columns of B, read
//           straight from the cache rows (8 consecutive d per lane);
//   softmax per head over the tile (16-lane reductions), in fp32;
//   P . V   on the VALU in fp32: each lane owns D/64 columns of d and adds
//           p[t][h] * V[t][col] for every token of the tile, the p row of
//           a token read from LDS as a broadcast.
// The waves are merged through LDS into one partial (output, max, sum) per
// (split, head), and a second kernel merges the splits of each head in
// split order.
#include "device_common.h"
#include "internal.h"

namespace starkv {
namespace {

typedef float f32x4v __attribute__((ext_vector_type(4)));

constexpr int kDecThreads = 256;
constexpr int kDecWaves = kDecThreads / 64;
constexpr int kTile = 32;

struct DecArgs {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  int64_t ls, gs, ts;   // element strides of the caches
  int H, G, hpg, n_tok, chunk, n_split;
  float scale;          // log2(e) / sqrt(d)
  float* part;          // [n_layers][G][n_split][hpg][D + 2]: output, max*scale, sum
  float* out;           // [n_layers][H][D]
};

__device__ inline float rescale2(float m, float mn, float scale) {
  return m == mn ? 1.0f : __builtin_amdgcn_exp2f((m - mn) * scale);
}

// Orders one wave's LDS writes before its later LDS reads (and the reads
// before the next writes) for the compiler: lanes of the wave exchange the
// p rows and rescale factors through LDS, which the hardware executes in
// program order within the wave, but without a fence the compiler may move
// a load above another lane's store.
__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// max and sum over the 16 lanes of a lane row (l / 16 fixed)
__device__ inline float row16_max(float v) {
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ inline float row16_sum(float v) {
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

template <int D, int HP>
__global__ __launch_bounds__(kDecThreads) void decode_split(DecArgs a) {
  constexpr int NK = D / 32;      // MFMA k-steps over d
  constexpr int NC = D / 64;      // d columns per lane in P.V
  __shared__ __align__(16) float pt[kDecWaves][kTile][HP];   // p[token][head] per wave
  __shared__ __align__(16) float al[kDecWaves][HP];          // rescale factor per head
  __shared__ float mw[kDecWaves][HP], lw[kDecWaves][HP];
  __shared__ float ow[kDecWaves][HP][D];

  const int split = blockIdx.x, g = blockIdx.y, layer = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, quad = lane >> 4;
  const __bf16* kg = a.k + (int64_t)layer * a.ls + (int64_t)g * a.gs;
  const __bf16* vg = a.v + (int64_t)layer * a.ls + (int64_t)g * a.gs;
  const int c0 = split * a.chunk;
  const int c1 = min(c0 + a.chunk, a.n_tok);

  // A operand: row l16 = head g*hpg + l16 (zero past hpg), k = 32kk + 8quad..
  bf16x8 qf[NK];
  {
    const int h = min(l16, a.hpg - 1);
    const __bf16* qr = a.q + ((size_t)layer * a.H + (size_t)g * a.hpg + h) * D;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      qf[kk] = *reinterpret_cast<const bf16x8*>(qr + 32 * kk + 8 * quad);
      if (l16 >= a.hpg) qf[kk] = bf16x8{};
    }
  }
  // running statistics of heads 4*quad + i (replicated over the lane row)
  float m[4], l[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) { m[i] = -INFINITY; l[i] = 0.f; }
  float o[HP][NC];
#pragma unroll
  for (int h = 0; h < HP; ++h)
#pragma unroll
    for (int c = 0; c < NC; ++c) o[h][c] = 0.f;

  const int n_tiles = (c1 - c0 + kTile - 1) / kTile;
  for (int tile = wave; tile < n_tiles; tile += kDecWaves) {
    const int t0 = c0 + tile * kTile;
    // K rows of the tile's two 16-token halves; token indices clamped to the
    // cache (the logits of tokens past c1 are masked below)
    bf16x8 kf[2][NK];
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      const int tok = min(t0 + 16 * h2 + l16, a.n_tok - 1);
      const __bf16* kr = kg + (int64_t)tok * a.ts + 8 * quad;
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) kf[h2][kk] = *reinterpret_cast<const bf16x8*>(kr + 32 * kk);
    }
    // this lane's V columns of every token of the tile
    uint32_t vv[kTile];
#pragma unroll
    for (int j = 0; j < kTile; ++j) {
      const int tok = min(t0 + j, a.n_tok - 1);
      const __bf16* vr = vg + (int64_t)tok * a.ts + NC * lane;
      if (NC == 2) vv[j] = *reinterpret_cast<const uint32_t*>(vr);
      else vv[j] = *reinterpret_cast<const uint16_t*>(vr);
    }
    f32x4v acc[2];
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      acc[h2] = f32x4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < NK; ++kk)
        acc[h2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[kk], kf[h2][kk], acc[h2], 0, 0, 0);
      if (t0 + 16 * h2 + l16 >= c1) acc[h2] = f32x4v{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    }
    // online softmax per head 4*quad + i; every tile has a valid token
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float mt = row16_max(fmaxf(acc[0][i], acc[1][i]));
      const float mn = fmaxf(m[i], mt);
      const float ms = mn * a.scale;
      const float p0 = __builtin_amdgcn_exp2f(fmaf(acc[0][i], a.scale, -ms));
      const float p1 = __builtin_amdgcn_exp2f(fmaf(acc[1][i], a.scale, -ms));
      const float alpha = rescale2(m[i], mn, a.scale);
      l[i] = l[i] * alpha + row16_sum(p0 + p1);
      m[i] = mn;
      const int h = 4 * quad + i;
      if (h < HP) {
        pt[wave][l16][h] = p0;
        pt[wave][16 + l16][h] = p1;
        if (l16 == 0) al[wave][h] = alpha;
      }
    }
    // the p rows and factors are read back by other lanes of the same wave
    wave_sync();
#pragma unroll
    for (int h = 0; h < HP; ++h) {
      const float f = al[wave][h];
#pragma unroll
      for (int c = 0; c < NC; ++c) o[h][c] *= f;
    }
#pragma unroll
    for (int j = 0; j < kTile; ++j) {
      float vc[NC];
      if (NC == 2) {
        vc[0] = __uint_as_float(vv[j] << 16);
        vc[NC - 1] = __uint_as_float(vv[j] & 0xFFFF0000u);
      } else {
        vc[0] = __uint_as_float(vv[j] << 16);
      }
      float pr[HP];
#pragma unroll
      for (int h4 = 0; h4 < HP; h4 += 4) {
        if (HP >= 4) {
          const f32x4v p4 = *reinterpret_cast<const f32x4v*>(&pt[wave][j][h4]);
#pragma unroll
          for (int u = 0; u < 4; ++u) pr[h4 + u] = p4[u];
        } else {
#pragma unroll
          for (int u = 0; u < HP; ++u) pr[u] = pt[wave][j][u];
        }
      }
#pragma unroll
      for (int h = 0; h < HP; ++h)
#pragma unroll
        for (int c = 0; c < NC; ++c) o[h][c] = fmaf(pr[h], vc[c], o[h][c]);
    }
    wave_sync();   // every lane's reads of this tile before the next tile's writes
  }

  // merge the waves: per head the largest max, then the rescaled sums
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int h = 4 * quad + i;
    if (h < HP && l16 == 0) { mw[wave][h] = m[i]; lw[wave][h] = l[i]; }
  }
#pragma unroll
  for (int h = 0; h < HP; ++h)
#pragma unroll
    for (int c = 0; c < NC; ++c) ow[wave][h][NC * lane + c] = o[h][c];
  __syncthreads();
  float* base = a.part + (((size_t)layer * a.G + g) * a.n_split + split) * a.hpg * (D + 2);
  for (int it = threadIdx.x; it < a.hpg * D; it += kDecThreads) {
    const int h = it / D, d = it % D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, mw[w][h]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      const float f = mw[w][h] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((mw[w][h] - M) * a.scale);
      L += lw[w][h] * f;
      O += ow[w][h][d] * f;
    }
    float* rec = base + (size_t)h * (D + 2);
    rec[d] = O;
    if (d == 0) { rec[D] = M * a.scale; rec[D + 1] = L; }
  }
}

// o[layer][h] from the split partials of head h, combined in split order.
template <int D>
__global__ __launch_bounds__(D) void decode_merge(DecArgs a) {
  const int h = blockIdx.x, layer = blockIdx.y, d = threadIdx.x;
  const int g = h / a.hpg, hl = h % a.hpg;
  const float* base = a.part + ((size_t)layer * a.G + g) * a.n_split * a.hpg * (D + 2) +
                      (size_t)hl * (D + 2);
  const size_t rs = (size_t)a.hpg * (D + 2);   // record stride between splits
  // one pass with a running max, sixteen splits' loads in flight at a time
  float M = -INFINITY, L = 0.f, O = 0.f;
  for (int s0 = 0; s0 < a.n_split; s0 += 16) {
    float mv[16], lv[16], ov[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const bool ok = s0 + j < a.n_split;
      const float* rec = base + (s0 + j) * rs;
      mv[j] = ok ? rec[D] : -INFINITY;
      lv[j] = ok ? rec[D + 1] : 0.f;
      ov[j] = ok ? rec[d] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (mv[j] == -INFINITY) continue;   // past the last split
      const float Mn = fmaxf(M, mv[j]);
      const float fo = M == Mn ? 1.0f : __builtin_amdgcn_exp2f(M - Mn);
      const float fj = __builtin_amdgcn_exp2f(mv[j] - Mn);
      L = L * fo + lv[j] * fj;
      O = O * fo + ov[j] * fj;
      M = Mn;
    }
  }
  a.out[((size_t)layer * a.H + h) * D + d] = O / L;
}

template <int D, int HP>
void launch_split(const DecArgs& a, int n_layers, hipStream_t st) {
  decode_split<D, HP><<<dim3(a.n_split, a.G, n_layers), kDecThreads, 0, st>>>(a);
}

template <int D>
void launch_d(const DecArgs& a, int n_layers, hipStream_t st) {
  if (a.hpg <= 1) launch_split<D, 1>(a, n_layers, st);
  else if (a.hpg <= 2) launch_split<D, 2>(a, n_layers, st);
  else if (a.hpg <= 4) launch_split<D, 4>(a, n_layers, st);
  else if (a.hpg <= 8) launch_split<D, 8>(a, n_layers, st);
  else launch_split<D, 16>(a, n_layers, st);
  decode_merge<D><<<dim3(a.H, n_layers), D, 0, st>>>(a);
}

}  // namespace

int launch_decode(const DecodeGeometry& g, const void* q, const void* k, const void* v,
                  const starkv_kv_layout& lay, float* out, void* ws, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  DecArgs a;
  a.q = static_cast<const __bf16*>(q);
  a.k = static_cast<const __bf16*>(k);
  a.v = static_cast<const __bf16*>(v);
  a.ls = lay.layer_stride;
  a.gs = lay.group_stride;
  a.ts = lay.token_stride;
  a.H = g.H;
  a.G = g.G;
  a.hpg = g.H / g.G;
  a.n_tok = g.n_tok;
  a.n_split = g.n_split;
  a.chunk = g.chunk;
  a.scale = 1.4426950408889634f / sqrtf((float)g.d);
  a.part = static_cast<float*>(ws);
  a.out = out;
  if (g.d == 128) launch_d<128>(a, g.n_layers, st);
  else launch_d<64>(a, g.n_layers, st);
  return (int)hipGetLastError();
}

}  // namespace starkv
