// Final score and global top-B (Eq. final_score, sec. 3.2; sec. 3.5 discount;
// sec. 3.7 selection).  One 1024-thread workgroup per layer:
//   1. s_t = max(sbar_t * beta_t * D_t, 0)^(1/T) for every past token,
//      written out and kept as a descending-order key in LDS;
//   2. MSB-first radix select (8-bit digits) of the B-th key in the order
//      (s descending, token index ascending);
//   3. one ordered pass in token order flags the selected tokens (keys past
//      the cut, plus the lowest-index ties at the cut) and compacts them with
//      a block scan, so idx comes out ascending.
#include "device_common.h"
#include "internal.h"

namespace starkv {
namespace {

constexpr int kThreads = 1024;
constexpr int kLdsKeys = 28 * 1024;   // keys cached in LDS (112 KiB)

struct SelArgs {
  const float* sbar;
  const uint8_t* gstar;
  const float* scal;
  float* s;
  int32_t* idx;
  int G, Lp, B, sc, frame, cache;
  float delta, d_min;
  int n_spans;
  int32_t start[STARKV_MAX_SPANS];
  int32_t end[STARKV_MAX_SPANS];
  int32_t sframe[STARKV_MAX_SPANS];
};

// Span holding token t, or -1 (spans sorted by start, disjoint).
__device__ inline int find_span(const SelArgs& a, int t) {
  if (a.n_spans == 0 || t < a.start[0]) return -1;
  int lo = 0, hi = a.n_spans - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.start[mid] <= t) lo = mid; else hi = mid - 1;
  }
  return t < a.end[lo] ? lo : -1;
}

__global__ __launch_bounds__(kThreads) void select_kernel(SelArgs a) {
  extern __shared__ __align__(16) uint32_t keys[];
  __shared__ int hist[256];
  __shared__ float w_s[STARKV_MAX_GROUPS], phi_s[STARKV_MAX_GROUPS];
  __shared__ uint32_t cut_key;
  __shared__ int cut_rank, cut_eq;
  __shared__ int sh_cnt[kThreads / 64];

  const int layer = blockIdx.x, tid = threadIdx.x;
  const float* scal = a.scal + (size_t)layer * a.sc;
  const float* sb = a.sbar + (size_t)layer * a.Lp;
  const uint8_t* gs = a.gstar + (size_t)layer * a.Lp;
  float* s_out = a.s + (size_t)layer * a.Lp;
  if (tid < a.G) {
    w_s[tid] = scal[STARKV_SCAL_W(a.G) + tid];
    phi_s[tid] = scal[STARKV_SCAL_PHI(a.G) + tid];
  }
  __syncthreads();
  const float lam = scal[STARKV_SCAL_LAMBDA(a.G)];
  const float T = scal[STARKV_SCAL_T(a.G)];
  const float inv_t = 1.0f / T;
  const float gl = (float)a.G * lam;

  // ---- 1. fused score
  for (int t = tid; t < a.Lp; t += kThreads) {
    const int g = min((int)gs[t], a.G - 1);
    const float beta = (1.0f - lam) + gl * w_s[g];
    float D = 1.0f;
    const int sp = find_span(a, t);
    if (sp >= 0) {
      const float dist = (float)(a.frame - a.sframe[sp]);
      D = a.d_min + (1.0f - a.d_min) * expf(-a.delta * dist * phi_s[g]);
    }
    const float sf = fmaxf(sb[t] * beta * D, 0.0f);
    const float sv = (inv_t == 1.0f || sf == 0.0f) ? sf : exp2f(inv_t * log2f(sf));
    s_out[t] = sv;
    if (t < a.cache) keys[t] = ~fkey(sv);
  }
  if (a.B == 0) return;
  __syncthreads();

  // ---- 2. radix select of rank B-1 in ascending ~key (= descending s)
  if (tid == 0) {
    cut_key = 0u;
    cut_rank = a.B - 1;
  }
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    const uint32_t hi_want = pass == 0 ? 0u : (cut_key >> (shift + 8));
    for (int t = tid; t < a.Lp; t += kThreads) {
      const uint32_t k = t < a.cache ? keys[t] : ~fkey(s_out[t]);
      const uint32_t hi = pass == 0 ? 0u : (k >> (shift + 8));
      if (hi == hi_want) atomicAdd(&hist[(k >> shift) & 255], 1);
    }
    __syncthreads();
    if (tid == 0) {
      int cum = 0;
      const int rank = cut_rank;
      for (int dg = 0; dg < 256; ++dg) {
        const int c = hist[dg];
        if (cum + c > rank) {
          cut_key |= (uint32_t)dg << shift;
          cut_rank = rank - cum;
          cut_eq = c;
          break;
        }
        cum += c;
      }
    }
    __syncthreads();
  }

  // ---- 3. ordered flag + compaction
  const uint32_t ck = cut_key;
  const int crank = cut_rank;
  const bool ties = cut_eq > 1;
  int32_t* out = a.idx + (size_t)layer * a.B;
  int carry = 0, carry_eq = 0;
  for (int base = 0; base < a.Lp; base += kThreads) {
    const int t = base + tid;
    uint32_t k = 0xFFFFFFFFu;
    if (t < a.Lp) k = t < a.cache ? keys[t] : ~fkey(s_out[t]);
    bool sel = (t < a.Lp) && (k < ck);
    if (ties) {
      const bool eq = (t < a.Lp) && (k == ck);
      int tot;
      const int pos = block_excl_count(eq, sh_cnt, &tot) + carry_eq;
      carry_eq += tot;
      sel = sel || (eq && pos <= crank);
    } else {
      sel = sel || ((t < a.Lp) && (k == ck));
    }
    int tot;
    const int pos = block_excl_count(sel, sh_cnt, &tot) + carry;
    carry += tot;
    if (sel && pos < a.B) out[pos] = t;
  }
}

}  // namespace

int launch_select(const Geometry& g, const starkv_params& p, const float* sbar,
                  const uint8_t* gstar, const float* scalars,
                  const starkv_span* spans, int32_t n_spans, int32_t frame,
                  int32_t B, float* s, int32_t* idx, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  SelArgs a;
  a.sbar = sbar;
  a.gstar = gstar;
  a.scal = scalars;
  a.s = s;
  a.idx = idx;
  a.G = g.G;
  a.Lp = g.Lp;
  a.B = B;
  a.sc = (int)scalars_count(g.G);
  a.frame = frame;
  a.cache = g.Lp < kLdsKeys ? g.Lp : kLdsKeys;
  a.delta = p.delta;
  a.d_min = p.d_min;
  a.n_spans = n_spans;
  for (int i = 0; i < n_spans; ++i) {
    a.start[i] = spans[i].start;
    a.end[i] = spans[i].start + spans[i].rows * spans[i].cols;
    a.sframe[i] = spans[i].frame;
  }
  const size_t lds = (size_t)a.cache * sizeof(uint32_t);
  hipFuncSetAttribute(reinterpret_cast<const void*>(&select_kernel),
                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  select_kernel<<<g.n_layers, kThreads, lds, st>>>(a);
  return (int)hipGetLastError();
}

}  // namespace starkv
