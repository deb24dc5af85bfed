// Online statistics of one step (sec. 3.4-3.6).
//
// stats kernel, G + 1 + ceil(G / 8) blocks per layer, 1024 threads (512 or
// 256 when the blocks outnumber the CUs, see StatsShape), where G is the
// call's number of scoring subspaces (the KV groups, or the query heads).
// Block g of a layer computes:
//   g < G       spatial MI of subspace g (sec. 3.4, Eq. MI);
//   g = G       the AEB statistic of sbar: normalised entropy H^ (sec. 3.6),
//               or one minus the normalised peak mass in the confidence
//               variant;
//   G + 1 + j   stability phi_g with the stability-mean update (sec. 3.5) of
//               subspaces 8j .. 8j + 7.
// The grid is one-dimensional with every layer's MI blocks first (layer-
// major), then the lighter blocks: consecutive workgroups go to different
// CUs, so when the blocks outnumber the CUs each CU gets nearly the same
// number of MI blocks.
// The last block of each layer to finish then runs the layer's finalize in
// one wave: MI EMA, min-max prior w, lambda schedule, temperature T, state
// bookkeeping.
//
// Equal-frequency binning ranks the visual tokens of a subspace by (value,
// token index).  The bin edges are the K-1 order statistics at ranks
// ceil(b N / K), found together by one MSB-first radix select over
// order-preserving 32-bit keys: the bits every key shares are skipped and
// the first digit is 12 bits wide (one LDS histogram, block-wide scan).
// The keys are cached in LDS up to the shape's key cache (20K keys, 6K in
// the narrow shape, 2K in the small one); beyond that every pass reads S,
// walking the visual tokens as one index space with a span cursor.
// Fused path (the edges' first-digit buckets hold at most half the
// candidate area, or half the key cache when the keys are not cached and
// the key cache holds candidates):
// the joint histogram pass bins every key outside those buckets (its bin is
// the number of edges in lower buckets) and keeps the others with their cell
// and token index; up to 256 of them rank themselves directly, more are
// finished by 8-bit digits (one histogram per distinct edge prefix, one wave
// per edge); then each kept key is binned, equal keys at an edge split by
// token index.  Otherwise the keys in those buckets are compacted for the
// later digits, and the joint histogram pass bins every key by comparison.
// Equal keys at an edge split by token index: with cached keys through an
// ordered block scan of all keys; with uncached keys at a split point found
// from per-chunk counts of the equal keys and an ordered scan of one chunk,
// so that the binning pass itself reads in any order with loads in flight.
// Either way ties resolve exactly as the ranking defines.
#include <algorithm>

#include "device_common.h"
#include "grid_cell.h"
#include "stats_shape.h"
#include "internal.h"
#include "select_body.h"

namespace starkv {
namespace {

struct SpanSet {
  int32_t n;
  int32_t start[STARKV_MAX_SPANS];
  int32_t rows[STARKV_MAX_SPANS];
  int32_t cols[STARKV_MAX_SPANS];
  int32_t frame[STARKV_MAX_SPANS];
  int32_t off[STARKV_MAX_SPANS + 1];   // visual tokens before span i
};

struct FinalArgs {
  float* scal;
  char* state;
  size_t state_stride;
  int G, sc, nf;      // nf = current frame tokens, or -1
  float rho_mi, tau, eps, lam, t_min, t_max;
  int n_warmup, n_ramp;
};

struct StatsArgs {
  const float* S;
  const float* sbar;
  float* scal;
  char* state;
  size_t state_stride;
  size_t m_off;
  int G, Lp, nbins, grid, cur, frame_cap, sc;
  int n_stab;             // stability blocks, kStabSubspaces subspaces each
  int n_layers;
  int aeb;                // starkv_aeb_mode
  float rho_t, eps;
  SpanSet sp;
  FinalArgs fin;          // the layer's finalize, run by its last block
};

constexpr int kBatch = 8;                 // loads in flight per thread
constexpr int kKeyBatch = 8;              // keys per thread per rank-binning step
constexpr int kLoadBatch = 16;            // loads in flight in the first pass over S
constexpr int kDirect = 256;              // candidates ranked directly, no more digits
constexpr int kTieChunks = 256;           // visual-index chunks for locating tie splits
constexpr int kFirstDigitBins = 4096;     // the 12-bit first digit

// Three block shapes.  The wide one (1024 threads, 152 KiB of LDS) fills a
// CU and serves calls whose blocks fit on the GPU at once; the narrow one
// (512 threads, 61 KiB) runs two blocks per CU for calls with more blocks
// than CUs (a subspace per head), and needs n_bins <= kNarrowMaxBins; the
// small one (256 threads, 29 KiB, at most 128 VGPRs) runs four per CU for
// calls with more blocks than two per CU, and needs n_bins <= kSmallMaxBins
// and grid^2 <= kSmallMaxCells.
//   kHistInts  digit or joint histograms
//   kKeyCache  visual keys kept in LDS
//   kCand      keys in the edges' first-digit buckets
//   kJointOff  joint histogram slot when digits follow
//   kMaxTies   tied edges whose split counts live in the key cache
template <int NT>
struct StatsShape;
template <>
struct StatsShape<1024> {
  static constexpr int kHistInts = 16384, kKeyCache = 20 * 1024, kCand = 2048,
                       kJointOff = 8192, kMaxTies = 63;
};
template <>
struct StatsShape<512> {
  static constexpr int kHistInts = 4096 + kNarrowMaxBins * 256, kKeyCache = 6 * 1024,
                       kCand = 1024, kJointOff = 4096, kMaxTies = kNarrowMaxBins - 1;
};
template <>
struct StatsShape<256> {
  static constexpr int kHistInts = 4096 + kSmallMaxBins * kSmallMaxCells, kKeyCache = 2048,
                       kCand = 512, kJointOff = 4096, kMaxTies = kSmallMaxBins - 1;
};
// The fused selection's key cache follows its fixed LDS in the wide shape's
// dynamic LDS.
constexpr size_t kSelKeysOff = (sizeof(SelShared) + 15) / 16 * 16;

template <int NT>
constexpr size_t stats_lds() {
  using C = StatsShape<NT>;
  return (size_t)C::kHistInts * 4 + (size_t)C::kKeyCache * 4 + (size_t)C::kCand * 4;
}
static_assert(StatsShape<1024>::kMaxTies * kTieChunks <= StatsShape<1024>::kKeyCache,
              "tie-split counts live in the key cache");
static_assert(StatsShape<512>::kMaxTies * kTieChunks <= StatsShape<512>::kKeyCache,
              "tie-split counts live in the key cache");
static_assert(StatsShape<256>::kMaxTies * kTieChunks <= StatsShape<256>::kKeyCache,
              "tie-split counts live in the key cache");
static_assert(kDirect <= 256 && StatsShape<256>::kJointOff >= (kSmallMaxBins - 1) * 256 &&
                  StatsShape<256>::kJointOff >= kFirstDigitBins,
              "direct ranking has a thread per candidate; the digits fit below the joint "
              "histogram");
static_assert(stats_lds<1024>() >= kSelKeysOff + 4096 * sizeof(uint32_t),
              "the fused selection's fixed LDS and a key cache fit the wide shape's LDS");
static_assert(StatsShape<512>::kJointOff >= (kNarrowMaxBins - 1) * 256 &&
                  StatsShape<512>::kJointOff >= kFirstDigitBins,
              "later digits and the first digit fit below the joint histogram");


// Sum over the wave's lanes (integers: exact in any order).
__device__ inline int wave_sum_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Layer and block-of-layer of this workgroup (the grid order above).
__device__ __forceinline__ void stats_block(const StatsArgs& a, int* layer, int* g) {
  const int id = blockIdx.x;
  const int n_mi = a.G * a.n_layers;
  if (id < n_mi) {
    *layer = id / a.G;
    *g = id - *layer * a.G;
  } else {
    const int per = 1 + a.n_stab, k = id - n_mi;
    *layer = k / per;
    *g = a.G + (k - *layer * per);
  }
}

template <int NT>
__device__ __forceinline__ void stats_body(const StatsArgs& a, int layer, int g) {
  constexpr int kThreads = NT, kWaves = NT / 64;
  constexpr int kHistInts = StatsShape<NT>::kHistInts, kKeyCache = StatsShape<NT>::kKeyCache,
                kCand = StatsShape<NT>::kCand, kJointOff = StatsShape<NT>::kJointOff;
  constexpr int kScanBins = kFirstDigitBins / NT;   // first-digit bins per thread
  extern __shared__ __align__(16) unsigned char smem[];
  int* hist = reinterpret_cast<int*>(smem);
  uint32_t* kc = reinterpret_cast<uint32_t*>(smem + (size_t)kHistInts * 4);
  uint32_t* cand = kc + kKeyCache;
  __shared__ uint32_t t_key[64];          // edge key of target b
  __shared__ int t_rank[64];              // rank among keys sharing the prefix
  __shared__ int t_eq[64];                // keys equal to the edge key
  __shared__ int t_u[64];                 // histogram slot of the target
  __shared__ uint32_t n_key[64];          // first-digit results
  __shared__ int n_rank[64], n_eq[64];
  __shared__ uint32_t u_hi[64];
  __shared__ int n_u, cand_total;
  __shared__ uint32_t bucket_bits[128];   // first-digit buckets holding an edge
  __shared__ uint32_t seg_dg[64];         // distinct edge buckets, ascending
  __shared__ int seg_off[64], seg_cnt[64], seg_cur[64];
  __shared__ int n_seg;
  __shared__ int sp_start[STARKV_MAX_SPANS], sp_rows[STARKV_MAX_SPANS];
  __shared__ int sp_cols[STARKV_MAX_SPANS], sp_off[STARKV_MAX_SPANS + 1];
  __shared__ int nb_s[64];
  __shared__ int nc_s[256];
  __shared__ int sh_cnt[kWaves];
  __shared__ int carry_s[64];
  __shared__ uint32_t red_lo[kWaves], red_hi[kWaves];
  __shared__ double red[kWaves];
  __shared__ double red12[kWaves][12];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  float* scal = a.scal + (size_t)layer * a.sc;

  if (g == a.G) {   // ------------------------------------ entropy block
    const float* sb = a.sbar + (size_t)layer * a.Lp;
    double z = 0.0;
    float vmax = 0.f;     // s-bar is non-negative
    for (int t0 = tid; t0 < a.Lp; t0 += kBatch * kThreads) {
      float v[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {   // kBatch loads in flight
        const int t = t0 + u * kThreads;
        v[u] = t < a.Lp ? sb[t] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        z += (double)v[u];
        vmax = fmaxf(vmax, v[u]);
      }
    }
    z = block_sum_d(z, red);
    const double denom = z + (double)a.eps;
    if (a.aeb == STARKV_AEB_CONFIDENCE) {   // peak-mass variant: u = 1 - c
      vmax = wave_max(vmax);
      __shared__ float red_max[kWaves];
      if (lane == 0) red_max[wave] = vmax;
      __syncthreads();
      if (tid == 0) {
        float m = 0.f;
        for (int w = 0; w < kWaves; ++w) m = fmaxf(m, red_max[w]);
        double c = 1.0;
        if (a.Lp > 1) {
          const double inv = 1.0 / (double)a.Lp;
          c = fmin(1.0, fmax(0.0, ((double)m / denom - inv) / (1.0 - inv)));
        }
        scal[STARKV_SCAL_HHAT(a.G)] = (float)(1.0 - c);
      }
      return;
    }
    double e = 0.0;
    for (int t0 = tid; t0 < a.Lp; t0 += kBatch * kThreads) {
      float v[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int t = t0 + u * kThreads;
        v[u] = t < a.Lp ? sb[t] : -1.f;
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        if (v[u] >= 0.f) {
          const double p = (double)v[u] / denom;
          e += p * log(p + (double)a.eps);
        }
      }
    }
    e = block_sum_d(e, red);
    if (tid == 0) {
      double h = 0.0;
      if (a.Lp > 1) h = fmin(1.0, fmax(0.0, -e / log((double)a.Lp)));
      scal[STARKV_SCAL_HHAT(a.G)] = (float)h;
    }
    return;
  }

  if (g > a.G) {   // ------------------------------------ stability blocks
    const int g_lo = (g - a.G - 1) * kStabSubspaces;
    const int g_hi = min(g_lo + kStabSubspaces, a.G);
    if (a.cur < 0) {
      for (int j = g_lo + tid; j < g_hi; j += kThreads) scal[STARKV_SCAL_PHI(a.G) + j] = 0.f;
      return;
    }
    char* blk = a.state + (size_t)layer * a.state_stride;
    const StateHeader* hdr = reinterpret_cast<const StateHeader*>(blk);
    const int nf = a.sp.rows[a.cur] * a.sp.cols[a.cur];
    const bool reset = hdr->nf != nf;
    // up to four groups per pass: their 12 sums reduce together.  One pass
    // reads the old mean for the sums and writes the new one (element-wise,
    // each element by one thread), four iterations' loads in flight; a
    // thread's sums keep ascending token order.
    constexpr int kU = 4;
    for (int g0 = g_lo; g0 < g_hi; g0 += 4) {
      const int ng = min(4, g_hi - g0);
      double acc[12];
#pragma unroll
      for (int j = 0; j < 12; ++j) acc[j] = 0.0;
      const float* sg[4];
      float* mg[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int gg = g0 + min(j, ng - 1);
        sg[j] = a.S + (size_t)(layer * a.G + gg) * a.Lp + a.sp.start[a.cur];
        mg[j] = reinterpret_cast<float*>(blk + a.m_off) + (size_t)gg * a.frame_cap;
      }
      for (int i0 = tid; i0 < nf; i0 += kU * kThreads) {
        float sv[kU][4], mv[kU][4];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          const int i = i0 + u * kThreads;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const bool on = j < ng && i < nf;
            sv[u][j] = on ? sg[j][i] : 0.f;
            mv[u][j] = (on && !reset) ? mg[j][i] : 0.f;
          }
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          const int i = i0 + u * kThreads;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if (j < ng && i < nf) {
              const double sd = sv[u][j], md = mv[u][j];
              acc[3 * j] += sd * md;
              acc[3 * j + 1] += sd * sd;
              acc[3 * j + 2] += md * md;
              mg[j][i] = a.rho_t * mv[u][j] + (1.f - a.rho_t) * sv[u][j];
            }
          }
        }
      }
#pragma unroll
      for (int j = 0; j < 12; ++j) acc[j] = wave_sum_d(acc[j]);
      __syncthreads();
      if (lane == 0) {
#pragma unroll
        for (int j = 0; j < 12; ++j) red12[wave][j] = acc[j];
      }
      __syncthreads();
      if (tid < ng) {   // fixed summation order over the waves
        double dot = 0.0, ns = 0.0, nm = 0.0;
        for (int w = 0; w < kWaves; ++w) {
          dot += red12[w][3 * tid];
          ns += red12[w][3 * tid + 1];
          nm += red12[w][3 * tid + 2];
        }
        scal[STARKV_SCAL_PHI(a.G) + g0 + tid] =
            (float)(dot / (sqrt(ns) * sqrt(nm) + (double)a.eps));
      }
      __syncthreads();   // red12 is reused by the next four groups
    }
    return;
  }

  const float* Sg = a.S + (size_t)(layer * a.G + g) * a.Lp;
  const int N = a.sp.off[a.sp.n];
  const int K = a.nbins;
  const int M = a.grid;
  const int ncell = M * M;
  const bool cached = N <= kKeyCache;
  // Candidates (keys in the edges' first-digit buckets): the fused pass
  // keeps (key, cell << 24 | visual index) pairs, the compaction pass keys
  // only; in the candidate area while the keys are cached, else in the key
  // cache.
  uint32_t* ck = cached ? cand : kc;
  const int fcap = cached ? kCand / 2 : kKeyCache / 2;
  const int ccap = cached ? kCand : kKeyCache;
  uint32_t* cv = ck + fcap;
  // joint (bin, cell) histogram: at the start of hist, or past the digit
  // histograms when the fused pass fills it before the last digits
  int* jh = hist;
  double mi = 0.0;

  if (N > 0) {
    // span table to LDS, a span per wave (a wave-uniform index keeps the
    // argument in scalar loads)
    for (int s = __builtin_amdgcn_readfirstlane(wave); s < a.sp.n; s += kWaves) {
      if (lane == 0) {
        sp_off[s] = a.sp.off[s];
        sp_start[s] = a.sp.start[s];
        sp_rows[s] = a.sp.rows[s];
        sp_cols[s] = a.sp.cols[s];
      }
    }
    if (tid == 0) sp_off[a.sp.n] = N;
    __syncthreads();
    // Visual index i (ascending per thread) -> its span, by a cursor s.
    auto span_of = [&](int s, int i) {
      while (sp_off[s + 1] <= i) ++s;
      return s;
    };
    // Token positions of a thread's visual indices (ascending): the span
    // cursor keeps the current span's end and its token - index offset.
    int f_s = 0, f_end = 0, f_base = 0;
    auto token_of = [&](int i) {
      if (i >= f_end) {
        f_s = span_of(f_s, i);
        f_end = sp_off[f_s + 1];
        f_base = sp_start[f_s] - sp_off[f_s];
      }
      return f_base + i;
    };
    auto fetch_reset = [&]() { f_s = 0; f_end = 0; };
    // The kKeyBatch keys i0 + u * kThreads of this thread (0 past N), read
    // from S with kKeyBatch loads in flight.
    auto fetch = [&](int i0, uint32_t (&kv)[kKeyBatch]) {
      float v[kKeyBatch];
#pragma unroll
      for (int u = 0; u < kKeyBatch; ++u) {
        const int i = i0 + u * kThreads;
        v[u] = i < N ? Sg[token_of(i)] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kKeyBatch; ++u) kv[u] = i0 + u * kThreads < N ? fkey(v[u]) : 0u;
    };
    // the same from the key cache, or from S when the keys are not cached
    auto keys = [&](int i0, uint32_t (&kv)[kKeyBatch]) {
      if (!cached) {
        fetch(i0, kv);
        return;
      }
#pragma unroll
      for (int u = 0; u < kKeyBatch; ++u) {
        const int i = i0 + u * kThreads;
        kv[u] = i < N ? kc[i] : 0u;
      }
    };
    // Grid cell of visual index i.  A pass visits a thread's indices in
    // steps of kThreads, so (row, col) step inside a span and are recomputed
    // from the index only when it enters another span.  There the position
    // in the span is below kThreads (the previous index lay before the
    // span), so the row and every per-span constant come from reciprocal
    // estimates with one exact correction step; only a first index deep
    // inside a span takes the integer division.
    int q_s = 0, q_r = 0, q_c = 0, q_end = 0, q_next = -1, q_rows = 1, q_cols = 1,
        q_dq = 0, q_dr = 0;
    float q_fr = 0.f, q_fc = 0.f;
    auto cell_at = [&](int i) {
      if (i != q_next || i >= q_end) {
        q_s = span_of(q_s, i);
        q_rows = sp_rows[q_s];
        q_cols = sp_cols[q_s];
        q_end = sp_off[q_s + 1];
        const float rc = __builtin_amdgcn_rcpf((float)q_cols);
        const int p = i - sp_off[q_s];
        if (p < kSmallQuot) {
          q_r = small_quot(p, q_cols, rc);
          q_c = p - q_r * q_cols;
        } else {
          span_row_col(p, q_cols, &q_r, &q_c);
        }
        q_dq = small_quot(kThreads, q_cols, rc);
        q_dr = kThreads - q_dq * q_cols;
        // estimates of M / rows and M / cols: grid_cell corrects them
        q_fr = (float)M * __builtin_amdgcn_rcpf((float)q_rows);
        q_fc = (float)M * rc;
      } else {
        q_c += q_dr;
        q_r += q_dq;
        if (q_c >= q_cols) { q_c -= q_cols; ++q_r; }
      }
      q_next = i + kThreads;
      return grid_cell(q_r, q_c, q_rows, q_cols, M, q_fr, q_fc);
    };
    auto cell_reset = [&]() { q_s = 0; q_next = -1; };

    // ---- visual keys (LDS when they fit), min and max
    // (the first read of S: kLoadBatch loads in flight, so the five-frame
    // sizes take one round trip)
    uint32_t lo = 0xFFFFFFFFu, hi = 0u;
    {
      fetch_reset();
      for (int i0 = tid; i0 < N; i0 += kLoadBatch * kThreads) {
        float v[kLoadBatch];
#pragma unroll
        for (int u = 0; u < kLoadBatch; ++u) {
          const int i = i0 + u * kThreads;
          v[u] = i < N ? Sg[token_of(i)] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kLoadBatch; ++u) {
          const int i = i0 + u * kThreads;
          if (i < N) {
            const uint32_t key = fkey(v[u]);
            if (cached) kc[i] = key;
            lo = min(lo, key);
            hi = max(hi, key);
          }
        }
      }
    }
    lo = wave_min_u32(lo);
    hi = wave_max_u32(hi);
    if (lane == 0) { red_lo[wave] = lo; red_hi[wave] = hi; }
    // ---- edges: ranks ceil(b N / K), b = 1..K-1, that exist (rank < N)
    int n_t = 0;
    for (int b = 1; b < K; ++b)
      if (((int64_t)b * N + K - 1) / K < N) n_t = b;
    __syncthreads();
    uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
    for (int w = 0; w < kWaves; ++w) { kmin = min(kmin, red_lo[w]); kmax = max(kmax, red_hi[w]); }
    const int common = (kmin == kmax) ? 32 : __clz(kmin ^ kmax);
    const uint32_t cmask = common == 0 ? 0u : (common >= 32 ? 0xFFFFFFFFu : (0xFFFFFFFFu << (32 - common)));
    if (tid < n_t) {
      t_key[tid] = kmin & cmask;
      t_rank[tid] = (int)(((int64_t)(tid + 1) * N + K - 1) / K);
      t_eq[tid] = N;
    }
    __syncthreads();
    // ---- multi-target radix select: a 12-bit first digit (one histogram,
    // every target shares the common prefix), then 8-bit digits with one
    // histogram per distinct prefix.  After the first digit the keys in the
    // edges' buckets are kept in LDS when they fit, and the later digits scan
    // only those: the fused pass keeps them while it bins every other key
    // into the joint histogram; otherwise a compaction pass keeps their keys.
    bool first = true, compact = false, fused = false;
    int n_c = 0, f_shift = 0, f_nb = 1;
    // first-digit buckets of the edges (valid once the first digit is known)
    uint32_t eb[8];
    auto lower_edges = [&](uint32_t d) {
      int n = 0;
      if (n_t <= 8) {
#pragma unroll
        for (int j = 0; j < 8; ++j) n += eb[j] < d;
      } else {
        for (int b = 0; b < n_t; ++b) n += ((t_key[b] >> f_shift) & (uint32_t)(f_nb - 1)) < d;
      }
      return n;
    };
    // Few candidates, in one segment per edge bucket: each ranks itself
    // among its bucket's keys; the one whose rank range holds an edge's rank
    // is that edge's key.  Leaves the exact edges in t_*.
    auto direct_rank = [&](int shift) {
      const int ns = n_seg;
      if (tid < n_c) {
        const uint32_t key = ck[tid];
        const uint32_t pre = key_hi(key, shift);
        int sg = 0;
        while (sg + 1 < ns && seg_off[sg + 1] <= tid) ++sg;
        const int j_end = seg_off[sg] + seg_cnt[sg];
        int less = 0, eq = 0;
        for (int j0 = seg_off[sg]; j0 < j_end; j0 += 4) {
          uint32_t kv[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) kv[u] = ck[min(j0 + u, j_end - 1)];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const bool in = j0 + u < j_end;
            less += in && kv[u] < key;
            eq += in && kv[u] == key;
          }
        }
        for (int b = 0; b < n_t; ++b) {
          const int r = t_rank[b];
          if (key_hi(t_key[b], shift) == pre && less <= r && r < less + eq) {
            n_key[b] = key;      // equal keys write equal values
            n_rank[b] = r - less;
            n_eq[b] = eq;
          }
        }
      }
      __syncthreads();
      if (tid < n_t) {
        t_key[tid] = n_key[tid];
        t_rank[tid] = n_rank[tid];
        t_eq[tid] = n_eq[tid];
      }
      __syncthreads();
    };
    // segment of candidate slot j (segments are contiguous and ascending)
    auto seg_of = [&](int j) {
      int lo_s = 0, hi_s = n_seg - 1;
      while (lo_s < hi_s) {
        const int mid = (lo_s + hi_s + 1) >> 1;
        if (seg_off[mid] <= j) lo_s = mid; else hi_s = mid - 1;
      }
      return lo_s;
    };
    // segment of first-digit bucket d, which holds an edge
    auto seg_of_bucket = [&](uint32_t d) {
      int lo_s = 0, hi_s = n_seg - 1;
      while (lo_s < hi_s) {
        const int mid = (lo_s + hi_s) >> 1;
        if (seg_dg[mid] < d) lo_s = mid + 1; else hi_s = mid;
      }
      return lo_s;
    };
    for (int done = common; done < 32;) {
      const int width = min(first ? 12 : 8, 32 - done);
      const int shift = 32 - done - width;
      const int nb = 1 << width;
      if (wave == 0) {
        // targets ascend, so equal prefixes are adjacent: slot ids are a scan
        // of "prefix differs from the previous target's"
        const bool on = lane < n_t;
        const uint32_t h = on ? key_hi(t_key[lane], shift + width) : 0u;
        const uint32_t hp = (uint32_t)__shfl_up((int)h, 1);
        const bool fresh = on && (lane == 0 || hp != h);
        const int inc = wave_incl_scan(fresh ? 1 : 0);
        if (on) t_u[lane] = inc - 1;
        if (fresh) u_hi[inc - 1] = h;
        if (lane == 63) n_u = inc;
      }
      __syncthreads();
      const int nu = n_u;
      for (int i = tid; i < nu * nb; i += kThreads) hist[i] = 0;
      __syncthreads();
      auto count = [&](uint32_t key) {
        const uint32_t h = key_hi(key, shift + width);
        int u = 0;
        while (u < nu && u_hi[u] != h) ++u;
        if (u < nu) atomicAdd(&hist[u * nb + ((key >> shift) & (nb - 1))], 1);
      };
      if (first) {
        // every key shares the prefix: one histogram
        fetch_reset();
        for (int i0 = tid; i0 < N; i0 += kKeyBatch * kThreads) {
          uint32_t kv[kKeyBatch];
          keys(i0, kv);
#pragma unroll
          for (int u = 0; u < kKeyBatch; ++u)
            if (i0 + u * kThreads < N) atomicAdd(&hist[(kv[u] >> shift) & (nb - 1)], 1);
        }
      } else if (compact) {
        for (int i = tid; i < n_c; i += kThreads) count(ck[i]);
      } else {
        fetch_reset();
        for (int i0 = tid; i0 < N; i0 += kKeyBatch * kThreads) {
          uint32_t kv[kKeyBatch];
          keys(i0, kv);
#pragma unroll
          for (int u = 0; u < kKeyBatch; ++u)
            if (i0 + u * kThreads < N) count(kv[u]);
        }
      }
      __syncthreads();
      if (first) {
        // block-wide scan over the single histogram: a thread owns
        // kScanBins bins
        int c[kScanBins], sum = 0;
#pragma unroll
        for (int j = 0; j < kScanBins; ++j) {
          c[j] = (kScanBins * tid + j < nb) ? hist[kScanBins * tid + j] : 0;
          sum += c[j];
        }
        int tot;
        const int exc = block_excl_scan(sum, sh_cnt, &tot);
        // results go to separate arrays: every thread must read the old
        // ranks before any is replaced
        for (int b = 0; b < n_t; ++b) {
          const int r = t_rank[b];
          if (exc <= r && r < exc + sum) {
            int run = exc;
            for (int j = 0; j < kScanBins; ++j) {
              if (r < run + c[j]) {
                n_key[b] = t_key[b] | ((uint32_t)(kScanBins * tid + j) << shift);
                n_rank[b] = r - run;
                n_eq[b] = c[j];
                break;
              }
              run += c[j];
            }
          }
        }
        if (tid < 128) bucket_bits[tid] = 0u;
        __syncthreads();
        if (tid < n_t) {
          t_key[tid] = n_key[tid];
          t_rank[tid] = n_rank[tid];
          t_eq[tid] = n_eq[tid];
          const uint32_t dg = (n_key[tid] >> shift) & (uint32_t)(nb - 1);
          atomicOr(&bucket_bits[dg >> 5], 1u << (dg & 31));
        }
        if (wave == 0) {   // keys in the edges' buckets: one segment per bucket
          const bool on = lane < n_t;
          const uint32_t dg = on ? ((n_key[lane] >> shift) & (uint32_t)(nb - 1)) : 0u;
          const uint32_t dp = (uint32_t)__shfl_up((int)dg, 1);
          const bool fresh = on && (lane == 0 || dp != dg);
          const int cnt = fresh ? n_eq[lane] : 0;
          const int inc = wave_incl_scan(cnt);
          const int slot = wave_incl_scan(fresh ? 1 : 0) - 1;
          if (fresh) {
            seg_dg[slot] = dg;
            seg_off[slot] = inc - cnt;
            seg_cnt[slot] = cnt;
            seg_cur[slot] = 0;
          }
          if (lane == 63) { cand_total = inc; n_seg = slot + 1; }
        }
        __syncthreads();
        if (cand_total <= fcap && (K - 1) * 256 <= kJointOff &&
            kJointOff + K * ncell <= kHistInts && N < (1 << 24)) {
          // ---- fused pass: every key outside the edges' buckets goes to
          // the joint histogram (its bin is the number of edges in lower
          // buckets); the others are kept with their cell and visual index
          fused = true;
          f_shift = shift;
          f_nb = nb;
          jh = hist + kJointOff;
          for (int i = tid; i < K * ncell; i += kThreads) jh[i] = 0;
#pragma unroll
          for (int j = 0; j < 8; ++j)
            eb[j] = j < n_t ? ((t_key[j] >> shift) & (uint32_t)(nb - 1)) : 0xFFFFFFFFu;
          // per first-digit bucket, in the digit histogram's place (read
          // by the scan above, not needed again before the next digit): the
          // number of edges in lower buckets, i.e. the bin of a key outside
          // the edges' buckets, with bit 8 set for an edge's own bucket
          // (bins < 64)
          int* const d_lut = hist;
          for (int dd = tid; dd < nb; dd += kThreads)
            d_lut[dd] = lower_edges((uint32_t)dd) |
                        (int)(((bucket_bits[dd >> 5] >> (dd & 31)) & 1u) << 8);
          __syncthreads();
          fetch_reset();
          auto fuse_key_in = [&](int i, uint32_t key, int cell) {
            const uint32_t d = (key >> shift) & (uint32_t)(nb - 1);
            const int lut = d_lut[d];
            if (lut & 0x100) {
              const int sg = seg_of_bucket(d);
              const int pos = seg_off[sg] + atomicAdd(&seg_cur[sg], 1);
              ck[pos] = key;
              cv[pos] = ((uint32_t)cell << 24) | (uint32_t)i;
            } else {
              atomicAdd(&jh[lut * ncell + cell], 1);
            }
          };
          cell_reset();
          if (cached) {
            // keys in LDS: span by span, so that the span's constants are
            // uniform and a thread's (row, col) only steps inside the span
            for (int sp = 0; sp < a.sp.n; ++sp) {
              const int end = a.sp.off[sp + 1];
              const int rows = a.sp.rows[sp], cols = a.sp.cols[sp];
              const float rc = __builtin_amdgcn_rcpf((float)cols);
              const float fr = (float)M * __builtin_amdgcn_rcpf((float)rows), fc = (float)M * rc;
              const int dq = small_quot(kThreads, cols, rc), dr = kThreads - dq * cols;
              int r = small_quot(tid, cols, rc);
              int c = tid - r * cols;
#pragma unroll 2
              for (int i = a.sp.off[sp] + tid; i < end; i += kThreads) {
                fuse_key_in(i, kc[i], grid_cell(r, c, rows, cols, M, fr, fc));
                c += dr;
                r += dq;
                if (c >= cols) { c -= cols; ++r; }
              }
            }
          } else {        // kKeyBatch loads in flight
            fetch_reset();
            for (int i0 = tid; i0 < N; i0 += kKeyBatch * kThreads) {
              uint32_t kv[kKeyBatch];
              fetch(i0, kv);
#pragma unroll
              for (int u = 0; u < kKeyBatch; ++u) {
                const int i = i0 + u * kThreads;
                if (i < N) fuse_key_in(i, kv[u], cell_at(i));
              }
            }
          }
          __syncthreads();
          compact = true;
          n_c = cand_total;
          if (n_c <= kDirect) {
            direct_rank(shift);
            done = 32 - width;   // every edge is exact: no more digits
          }
        } else if (done + width < 32 && cand_total <= ccap) {
          // compaction: each bucket's keys in its own segment (in any order
          // inside it)
          fetch_reset();
          for (int i0 = tid; i0 < N; i0 += kKeyBatch * kThreads) {
            uint32_t kv[kKeyBatch];
            keys(i0, kv);
#pragma unroll
            for (int u = 0; u < kKeyBatch; ++u) {
              const uint32_t dg = (kv[u] >> shift) & (uint32_t)(nb - 1);
              if (i0 + u * kThreads < N && ((bucket_bits[dg >> 5] >> (dg & 31)) & 1u)) {
                const int sg = seg_of_bucket(dg);
                ck[seg_off[sg] + atomicAdd(&seg_cur[sg], 1)] = kv[u];
              }
            }
          }
          __syncthreads();
          compact = true;
          n_c = cand_total;
          if (n_c <= kDirect) {
            direct_rank(shift);
            done = 32 - width;   // every edge is exact: no more digits
          }
        }
      } else {
        for (int b = wave; b < n_t; b += kWaves) {
          int d, before, cnt;
          wave_find_bin(hist + t_u[b] * nb, nb, t_rank[b], &d, &before, &cnt);
          if (lane == 0) {
            t_key[b] |= (uint32_t)d << shift;
            t_rank[b] -= before;
            t_eq[b] = cnt;
          }
        }
      }
      __syncthreads();
      done += width;
      first = false;
    }

    if (fused) {
      // ---- the kept tokens, now that the edges are exact: a key above an
      // edge of its bucket is past it; equal keys at an edge split by
      // visual index (the ranking's tie rule)
      for (int j = tid; j < n_c; j += kThreads) {
        const uint32_t key = ck[j];
        const uint32_t v = cv[j] & 0xFFFFFFu;
        const int cell = (int)(cv[j] >> 24);
        const uint32_t d = (key >> f_shift) & (uint32_t)(f_nb - 1);
        const int sg = seg_of(j);
        const int j0 = seg_off[sg], j_end = j0 + seg_cnt[sg];
        int bin = lower_edges(d);
        for (int b = 0; b < n_t; ++b) {
          const uint32_t tkb = t_key[b];
          if (((tkb >> f_shift) & (uint32_t)(f_nb - 1)) != d) continue;
          if (key > tkb) {
            ++bin;
          } else if (key == tkb) {
            if (t_eq[b] == 1) {
              ++bin;       // the edge's own token, the only one with its key
            } else {
              int pos = 0;   // equal keys before this token in visual order
              for (int jj = j0; jj < j_end; ++jj) pos += ck[jj] == key && (cv[jj] & 0xFFFFFFu) < v;
              bin += pos >= t_rank[b];
            }
          }
        }
        atomicAdd(&jh[bin * ncell + cell], 1);
      }
      __syncthreads();
    } else if (!cached) {
      // ---- joint histogram of (bin, cell), keys read from S with kKeyBatch
      // loads in flight, in any order.  Equal keys at a tied edge split by
      // visual index (the ranking's tie rule): the split point t_vis comes
      // from per-chunk counts of the equal keys (any order) and an ordered
      // scan of the one chunk that holds the split.
      for (int i = tid; i < K * ncell; i += kThreads) hist[i] = 0;
      bool any_tie = false;
      for (int b = 0; b < n_t; ++b) any_tie |= (t_eq[b] > 1);
      // LDS arrays free in this branch (static LDS is at its limit):
      // t_vis[b], the first visual index above tied edge b, in the cached
      // branch's carries; the chunk and residual rank of a split in the
      // first digit's results
      int* const t_vis = carry_s;
      int& tie_c = n_rank[0];
      int& tie_r = n_rank[1];
      if (any_tie) {
        const int chunk =
            ((N + kTieChunks - 1) / kTieChunks + kThreads - 1) / kThreads * kThreads;
        int* tc = reinterpret_cast<int*>(kc);   // the key cache holds no keys here
        for (int i = tid; i < n_t * kTieChunks; i += kThreads) tc[i] = 0;
        __syncthreads();
        fetch_reset();
        for (int i0 = tid; i0 < N; i0 += kKeyBatch * kThreads) {
          uint32_t kv[kKeyBatch];
          fetch(i0, kv);
#pragma unroll
          for (int u = 0; u < kKeyBatch; ++u) {
            const int i = i0 + u * kThreads;
            if (i < N)
              for (int b = 0; b < n_t; ++b)
                if (t_eq[b] > 1 && kv[u] == t_key[b]) atomicAdd(&tc[b * kTieChunks + i / chunk], 1);
          }
        }
        __syncthreads();
        for (int b = 0; b < n_t; ++b) {
          if (t_eq[b] <= 1) continue;   // uniform
          if (wave == 0) {
            // the chunk holding the equal key at position t_rank[b]
            int c4[4], sum = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              c4[j] = tc[b * kTieChunks + 4 * lane + j];
              sum += c4[j];
            }
            const int inc = wave_incl_scan(sum);
            const int total = __shfl(inc, 63);
            const int r = t_rank[b];
            if (lane == 0) t_vis[b] = N;
            if (r >= total) {
              if (lane == 0) tie_c = -1;
            } else if (inc - sum <= r && r < inc) {
              int run = inc - sum;
              for (int j = 0; j < 4; ++j) {
                if (r < run + c4[j]) {
                  tie_c = 4 * lane + j;
                  tie_r = r - run;
                  break;
                }
                run += c4[j];
              }
            }
          }
          __syncthreads();
          const int c = tie_c, rr = tie_r;
          if (c >= 0) {
            fetch_reset();
            const int i_end = min(N, (c + 1) * chunk);
            int carry = 0;   // equal keys seen so far in the chunk (uniform)
            for (int i0 = c * chunk; i0 < i_end && carry <= rr; i0 += kThreads) {
              const int i = i0 + tid;
              const bool eq = i < i_end && fkey(Sg[token_of(i)]) == t_key[b];
              int tot;
              const int pos = block_excl_count(eq, sh_cnt, &tot) + carry;
              if (eq && pos == rr) t_vis[b] = i;
              carry += tot;
            }
          }
          __syncthreads();
        }
      }
      __syncthreads();   // the cleared histogram, the split points
      fetch_reset();
      cell_reset();
      for (int i0 = tid; i0 < N; i0 += kKeyBatch * kThreads) {
        uint32_t kv[kKeyBatch];
        fetch(i0, kv);
#pragma unroll
        for (int u = 0; u < kKeyBatch; ++u) {
          const int i = i0 + u * kThreads;
          if (i < N) {
            const uint32_t key = kv[u];
            int bin = 0;
            for (int b = 0; b < n_t; ++b) {
              const uint32_t tkb = t_key[b];
              bin += key > tkb || (key == tkb && (t_eq[b] == 1 || i >= t_vis[b]));
            }
            atomicAdd(&hist[bin * ncell + cell_at(i)], 1);
          }
        }
      }
      __syncthreads();
    } else {
      // ---- joint histogram of (bin, cell) from the cached keys in
      // visual-token order (the order the ranking's tie rule refers to):
      // block-wide batches of kThreads consecutive tokens
      for (int i = tid; i < K * ncell; i += kThreads) hist[i] = 0;
      bool any_tie = false;
      for (int b = 0; b < n_t; ++b) any_tie |= (t_eq[b] > 1);
      if (tid < 64) carry_s[tid] = 0;
      uint32_t tk[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) tk[j] = j < n_t ? t_key[j] : 0u;
      __syncthreads();
      cell_reset();
#pragma unroll 1
      for (int i0 = 0; i0 < N; i0 += kThreads) {
        {
          const int i = i0 + tid;
          const bool valid = i < N;
          const uint32_t key = valid ? kc[i] : 0u;
          int bin = 0;
          if (!any_tie) {
            if (n_t <= 8) {
#pragma unroll
              for (int j = 0; j < 8; ++j) bin += (j < n_t) & (key >= tk[j]);
            } else {
              for (int b = 0; b < n_t; ++b) bin += (key >= t_key[b]);
            }
          } else {
            for (int b = 0; b < n_t; ++b) {
              if (t_eq[b] > 1) {   // uniform branch: ordered split of equal keys
                const bool eq = valid && (key == t_key[b]);
                const int c0 = carry_s[b];
                int tot;
                const int pos = block_excl_count(eq, sh_cnt, &tot) + c0;
                bin += (key > t_key[b]) || (eq && pos >= t_rank[b]);
                __syncthreads();
                if (tid == 0) carry_s[b] = c0 + tot;
                __syncthreads();
              } else {
                bin += (key >= t_key[b]);
              }
            }
          }
          if (valid) atomicAdd(&hist[bin * ncell + cell_at(i)], 1);
        }
      }
      __syncthreads();
    }
    // ---- plug-in MI from the counts (fixed summation order; integer sums)
    for (int b = wave; b < K; b += kWaves) {   // bin totals: a wave per bin
      int sum = 0;
      for (int cc = lane; cc < ncell; cc += 64) sum += jh[b * ncell + cc];
      sum = wave_sum_i(sum);
      if (lane == 0) nb_s[b] = sum;
    }
    if (tid < ncell) {
      int sum = 0;
      for (int b = 0; b < K; ++b) sum += jh[b * ncell + tid];
      nc_s[tid] = sum;
    }
    __syncthreads();
    double part = 0.0;
    for (int i = tid; i < K * ncell; i += kThreads) {
      const int n = jh[i];
      if (n > 0) {
        const double nn = (double)n, NN = (double)N;
        part += (nn / NN) * log(nn * NN / ((double)nb_s[i / ncell] * (double)nc_s[i % ncell]));
      }
    }
    mi = block_sum_d(part, red);
  }
  if (tid == 0) scal[STARKV_SCAL_MI(a.G) + g] = (float)mi;
}


// One wave, one lane per group (G <= 64); wave reductions in a fixed order.
__device__ __forceinline__ void finalize_layer(const FinalArgs& a, int layer, int lane) {
  float* scal = a.scal + (size_t)layer * a.sc;
  char* blk = a.state + (size_t)layer * a.state_stride;
  StateHeader* hdr = reinterpret_cast<StateHeader*>(blk);
  float* mibar = reinterpret_cast<float*>(blk + sizeof(StateHeader));
  const int G = a.G;
  const bool on = lane < G;
  const int n_prev = hdr->n;
  const float h = scal[STARKV_SCAL_HHAT(G)];
  double v = 0.0;
  if (on) {
    v = (double)a.rho_mi * (double)mibar[lane] +
        (1.0 - (double)a.rho_mi) * (double)scal[STARKV_SCAL_MI(G) + lane];
    v = (double)(float)v;                 // the state keeps float32
  }
  double lo = on ? v : 1e300, hi = on ? v : -1e300;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    lo = fmin(lo, __shfl_xor(lo, o));
    hi = fmax(hi, __shfl_xor(hi, o));
  }
  const double z = on ? ((v - lo) / (hi - lo + (double)a.eps)) / (double)a.tau : -1e300;
  double zmax = z;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) zmax = fmax(zmax, __shfl_xor(zmax, o));
  const double ez = on ? exp(z - zmax) : 0.0;
  const double zs = wave_sum_d(ez);
  if (on) {
    mibar[lane] = (float)v;
    scal[STARKV_SCAL_MIBAR(G) + lane] = (float)v;
    scal[STARKV_SCAL_W(G) + lane] = (float)(ez / zs);
  }
  if (lane == 0) {
    const int n = n_prev + 1;
    double lam = 0.0;
    if (n > a.n_warmup) {
      lam = a.n_ramp <= 0 ? (double)a.lam
                          : (double)a.lam * fmin(1.0, (double)(n - a.n_warmup) / (double)a.n_ramp);
    }
    scal[STARKV_SCAL_LAMBDA(G)] = (float)lam;
    scal[STARKV_SCAL_T(G)] =
        (float)((double)a.t_min + ((double)a.t_max - (double)a.t_min) * (double)h);
    scal[STARKV_SCAL_N(G)] = (float)n;
    hdr->n = n;
    if (a.nf >= 0) hdr->nf = a.nf;
  }
}

// Every block of a layer counts itself in the layer's state header after
// its results are out; the last one to arrive runs the layer's finalize and
// clears the count.  No block waits for another.
// With SEL, the block that runs a layer's finalize then runs that layer's
// selection (select_body) in the same workgroup, its LDS carved from the
// statistics' dynamic LDS, which no longer holds anything live by then.
template <int NT, bool SEL>
__global__ __launch_bounds__(NT, 1024 / NT) void stats_kernel(StatsArgs a, SelArgs sel) {
  static_assert(!SEL || NT == kSelThreads, "the selection body needs a 1024-thread block");
  __shared__ int last_s;
  int layer, g;
  stats_block(a, &layer, &g);
  StateHeader* hdr = reinterpret_cast<StateHeader*>(a.state + (size_t)layer * a.state_stride);
  // A state block built for other dimensions (another subspace count or
  // frame capacity, or never initialised) is left untouched: the layer's
  // scalars become NaN and no block reads or writes its statistics.  The
  // checked fields are written only by starkv_state_init, so reading them
  // here races with nothing.  With SEL, block 0 then selects on the NaN
  // scalars, as a separate selection call would.
  if (hdr->magic != kStateMagic || hdr->G != a.G || hdr->frame_cap != a.frame_cap) {
    if (g != 0) return;
    for (int i = threadIdx.x; i < a.sc; i += NT)
      a.scal[(size_t)layer * a.sc + i] = __builtin_nanf("");
  } else {
    stats_body<NT>(a, layer, g);
    // Lanes of wave 0 wrote every value the finalize and a fused selection
    // read from this block (MI_g or H^ by thread 0, phi by the first four
    // lanes); thread 0's fence, in that wave, publishes them before it
    // counts the block.
    __syncthreads();
    if (threadIdx.x == 0) {
      __threadfence();
      last_s = atomicAdd(&hdr->arrive, 1) == a.G + a.n_stab;
    }
    __syncthreads();
    if (!last_s) return;
    if (threadIdx.x < 64) {
      __threadfence();          // the other blocks' values
      finalize_layer(a.fin, layer, threadIdx.x);
    }
    if (threadIdx.x == 0) hdr->arrive = 0;
  }
  if constexpr (SEL) {
    extern __shared__ __align__(16) unsigned char smem_sel[];
    __syncthreads();   // the layer's scalars are out; the LDS is free
    select_body(sel, layer, *reinterpret_cast<SelShared*>(smem_sel),
                reinterpret_cast<uint32_t*>(smem_sel + kSelKeysOff));
  }
}

__global__ __launch_bounds__(256) void state_init_kernel(char* state, size_t stride,
                                                         int G, int frame_cap) {
  char* blk = state + (size_t)blockIdx.x * stride;
  float* f = reinterpret_cast<float*>(blk);
  for (size_t i = threadIdx.x; i < stride / 4; i += blockDim.x) f[i] = 0.f;
  __syncthreads();
  if (threadIdx.x == 0) {
    StateHeader* h = reinterpret_cast<StateHeader*>(blk);
    h->magic = kStateMagic;
    h->G = G;
    h->frame_cap = frame_cap;
    h->n = 0;
    h->nf = 0;
  }
}

StatsArgs make_stats_args(const Geometry& g, const starkv_params& p, const float* S,
                          const float* sbar, const starkv_span* spans, int32_t n_spans,
                          int32_t frame, void* state, int32_t frame_cap, float* scalars) {
  StatsArgs a;
  a.S = S;
  a.sbar = sbar;
  a.scal = scalars;
  a.state = static_cast<char*>(state);
  // every per-group statistic here is per scoring subspace
  a.state_stride = state_stride(g.Ns, frame_cap);
  a.m_off = state_m_off(g.Ns);
  a.G = g.Ns;
  a.Lp = g.Lp;
  a.nbins = p.n_bins;
  a.grid = p.grid;
  a.cur = current_span(spans, n_spans, frame);
  a.frame_cap = frame_cap;
  a.sc = (int)scalars_count(g.Ns);
  a.n_stab = stats_stab_blocks(g.Ns);
  a.n_layers = g.n_layers;
  a.aeb = p.aeb_mode;
  a.rho_t = p.rho_t;
  a.eps = p.eps;
  a.sp.n = n_spans;
  a.sp.off[0] = 0;
  for (int i = 0; i < n_spans; ++i) {
    a.sp.start[i] = spans[i].start;
    a.sp.rows[i] = spans[i].rows;
    a.sp.cols[i] = spans[i].cols;
    a.sp.frame[i] = spans[i].frame;
    a.sp.off[i + 1] = a.sp.off[i] + spans[i].rows * spans[i].cols;
  }
  FinalArgs& f = a.fin;
  f.scal = scalars;
  f.state = a.state;
  f.state_stride = a.state_stride;
  f.G = g.Ns;
  f.sc = a.sc;
  f.nf = a.cur >= 0 ? spans[a.cur].rows * spans[a.cur].cols : -1;
  f.rho_mi = p.rho_mi;
  f.tau = p.tau;
  f.eps = p.eps;
  f.lam = p.lam;
  f.t_min = p.t_min;
  f.t_max = p.t_max;
  f.n_warmup = p.n_warmup;
  f.n_ramp = p.n_ramp;
  return a;
}

// The wide shape's dynamic LDS is above the default limit; raised once per
// process (function-local static initialisation is thread-safe).
void set_wide_lds_attributes() {
  static const hipError_t attr_plain = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&stats_kernel<1024, false>),
      hipFuncAttributeMaxDynamicSharedMemorySize, (int)stats_lds<1024>());
  static const hipError_t attr_sel = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&stats_kernel<1024, true>),
      hipFuncAttributeMaxDynamicSharedMemorySize, (int)stats_lds<1024>());
  (void)attr_plain;
  (void)attr_sel;
}

// The statistics block shape for this call (stats_shape.h); -1 when the
// device cannot be queried.
int stats_shape(const Geometry& g, const starkv_params& p) {
  int dev = 0, n_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      n_cu <= 0)
    return -1;
  return stats_shape_for((long)stats_layer_blocks(g.Ns) * g.n_layers, n_cu, p.n_bins, p.grid);
}

}  // namespace

int launch_update_state(const Geometry& g, const starkv_params& p,
                        const float* S, const float* sbar,
                        const starkv_span* spans, int32_t n_spans,
                        int32_t frame, void* state, int32_t frame_cap,
                        float* scalars, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const StatsArgs a = make_stats_args(g, p, S, sbar, spans, n_spans, frame, state, frame_cap,
                                      scalars);
  set_wide_lds_attributes();
  const int nt = stats_shape(g, p);
  if (nt < 0) return (int)hipErrorInvalidDevice;
  const dim3 grid(stats_layer_blocks(g.Ns) * g.n_layers);
  SelArgs none{};
  if (nt == 256)
    stats_kernel<256, false><<<grid, 256, stats_lds<256>(), st>>>(a, none);
  else if (nt == 512)
    stats_kernel<512, false><<<grid, 512, stats_lds<512>(), st>>>(a, none);
  else
    stats_kernel<1024, false><<<grid, 1024, stats_lds<1024>(), st>>>(a, none);
  return (int)hipGetLastError();
}

int launch_update_state_select(const Geometry& g, const starkv_params& p, const float* S,
                               const float* sbar, const uint8_t* gstar,
                               const starkv_span* spans, int32_t n_spans, int32_t frame,
                               void* state, int32_t frame_cap, float* scalars, int32_t B,
                               float* s, int32_t* idx, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int nt = stats_shape(g, p);
  if (nt < 0) return (int)hipErrorInvalidDevice;
  if (nt != 1024) {
    // the selection needs a 1024-thread block: two launches
    if (int err = launch_update_state(g, p, S, sbar, spans, n_spans, frame, state, frame_cap,
                                      scalars, stream))
      return err;
    return launch_select(g, p, sbar, gstar, scalars, spans, n_spans, frame, B, s, idx, stream);
  }
  const StatsArgs a = make_stats_args(g, p, S, sbar, spans, n_spans, frame, state, frame_cap,
                                      scalars);
  SelArgs sel;
  const long room = (long)((stats_lds<1024>() - kSelKeysOff) / sizeof(uint32_t));
  fill_sel_args(sel, g, p, sbar, gstar, scalars, spans, n_spans, frame, B, s, idx,
                (int)std::min<long>({(long)g.Lp, (long)kSelLdsKeys, room}));
  set_wide_lds_attributes();
  stats_kernel<1024, true><<<stats_layer_blocks(g.Ns) * g.n_layers, 1024, stats_lds<1024>(),
                             st>>>(a, sel);
  return (int)hipGetLastError();
}

int launch_state_init(const Geometry& g, void* state, int32_t frame_cap, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  state_init_kernel<<<g.n_layers, 256, 0, st>>>(static_cast<char*>(state),
                                                state_stride(g.Ns, frame_cap), g.Ns,
                                                frame_cap);
  return (int)hipGetLastError();
}

}  // namespace starkv
