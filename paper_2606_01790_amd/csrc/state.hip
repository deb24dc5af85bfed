// Online statistics of one step (sec. 3.4-3.6).
//
// stats kernel, grid (G + 1, n_layers), 1024 threads:
//   block g < G   spatial MI of group g (sec. 3.4, Eq. MI) and its stability
//                 phi_g with the stability-mean update (sec. 3.5);
//   block G       normalised entropy H^ of sbar (sec. 3.6).
// finalize kernel, one wave per layer: MI EMA, min-max prior w, lambda
// schedule, temperature T, state bookkeeping.
//
// Equal-frequency binning ranks the visual tokens of a group by (value,
// token index).  The bin edges are the K-1 order statistics at ranks
// ceil(b N / K), found by an MSB-first radix select over order-preserving
// 32-bit keys (8-bit digits, histograms in LDS).  A token's bin is the number
// of edges at or below it.  Equal keys at an edge are split by token index
// with an ordered block scan, so ties resolve exactly as the ranking defines.
#include "device_common.h"
#include "internal.h"

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

struct StatsArgs {
  const float* S;
  const float* sbar;
  float* scal;
  char* state;
  size_t state_stride;
  size_t m_off;
  int G, Lp, nbins, grid, cur, frame_cap, sc;
  float rho_t, eps;
  SpanSet sp;
};

constexpr int kThreads = 1024;

// visual index v (spans in token order) -> token, row, column, span
__device__ inline void visual_token(const SpanSet& sp, int v, int* t, int* r, int* c, int* s) {
  int lo = 0, hi = sp.n - 1;
  while (lo < hi) {           // last span with off <= v
    const int mid = (lo + hi + 1) >> 1;
    if (sp.off[mid] <= v) lo = mid; else hi = mid - 1;
  }
  const int i = v - sp.off[lo];
  *s = lo;
  *r = i / sp.cols[lo];
  *c = i % sp.cols[lo];
  *t = sp.start[lo] + i;
}

__global__ __launch_bounds__(kThreads) void stats_kernel(StatsArgs a) {
  __shared__ int hist[64 * 256];          // radix histograms, then joint counts
  __shared__ uint32_t t_key[64];          // edge key of target b
  __shared__ int t_rank[64];              // rank among equal keys
  __shared__ int t_eq[64];                // elements with that key
  __shared__ int t_u[64];                 // histogram slot of the target
  __shared__ uint32_t u_hi[64];
  __shared__ int n_u;
  __shared__ int nb_s[64];
  __shared__ int nc_s[256];
  __shared__ int sh_cnt[kThreads / 64];
  __shared__ int carry_s[64];
  __shared__ double red[kThreads / 64];

  const int layer = blockIdx.y, g = blockIdx.x;
  const int tid = threadIdx.x;
  float* scal = a.scal + (size_t)layer * a.sc;

  if (g == a.G) {   // ------------------------------------ entropy block
    const float* sb = a.sbar + (size_t)layer * a.Lp;
    double z = 0.0;
    for (int t = tid; t < a.Lp; t += kThreads) z += (double)sb[t];
    z = block_sum_d(z, red);
    const double denom = z + (double)a.eps;
    double e = 0.0;
    for (int t = tid; t < a.Lp; t += kThreads) {
      const double p = (double)sb[t] / denom;
      e += p * log(p + (double)a.eps);
    }
    e = block_sum_d(e, red);
    if (tid == 0) {
      double h = 0.0;
      if (a.Lp > 1) h = fmin(1.0, fmax(0.0, -e / log((double)a.Lp)));
      scal[STARKV_SCAL_HHAT(a.G)] = (float)h;
    }
    return;
  }

  const float* Sg = a.S + (size_t)(layer * a.G + g) * a.Lp;
  const int N = a.sp.off[a.sp.n];
  const int K = a.nbins;
  const int M = a.grid;
  double mi = 0.0;

  if (N > 0) {
    // ---- edges: ranks ceil(b N / K), b = 1..K-1, that exist (rank < N)
    int n_t = 0;
    for (int b = 1; b < K; ++b)
      if (((int64_t)b * N + K - 1) / K < N) n_t = b;
    if (tid < n_t) {
      t_key[tid] = 0u;
      t_rank[tid] = (int)(((int64_t)(tid + 1) * N + K - 1) / K);
    }
    __syncthreads();
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      if (tid == 0) {   // distinct fixed prefixes share one histogram
        int nu = 0;
        for (int b = 0; b < n_t; ++b) {
          const uint32_t hi = pass == 0 ? 0u : (t_key[b] >> (shift + 8));
          int u = 0;
          while (u < nu && u_hi[u] != hi) ++u;
          if (u == nu) u_hi[nu++] = hi;
          t_u[b] = u;
        }
        n_u = nu;
      }
      __syncthreads();
      const int nu = n_u;
      for (int i = tid; i < nu * 256; i += kThreads) hist[i] = 0;
      __syncthreads();
      for (int s = 0; s < a.sp.n; ++s) {
        const int n_s = a.sp.rows[s] * a.sp.cols[s];
        const float* src = Sg + a.sp.start[s];
        for (int i = tid; i < n_s; i += kThreads) {
          const uint32_t key = fkey(src[i]);
          const uint32_t hi = pass == 0 ? 0u : (key >> (shift + 8));
          int u = 0;
          while (u < nu && u_hi[u] != hi) ++u;
          if (u < nu) atomicAdd(&hist[u * 256 + ((key >> shift) & 255)], 1);
        }
      }
      __syncthreads();
      if (tid < n_t) {
        const int* h = hist + t_u[tid] * 256;
        int cum = 0, rank = t_rank[tid];
        for (int dg = 0; dg < 256; ++dg) {
          const int c = h[dg];
          if (cum + c > rank) {
            t_key[tid] |= (uint32_t)dg << shift;
            t_rank[tid] = rank - cum;
            t_eq[tid] = c;
            break;
          }
          cum += c;
        }
      }
      __syncthreads();
    }

    // ---- joint histogram of (bin, cell), visual tokens in index order
    const int ncell = M * M;
    for (int i = tid; i < K * ncell; i += kThreads) hist[i] = 0;
    bool any_tie = false;
    for (int b = 0; b < n_t; ++b) any_tie |= (t_eq[b] > 1);
    if (tid < 64) carry_s[tid] = 0;
    __syncthreads();
    for (int base = 0; base < N; base += kThreads) {
      const int v = base + tid;
      int t = 0, r = 0, c = 0, s = 0;
      uint32_t key = 0u;
      if (v < N) {
        visual_token(a.sp, v, &t, &r, &c, &s);
        key = fkey(Sg[t]);
      }
      int bin = 0;
      if (!any_tie) {
        for (int b = 0; b < n_t; ++b) bin += (key >= t_key[b]);
      } else {
        for (int b = 0; b < n_t; ++b) {
          if (t_eq[b] > 1) {   // uniform branch: ordered split of equal keys
            const bool eq = (v < N) && (key == t_key[b]);
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
      if (v < N) {
        const int cell = (r * M / a.sp.rows[s]) * M + (c * M / a.sp.cols[s]);
        atomicAdd(&hist[bin * ncell + cell], 1);
      }
    }
    __syncthreads();
    // ---- plug-in MI from the counts (fixed summation order)
    if (tid < K) {
      int sum = 0;
      for (int cc = 0; cc < ncell; ++cc) sum += hist[tid * ncell + cc];
      nb_s[tid] = sum;
    }
    if (tid < ncell) {
      int sum = 0;
      for (int b = 0; b < K; ++b) sum += hist[b * ncell + tid];
      nc_s[tid] = sum;
    }
    __syncthreads();
    double part = 0.0;
    for (int i = tid; i < K * ncell; i += kThreads) {
      const int n = hist[i];
      if (n > 0) {
        const double nn = (double)n, NN = (double)N;
        part += (nn / NN) * log(nn * NN / ((double)nb_s[i / ncell] * (double)nc_s[i % ncell]));
      }
    }
    mi = block_sum_d(part, red);
  }
  if (tid == 0) scal[STARKV_SCAL_MI(a.G) + g] = (float)mi;

  // ---- stability of the current frame's row (sec. 3.5)
  if (a.cur < 0) {
    if (tid == 0) scal[STARKV_SCAL_PHI(a.G) + g] = 0.f;
    return;
  }
  char* blk = a.state + (size_t)layer * a.state_stride;
  const StateHeader* hdr = reinterpret_cast<const StateHeader*>(blk);
  float* m = reinterpret_cast<float*>(blk + a.m_off) + (size_t)g * a.frame_cap;
  const int nf = a.sp.rows[a.cur] * a.sp.cols[a.cur];
  const bool reset = hdr->nf != nf;
  const float* scur = Sg + a.sp.start[a.cur];
  double dot = 0.0, ns = 0.0, nm = 0.0;
  for (int i = tid; i < nf; i += kThreads) {
    const double s = scur[i];
    const double mv = reset ? 0.0 : (double)m[i];
    dot += s * mv;
    ns += s * s;
    nm += mv * mv;
  }
  dot = block_sum_d(dot, red);
  ns = block_sum_d(ns, red);
  nm = block_sum_d(nm, red);
  const double phi = dot / (sqrt(ns) * sqrt(nm) + (double)a.eps);
  for (int i = tid; i < nf; i += kThreads) {
    const float mv = reset ? 0.f : m[i];
    m[i] = a.rho_t * mv + (1.f - a.rho_t) * scur[i];
  }
  if (tid == 0) scal[STARKV_SCAL_PHI(a.G) + g] = (float)phi;
}

struct FinalArgs {
  float* scal;
  char* state;
  size_t state_stride;
  int G, sc, nf;      // nf = current frame tokens, or -1
  float rho_mi, tau, eps, lam, t_min, t_max;
  int n_warmup, n_ramp;
};

__global__ __launch_bounds__(64) void finalize_kernel(FinalArgs a) {
  if (threadIdx.x != 0) return;
  const int layer = blockIdx.x;
  float* scal = a.scal + (size_t)layer * a.sc;
  char* blk = a.state + (size_t)layer * a.state_stride;
  StateHeader* hdr = reinterpret_cast<StateHeader*>(blk);
  float* mibar = reinterpret_cast<float*>(blk + sizeof(StateHeader));
  const int G = a.G;
  double lo = 0.0, hi = 0.0;
  for (int g = 0; g < G; ++g) {
    const double v = (double)a.rho_mi * (double)mibar[g] +
                     (1.0 - (double)a.rho_mi) * (double)scal[STARKV_SCAL_MI(G) + g];
    mibar[g] = (float)v;
    scal[STARKV_SCAL_MIBAR(G) + g] = (float)v;
    lo = g == 0 ? v : fmin(lo, v);
    hi = g == 0 ? v : fmax(hi, v);
  }
  double zmax = -1e300, zs = 0.0;
  for (int g = 0; g < G; ++g) {
    const double z = (((double)mibar[g] - lo) / (hi - lo + (double)a.eps)) / (double)a.tau;
    zmax = fmax(zmax, z);
  }
  for (int g = 0; g < G; ++g) {
    const double z = (((double)mibar[g] - lo) / (hi - lo + (double)a.eps)) / (double)a.tau;
    zs += exp(z - zmax);
  }
  for (int g = 0; g < G; ++g) {
    const double z = (((double)mibar[g] - lo) / (hi - lo + (double)a.eps)) / (double)a.tau;
    scal[STARKV_SCAL_W(G) + g] = (float)(exp(z - zmax) / zs);
  }
  const int n = hdr->n + 1;
  double lam = 0.0;
  if (n > a.n_warmup) {
    lam = a.n_ramp <= 0 ? (double)a.lam
                        : (double)a.lam * fmin(1.0, (double)(n - a.n_warmup) / (double)a.n_ramp);
  }
  scal[STARKV_SCAL_LAMBDA(G)] = (float)lam;
  const double h = scal[STARKV_SCAL_HHAT(G)];
  scal[STARKV_SCAL_T(G)] = (float)((double)a.t_min + ((double)a.t_max - (double)a.t_min) * h);
  scal[STARKV_SCAL_N(G)] = (float)n;
  hdr->n = n;
  if (a.nf >= 0) hdr->nf = a.nf;
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

}  // namespace

int launch_update_state(const Geometry& g, const starkv_params& p,
                        const float* S, const float* sbar,
                        const starkv_span* spans, int32_t n_spans,
                        int32_t frame, void* state, int32_t frame_cap,
                        float* scalars, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  StatsArgs a;
  a.S = S;
  a.sbar = sbar;
  a.scal = scalars;
  a.state = static_cast<char*>(state);
  a.state_stride = state_stride(g.G, frame_cap);
  a.m_off = state_m_off(g.G);
  a.G = g.G;
  a.Lp = g.Lp;
  a.nbins = p.n_bins;
  a.grid = p.grid;
  a.cur = current_span(spans, n_spans, frame);
  a.frame_cap = frame_cap;
  a.sc = (int)scalars_count(g.G);
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
  stats_kernel<<<dim3(g.G + 1, g.n_layers), kThreads, 0, st>>>(a);
  FinalArgs f;
  f.scal = scalars;
  f.state = a.state;
  f.state_stride = a.state_stride;
  f.G = g.G;
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
  finalize_kernel<<<g.n_layers, 64, 0, st>>>(f);
  return (int)hipGetLastError();
}

int launch_state_init(const Geometry& g, void* state, int32_t frame_cap, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  state_init_kernel<<<g.n_layers, 256, 0, st>>>(static_cast<char*>(state),
                                                state_stride(g.G, frame_cap), g.G,
                                                frame_cap);
  return (int)hipGetLastError();
}

}  // namespace starkv
