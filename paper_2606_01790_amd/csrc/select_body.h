// Final score and global top-B (Eq. final_score, sec. 3.2; sec. 3.5 discount;
// sec. 3.7 selection): the body one 1024-thread workgroup runs for one layer,
// shared by the selection kernel and the statistics kernel (which can run it
// for a layer right after that layer's finalize):
//   1. s_t = max(sbar_t * beta_t * D_t, 0)^(1/T) for every past token
//      (D_t with the configured decay: exponential, linear or gamma),
//      written out and kept as a descending-order key in LDS.  beta_t and
//      D_t depend on the token only through g*_t and its span, so both come
//      from tables filled once per block (per group; per group and span);
//      the span of a token comes from an LDS copy of the span table, walked
//      by a cursor since each thread's tokens ascend;
//   2. MSB-first radix select of the B-th key in the order (s descending,
//      token index ascending): the bits every key shares are skipped, the
//      first digit is 12 bits wide (one histogram, block-wide scan); the keys
//      in the cut's bucket are then compacted into LDS when they fit: at most
//      256 of them rank themselves directly, more are finished by 8-bit
//      digits counting only those;
//   3. ordered compaction: each wave owns a contiguous token segment, counts
//      its selected tokens (keys past the cut, plus the lowest-index ties at
//      the cut) with ballots, and writes them at its segment's offset, so idx
//      comes out ascending.
// Keys past the LDS cache (28K tokens) are read back from s; those passes
// keep eight loads in flight per thread.
#pragma once
#include "device_common.h"
#include "internal.h"

namespace starkv {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSelBatch = 8;             // loads in flight per thread
constexpr int kSelScoreBatch = 16;       // tokens per thread per step of the fused score
constexpr int kSelLdsKeys = 28 * 1024;   // keys cached in LDS (112 KiB)
constexpr int kSelCand = 2048;           // keys of the cut's first-digit bucket
constexpr int kSelDirect = 256;          // candidates ranked directly, no more digits

struct SelArgs {
  const float* sbar;
  const uint8_t* gstar;
  const float* scal;
  float* s;
  int32_t* idx;
  int G, Lp, B, sc, frame, cache;
  float delta, d_min;
  int tem;              // starkv_tem_decay
  int n_spans;
  int32_t start[STARKV_MAX_SPANS];
  int32_t end[STARKV_MAX_SPANS];
  int32_t sframe[STARKV_MAX_SPANS];
};


// The selection's fixed LDS: static in the selection kernel, carved from the
// statistics kernel's dynamic LDS when that kernel runs the selection.
struct SelShared {
  int hist[4096];                          // first digit; later per-wave digits
  __align__(16) uint32_t cand[kSelCand];
  int sp_start[STARKV_MAX_SPANS], sp_end[STARKV_MAX_SPANS];
  int sh_cnt[kSelWaves];
  float beta_s[STARKV_MAX_GROUPS];
  // D of a visual token depends only on its group g* and its span (the
  // frame distance): one entry per (group, span), row-major by group
  float d_tab[STARKV_MAX_GROUPS * STARKV_MAX_SPANS];
  uint32_t red_lo[kSelWaves], red_hi[kSelWaves];
  int wsel[kSelWaves], weq[kSelWaves];
  int n_cand, cut_rank, cut_eq;
  uint32_t cut_key;
};

// Fills the selection's arguments; `cache` is the number of keys the
// caller's LDS holds (at most L_p).
void fill_sel_args(SelArgs& a, const Geometry& g, const starkv_params& p, const float* sbar,
                   const uint8_t* gstar, const float* scalars, const starkv_span* spans,
                   int32_t n_spans, int32_t frame, int32_t B, float* s, int32_t* idx,
                   int cache);

namespace {

__device__ __forceinline__ void select_body(const SelArgs& a, int layer, SelShared& sh,
                                            uint32_t* keys) {
  int* const hist = sh.hist;
  uint32_t* const cand = sh.cand;
  int* const sp_start = sh.sp_start;
  int* const sp_end = sh.sp_end;
  int* const sh_cnt = sh.sh_cnt;
  float* const beta_s = sh.beta_s;
  float* const d_tab = sh.d_tab;
  uint32_t* const red_lo = sh.red_lo;
  uint32_t* const red_hi = sh.red_hi;
  int* const wsel = sh.wsel;
  int* const weq = sh.weq;
  int& n_cand = sh.n_cand;
  uint32_t& cut_key = sh.cut_key;
  int& cut_rank = sh.cut_rank;
  int& cut_eq = sh.cut_eq;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const float* scal = a.scal + (size_t)layer * a.sc;
  const float* sb = a.sbar + (size_t)layer * a.Lp;
  const uint8_t* gs = a.gstar + (size_t)layer * a.Lp;
  float* s_out = a.s + (size_t)layer * a.Lp;
  const float lam = scal[STARKV_SCAL_LAMBDA(a.G)];
  const float T = scal[STARKV_SCAL_T(a.G)];
  const float inv_t = 1.0f / T;
  const float gl = (float)a.G * lam;
  // the tables, straight from the layer's scalars (one barrier)
  if (tid < a.G) beta_s[tid] = (1.0f - lam) + gl * scal[STARKV_SCAL_W(a.G) + tid];
  if (tid < a.n_spans) {
    sp_start[tid] = a.start[tid];
    sp_end[tid] = a.end[tid];
  }
  for (int e = tid; e < a.G * a.n_spans; e += kSelThreads) {
    const int g = e / a.n_spans, sp = e - g * a.n_spans;
    const float phi = scal[STARKV_SCAL_PHI(a.G) + g];
    const float dist = (float)(a.frame - a.sframe[sp]);
    const float dp = a.delta * phi;
    float f;
    if (a.tem == STARKV_TEM_EXP) f = __expf(-a.delta * dist * phi);
    else if (a.tem == STARKV_TEM_LINEAR) f = fmaxf(0.0f, 1.0f - dp * dist);
    else f = exp2f(-dp * __log2f(1.0f + dist));   // gamma: (1 + distance)^(-delta phi)
    d_tab[e] = a.d_min + (1.0f - a.d_min) * f;
  }
  __syncthreads();

  // Keys of tokens t0 + u * step, u < kSelBatch, at or past the LDS cache
  // (0xFFFFFFFF past Lp), read back from s with kSelBatch loads in flight.
  auto far_keys = [&](int t0, int step, uint32_t (&kv)[kSelBatch]) {
    float v[kSelBatch];
#pragma unroll
    for (int u = 0; u < kSelBatch; ++u) {
      const int t = t0 + u * step;
      v[u] = t < a.Lp ? s_out[t] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kSelBatch; ++u) kv[u] = t0 + u * step < a.Lp ? ~fkey(v[u]) : 0xFFFFFFFFu;
  };
  const int n_near = min(a.cache, a.Lp);   // tokens whose keys are in LDS

  // ---- 1. fused score; keys order tokens by descending s
  uint32_t lo = 0xFFFFFFFFu, hi = 0u;
  // the first span that does not end at or before this thread's token, and
  // its bounds (past the last span: none)
  int cur = 0;
  int c_start = a.n_spans > 0 ? sp_start[0] : 0x7FFFFFFF;
  int c_end = a.n_spans > 0 ? sp_end[0] : 0x7FFFFFFF;
  for (int t0 = tid; t0 < a.Lp; t0 += kSelScoreBatch * kSelThreads) {
    float sbv[kSelScoreBatch];
    int gv[kSelScoreBatch];
#pragma unroll
    for (int u = 0; u < kSelScoreBatch; ++u) {   // 2 * kSelScoreBatch loads in flight
      const int t = t0 + u * kSelThreads;
      sbv[u] = t < a.Lp ? sb[t] : 0.f;
      gv[u] = t < a.Lp ? (int)gs[t] : 0;
    }
#pragma unroll
    for (int u = 0; u < kSelScoreBatch; ++u) {
      const int t = t0 + u * kSelThreads;
      if (t < a.Lp) {
        const int g = min(gv[u], a.G - 1);
        const float beta = beta_s[g];
        float D = 1.0f;
        while (t >= c_end) {
          ++cur;
          c_start = cur < a.n_spans ? sp_start[cur] : 0x7FFFFFFF;
          c_end = cur < a.n_spans ? sp_end[cur] : 0x7FFFFFFF;
        }
        if (t >= c_start) D = d_tab[g * a.n_spans + cur];
        const float sf = fmaxf(sbv[u] * beta * D, 0.0f);
        const float sv = (inv_t == 1.0f || sf == 0.0f) ? sf : exp2f(inv_t * __log2f(sf));
        s_out[t] = sv;
        const uint32_t k = ~fkey(sv);
        if (t < a.cache) keys[t] = k;
        lo = min(lo, k);
        hi = max(hi, k);
      }
    }
  }
  if (a.B == 0) return;
  lo = wave_min_u32(lo);
  hi = wave_max_u32(hi);
  if (lane == 0) { red_lo[wave] = lo; red_hi[wave] = hi; }
  __syncthreads();
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
  for (int w = 0; w < kSelWaves; ++w) { kmin = min(kmin, red_lo[w]); kmax = max(kmax, red_hi[w]); }

  // ---- 2. radix select of rank B-1, skipping the bits all keys share
  const int common = (kmin == kmax) ? 32 : __clz(kmin ^ kmax);
  const uint32_t cmask = common == 0 ? 0u : (common >= 32 ? 0xFFFFFFFFu : (0xFFFFFFFFu << (32 - common)));
  uint32_t ck = kmin & cmask;
  int crank = a.B - 1;
  bool first = true, compact = false;
  int n_c = 0;
  for (int done = common; done < 32;) {
    const int width = min(first ? 12 : 8, 32 - done);
    const int shift = 32 - done - width;
    const int nb = 1 << width;
    const uint32_t want = key_hi(ck, shift + width);
    if (first) {
      for (int i = tid; i < nb; i += kSelThreads) hist[i] = 0;
      __syncthreads();
      // every key shares the prefix: one histogram of the first digit
      for (int t = tid; t < n_near; t += kSelThreads) atomicAdd(&hist[(keys[t] >> shift) & (nb - 1)], 1);
      for (int t0 = n_near + tid; t0 < a.Lp; t0 += kSelBatch * kSelThreads) {
        uint32_t kv[kSelBatch];
        far_keys(t0, kSelThreads, kv);
#pragma unroll
        for (int u = 0; u < kSelBatch; ++u)
          if (t0 + u * kSelThreads < a.Lp) atomicAdd(&hist[(kv[u] >> shift) & (nb - 1)], 1);
      }
      __syncthreads();
      int c[4], sum = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        c[j] = (4 * tid + j < nb) ? hist[4 * tid + j] : 0;
        sum += c[j];
      }
      int tot;
      const int exc = block_excl_scan(sum, sh_cnt, &tot);
      if (exc <= crank && crank < exc + sum) {
        int run = exc;
        for (int j = 0; j < 4; ++j) {
          if (crank < run + c[j]) {
            cut_key = ck | ((uint32_t)(4 * tid + j) << shift);
            cut_rank = crank - run;
            cut_eq = c[j];
            break;
          }
          run += c[j];
        }
      }
      if (tid == 0) n_cand = 0;
      __syncthreads();
      ck = cut_key;
      crank = cut_rank;
      if (done + width < 32 && cut_eq <= kSelCand) {
        // the keys of the cut's bucket, in any order
        const uint32_t pre = key_hi(ck, shift);
        const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
        auto keep = [&](uint32_t k, bool valid) {   // the whole wave calls it
          const bool m = valid && key_hi(k, shift) == pre;
          const uint64_t bal = __ballot(m);
          int base = 0;
          if (lane == 0 && bal) base = atomicAdd(&n_cand, __popcll(bal));
          base = __shfl(base, 0);
          if (m) cand[base + __popcll(bal & below)] = k;
        };
        for (int t0 = 0; t0 < n_near; t0 += kSelThreads) {
          const int t = t0 + tid;
          keep(t < n_near ? keys[t] : 0u, t < n_near);
        }
        for (int b0 = n_near; b0 < a.Lp; b0 += kSelBatch * kSelThreads) {
          uint32_t kv[kSelBatch];
          far_keys(b0 + tid, kSelThreads, kv);
#pragma unroll
          for (int u = 0; u < kSelBatch; ++u) keep(kv[u], b0 + u * kSelThreads + tid < a.Lp);
        }
        __syncthreads();
        compact = true;
        n_c = n_cand;
        if (n_c <= kSelDirect) {
          // few candidates: each ranks itself; the one whose rank range holds
          // the cut's rank is the cut key
          if (tid < n_c) {
            const uint32_t key = cand[tid];
            int less = 0, eq = 0;
            for (int j0 = 0; j0 < n_c; j0 += 8) {   // 8 keys per trip, 2 reads in flight
              const i32x4 v0 = *reinterpret_cast<const i32x4*>(cand + j0);
              const i32x4 v1 = *reinterpret_cast<const i32x4*>(cand + j0 + 4);
#pragma unroll
              for (int u = 0; u < 8; ++u) {
                const uint32_t kj = (uint32_t)(u < 4 ? v0[u] : v1[u - 4]);
                if (j0 + u < n_c) {
                  less += kj < key;
                  eq += kj == key;
                }
              }
            }
            if (less <= crank && crank < less + eq) {
              cut_key = key;         // equal keys write equal values
              cut_rank = crank - less;
            }
          }
          __syncthreads();
          ck = cut_key;
          crank = cut_rank;
          done = 32 - width;   // the cut is exact: no more digits
        }
      }
    } else {
      for (int i = tid; i < kSelWaves * 256; i += kSelThreads) hist[i] = 0;
      __syncthreads();
      if (compact) {
        for (int i = tid; i < n_c; i += kSelThreads) {
          const uint32_t k = cand[i];
          if (key_hi(k, shift + width) == want)
            atomicAdd(&hist[wave * 256 + ((k >> shift) & (nb - 1))], 1);
        }
      } else {
        auto count = [&](uint32_t k) {
          if (key_hi(k, shift + width) == want)
            atomicAdd(&hist[wave * 256 + ((k >> shift) & (nb - 1))], 1);
        };
        for (int t = tid; t < n_near; t += kSelThreads) count(keys[t]);
        for (int t0 = n_near + tid; t0 < a.Lp; t0 += kSelBatch * kSelThreads) {
          uint32_t kv[kSelBatch];
          far_keys(t0, kSelThreads, kv);
#pragma unroll
          for (int u = 0; u < kSelBatch; ++u)
            if (t0 + u * kSelThreads < a.Lp) count(kv[u]);
        }
      }
      __syncthreads();
      if (tid < nb) {
        int sum = 0;
        for (int w = 0; w < kSelWaves; ++w) sum += hist[w * 256 + tid];
        hist[tid] = sum;
      }
      __syncthreads();
      if (wave == 0) {
        int d, before, cnt;
        wave_find_bin(hist, nb, crank, &d, &before, &cnt);
        if (lane == 0) {
          cut_key = ck | ((uint32_t)d << shift);
          cut_rank = crank - before;
          cut_eq = cnt;
        }
      }
      __syncthreads();
      ck = cut_key;
      crank = cut_rank;
    }
    done += width;
    first = false;
  }

  // ---- 3. ordered compaction: each wave owns a contiguous token segment.
  // Selected: key < ck, or key == ck among the first crank+1 such tokens.
  const int seg = ((a.Lp + kSelWaves * 64 - 1) / (kSelWaves * 64)) * 64;
  const int t0 = wave * seg, t1 = min(t0 + seg, a.Lp);
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  // the segment's tokens in LDS, then the ones past the cache
  const int tn = min(max(t0, n_near), t1);
  int n_strict = 0, n_eq = 0;
  auto tally = [&](int t, uint32_t k) {
    n_strict += __popcll(__ballot(t < t1 && k < ck));
    n_eq += __popcll(__ballot(t < t1 && k == ck));
  };
  for (int base = t0; base < tn; base += 64) {
    const int t = base + lane;
    tally(t < tn ? t : t1, t < tn ? keys[t] : 0xFFFFFFFFu);
  }
  for (int b = tn; b < t1; b += kSelBatch * 64) {
    uint32_t kv[kSelBatch];
    far_keys(b + lane, 64, kv);
#pragma unroll
    for (int u = 0; u < kSelBatch; ++u) tally(b + u * 64 + lane, kv[u]);
  }
  if (lane == 0) { wsel[wave] = n_strict; weq[wave] = n_eq; }
  __syncthreads();
  int off = 0, eq_off = 0;
  for (int w = 0; w < wave; ++w) {
    off += wsel[w] + max(0, min(crank + 1 - eq_off, weq[w]));
    eq_off += weq[w];
  }
  int32_t* out = a.idx + (size_t)layer * a.B;
  auto emit = [&](int t, uint32_t k) {   // tokens in ascending order
    const bool strict = t < t1 && k < ck;
    const bool eq = t < t1 && k == ck;
    const uint64_t meq = __ballot(eq);
    const int eqpos = eq_off + __popcll(meq & below);
    const bool sel = strict || (eq && eqpos <= crank);
    const uint64_t msel = __ballot(sel);
    const int pos = off + __popcll(msel & below);
    if (sel && pos < a.B) out[pos] = t;
    off += __popcll(msel);
    eq_off += __popcll(meq);
  };
  for (int base = t0; base < tn; base += 64) {
    const int t = base + lane;
    emit(t < tn ? t : t1, t < tn ? keys[t] : 0xFFFFFFFFu);
  }
  for (int b = tn; b < t1; b += kSelBatch * 64) {
    uint32_t kv[kSelBatch];
    far_keys(b + lane, 64, kv);
#pragma unroll
    for (int u = 0; u < kSelBatch; ++u) emit(b + u * 64 + lane, kv[u]);
  }
}

}  // namespace
}  // namespace starkv
