// Window attention scoring (sec. 3.3): A_raw summed over the window rows and
// the heads of each KV group, then AvgPool1D, group mean, sbar and g*.
//
// The window softmax of every query row needs that row's max and sum over
// all L_p past keys before any key's normalised mass is known, so scoring
// runs in two passes over K:
//   pass 1  per (layer, group, token chunk): for each window row r, a
//           reference M_r no larger than the chunk's max and the sum of
//           2^(y - M_r), y = q.k * log2(e)/sqrt(d);
//   pass 2  merges the chunk statistics into c_r = M_r + log2(l_r) (every
//           block for its own group) and sums 2^(y_rt - c_r) over the
//           group's rows for every token t.
// Both passes run the Q_g x K^T contraction on 32x32 MFMA tiles.  A block
// has one wave per 32-row block of the group's R = W*H/G window rows; each
// wave keeps its rows' Q fragments in registers for the whole kernel, and
// the block streams its token range of K through double-buffered LDS tiles
// that every wave reads.  Pass 1 puts tokens on the MFMA M axis, so each lane
// owns one query row and reduces over its tokens in registers.  Pass 2 puts
// query rows on M, so each lane owns one token and reduces over its rows.
#pragma once
#include "device_common.h"
#include "internal.h"

namespace starkv {

struct ScoreArgs {
  const void* q;
  const void* k;
  int64_t ls, gs, ts;   // element strides of the K cache
  int H, G, W, R, Rpad, Lp;
  int chunk, n_chunks, n_chunks_max;
  float scale;          // log2(e) / sqrt(d)
  float2* part;         // [n_layers][G][n_chunks_max][Rpad]  (M, l)
  float* sraw;          // [n_layers][Ns][Lp]
  // pass-2 output per KV group: n_out subspaces (1, or H/G per head), each
  // the sum of upo stored partials; a wave stores n_part partials per token
  // (1: its 32 rows, 4: one per 8-row group)
  int n_out, upo, n_part, Ns;
};

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegBig = -1e30f;

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

// The value lane l ^ 32 holds.  v_permlane32_swap exchanges the upper lane
// half of its first operand with the lower half of its second, so with both
// operands = v the first result holds the lower half's values in the upper
// lanes and the second the upper half's values in the lower lanes.
__device__ inline float other_half(float v, int half) {
  const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(half ? sw[0] : sw[1]);
}

// Work item of a scoring block: (chunk, group, layer).  Blocks are dealt to
// the 8 XCDs round-robin by id, so the id is permuted to give every XCD a
// contiguous range of items: the chunks of one (layer, group) then share
// that XCD's L2 for their window queries.  The map is a bijection of
// [0, n), so it is correct whatever the placement.
__device__ inline void score_item(const ScoreArgs& a, int* chunk, int* g, int* layer) {
  const int n = gridDim.x, b = blockIdx.x;
  const int xcd = b & 7, local = b >> 3, per = n >> 3, rem = n & 7;
  const int id = xcd < rem ? xcd * (per + 1) + local
                           : rem * (per + 1) + (xcd - rem) * per + local;
  *chunk = id % a.n_chunks;
  const int lg = id / a.n_chunks;
  *g = lg % a.G;
  *layer = lg / a.G;
}

// K is staged through LDS in 128-token tiles (rows padded by 16 bytes), two
// tiles in flight: the next tile's rows are fetched into registers while the
// current tile is multiplied, then written to the other LDS buffer.
template <typename T, int D, int NTHREADS>
struct KStage {
  static constexpr int kRows = 128;
  static constexpr int kStride = D + 16 / (int)sizeof(T);
  static constexpr int kVecPerRow = D * (int)sizeof(T) / 16;
  static constexpr int kElemPerVec = 16 / (int)sizeof(T);
  static constexpr int kVecs = kRows * kVecPerRow;
  static constexpr int kPerThread = (kVecs + NTHREADS - 1) / NTHREADS;
  static constexpr int kElems = kRows * kStride;
  // Thread t stages vectors t + j*NTHREADS: the same 16-byte column of rows
  // t/kVecPerRow + j*kRowStep, since NTHREADS is a multiple of kVecPerRow.
  static_assert(NTHREADS % kVecPerRow == 0, "row-aligned staging");
  static constexpr int kRowStep = NTHREADS / kVecPerRow;
  // vector j may fall past the tile's last row (then it repeats that row)
  static constexpr bool may_pass(int j) { return (kRowStep - 1) + j * kRowStep >= kRows; }
};

// Tile staging.  stage_fetch loads the 16-byte vectors a thread stages of
// the tile of rows t0 .. t0+127 into registers; stage_store writes them to
// an LDS tile buffer.  Every load and store is unconditional: rows past the
// tile repeat its last row, and with `full` false (the tile reaches past
// L_p) tokens are clamped to L_p - 1.  With `full` true every row lies
// before L_p, so the addresses step by one uniform stride.  Both are forced
// inline so that the staging array stays in registers.
template <typename KS, typename T>
__device__ __forceinline__ void stage_fetch(i32x4 (&r)[KS::kPerThread], const T* kg,
                                            int64_t ts, int t0, int Lp, bool full) {
  const int r0 = (int)threadIdx.x / KS::kVecPerRow;
  const int c0 = ((int)threadIdx.x % KS::kVecPerRow) * KS::kElemPerVec;
  if (full) {
    const T* p = kg + (int64_t)(t0 + r0) * ts + c0;
#pragma unroll
    for (int j = 0; j < KS::kPerThread; ++j) {
      if (KS::may_pass(j)) {
        const int row = min(r0 + j * KS::kRowStep, KS::kRows - 1);
        r[j] = *reinterpret_cast<const i32x4*>(kg + (int64_t)(t0 + row) * ts + c0);
      } else {
        r[j] = *reinterpret_cast<const i32x4*>(p + (int64_t)(j * KS::kRowStep) * ts);
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < KS::kPerThread; ++j) {
      const int row = min(r0 + j * KS::kRowStep, KS::kRows - 1);
      const int tok = min(t0 + row, Lp - 1);
      r[j] = *reinterpret_cast<const i32x4*>(kg + (int64_t)tok * ts + c0);
    }
  }
}

template <typename KS, typename T>
__device__ __forceinline__ void stage_store(const i32x4 (&r)[KS::kPerThread], T* buf) {
  const int r0 = (int)threadIdx.x / KS::kVecPerRow;
  const int c0 = ((int)threadIdx.x % KS::kVecPerRow) * KS::kElemPerVec;
  T* q = buf + r0 * KS::kStride + c0;
#pragma unroll
  for (int j = 0; j < KS::kPerThread; ++j) {
    if (KS::may_pass(j)) {
      const int row = min(r0 + j * KS::kRowStep, KS::kRows - 1);
      *reinterpret_cast<i32x4*>(buf + row * KS::kStride + c0) = r[j];
    } else {
      *reinterpret_cast<i32x4*>(q + j * KS::kRowStep * KS::kStride) = r[j];
    }
  }
}

// Q fragments of the 32 window rows a wave owns (row block `wave` of the
// group), held in registers for the whole kernel; rows past R are zero.
template <typename T, int D>
__device__ inline void load_q_frags(const T* qg, int R, int wave,
                                    typename Mfma<T>::frag* qf) {
  using M = Mfma<T>;
  constexpr int NK = D / M::kStep;
  const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  const int row = wave * 32 + l32;
  const T* qrow = qg + (size_t)min(row, R - 1) * D;
#pragma unroll
  for (int kk = 0; kk < NK; ++kk) {
    qf[kk] = M::load(qrow, kk, half);
    if (row >= R) qf[kk] = typename M::frag{};
  }
}

// ---------------------------------------------------------------- pass 1
// One wave per 32-row block of the group's window rows (NRB waves).  Tokens
// sit on the MFMA M axis, so each lane keeps (max, sum) for one query row
// over the 16 tokens it receives per 32-token block.
template <typename T, int D, int NRB>
__global__ __launch_bounds__(NRB * 64) void score_pass1(ScoreArgs a) {
  using M = Mfma<T>;
  using KS = KStage<T, D, NRB * 64>;
  constexpr int NK = D / M::kStep;
  extern __shared__ __align__(16) unsigned char smem[];
  T* kbuf = reinterpret_cast<T*>(smem);

  int chunk, g, layer;
  score_item(a, &chunk, &g, &layer);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const T* kg = group_k<T>(a, layer, g);
  const int t_begin = chunk * a.chunk;
  const int t_end = min(t_begin + a.chunk, a.Lp);

  typename M::frag qf[NK];
  load_q_frags<T, D>(group_q<T, D>(a, layer, g), a.R, wave, qf);
  i32x4 sr[KS::kPerThread];
  stage_fetch<KS>(sr, kg, a.ts, t_begin, a.Lp, t_begin + KS::kRows <= a.Lp);
  stage_store<KS>(sr, kbuf);
  __syncthreads();

  // (m, l): reference logit and sum of 2^((y - m) * log2e/sqrt(d)) of the
  // lane's row over the tokens seen so far.  Any reference gives the same
  // statistics once merged, so m is not the running max: it is moved only
  // when a block's sum would leave [0, 2^32), i.e. before the first block
  // and when logits rise well above it.
  float m = kNegBig, ms = kNegBig * a.scale, l = 0.f;
  // MFMA chain of one 32-token block: acc[4i+j] = token 32b + 8i + 4*half + j,
  // query row wave*32 + l32
  auto chain = [&](const T* tile, int b) {
    const T* krow = tile + (32 * b + l32) * KS::kStride;
    f32x16 acc = {};
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) acc = M::mma(M::load(krow, kk, half), qf[kk], acc);
    return acc;
  };
  auto epilogue = [&](f32x16& acc, int tb, bool full) {
    if (full) {
      // against the kept reference: no max and no rescale.  With no
      // reference yet (m = -1e30) the sum is +inf; a sum of 2^32 or more
      // means the block's logits exceed m by more than 18 log2 units (l
      // counts at most 2^14 tokens of mass <= 1 otherwise).  Both, and a NaN,
      // redo the block below against the block's exact max.
      float sum = __builtin_amdgcn_exp2f(fmaf(acc[0], a.scale, -ms));
#pragma unroll
      for (int e = 1; e < 16; ++e) sum += __builtin_amdgcn_exp2f(fmaf(acc[e], a.scale, -ms));
      const float ln = l + sum;
      if (ln < 4294967296.0f) {
        l = ln;
        return;
      }
    }
    float mt;
    if (full) {
      mt = acc[0];
#pragma unroll
      for (int e = 1; e < 16; ++e) mt = fmaxf(mt, acc[e]);
    } else {
      mt = -INFINITY;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int t = tb + 8 * (e >> 2) + 4 * half + (e & 3);
        acc[e] = (t < t_end) ? acc[e] : -INFINITY;
        mt = fmaxf(mt, acc[e]);
      }
    }
    const float mn = fmaxf(m, mt);
    const float msn = mn * a.scale;
    float sum = __builtin_amdgcn_exp2f(fmaf(acc[0], a.scale, -msn));
#pragma unroll
    for (int e = 1; e < 16; ++e) sum += __builtin_amdgcn_exp2f(fmaf(acc[e], a.scale, -msn));
    l = l * rescale(m, mn, msn, a.scale) + sum;
    m = mn;
    ms = msn;
  };
  int buf = 0;
  for (int t0 = t_begin; t0 < t_end; t0 += KS::kRows) {
    const bool more = t0 + KS::kRows < t_end;
    if (more) stage_fetch<KS>(sr, kg, a.ts, t0 + KS::kRows, a.Lp, t0 + 2 * KS::kRows <= a.Lp);
    const T* tile = kbuf + buf * KS::kElems;
    if (t0 + KS::kRows <= t_end) {
      // full tile: branch-free, the MFMA chain of block b+1 is issued before
      // the epilogue of block b so that the matrix core and the VALU overlap
      f32x16 a0 = chain(tile, 0), a1;
#pragma unroll
      for (int b = 0; b < KS::kRows / 32; ++b) {
        if (b + 1 < KS::kRows / 32) a1 = chain(tile, b + 1);
        epilogue(a0, t0 + 32 * b, true);
        a0 = a1;
      }
    } else {
#pragma unroll
      for (int b = 0; b < KS::kRows / 32; ++b) {
        const int tb = t0 + 32 * b;
        if (tb < t_end) {
          f32x16 acc = chain(tile, b);
          epilogue(acc, tb, false);
        }
      }
    }
    if (more) stage_store<KS>(sr, kbuf + (buf ^ 1) * KS::kElems);
    __syncthreads();
    buf ^= 1;
  }
  // the two lane halves hold the same query row over other tokens
  const float mo = other_half(m, half), lo = other_half(l, half);
  const float mn = fmaxf(m, mo);
  const float msn = mn * a.scale;
  l = l * rescale(m, mn, msn, a.scale) + lo * rescale(mo, mn, msn, a.scale);
  if (half == 0) {
    float2* out = a.part + ((size_t)(layer * a.G + g) * a.n_chunks_max + chunk) * a.Rpad;
    out[wave * 32 + l32] = make_float2(msn, l);
  }
}

// ---------------------------------------------------------------- merge
// c_r = M_r + log2(l_r) of row r of one (layer, group) from its chunks'
// statistics, in a fixed merge order; rows past R get +inf so that their
// 2^(y - c) vanishes in pass 2.
__device__ inline float merge_row(const ScoreArgs& a, const float2* part, int r) {
  float Mx = kNegBig, lx = 0.f;
  for (int c0 = 0; c0 < a.n_chunks; c0 += 8) {
    float2 p[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)   // eight loads in flight
      p[j] = c0 + j < a.n_chunks ? part[(size_t)(c0 + j) * a.Rpad + r]
                                 : make_float2(kNegBig, 0.f);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float mn = fmaxf(Mx, p[j].x);
      lx = lx * __builtin_amdgcn_exp2f(Mx - mn) + p[j].y * __builtin_amdgcn_exp2f(p[j].x - mn);
      Mx = mn;
    }
  }
  return (r < a.R) ? Mx + log2f(lx) : INFINITY;
}

// ---------------------------------------------------------------- pass 2
// Query rows on the MFMA M axis: each lane owns one token of the 32-token
// block and sums 2^(y - c_r) over the 16 rows of the wave's row block it
// holds (c_r in registers), or four partial sums of its 8-row groups when
// heads are narrower than the row block; the two lane halves are added by a
// lane swap, then the partials of each output subspace in a fixed order
// through LDS.  Each block first merges its
// group's chunk statistics into c_r (one row per thread) while its first K
// tile is in flight.
// SUB: several subspaces per KV group (per-head scores); otherwise the
// block writes one sum per token and the layout fields are not read.
template <typename T, int D, int NRB, bool SUB>
__global__ __launch_bounds__(NRB * 64) void score_pass2(ScoreArgs a) {
  using M = Mfma<T>;
  using KS = KStage<T, D, NRB * 64>;
  constexpr int NK = D / M::kStep;
  extern __shared__ __align__(16) unsigned char smem[];
  T* kbuf = reinterpret_cast<T*>(smem);
  float* red = reinterpret_cast<float*>(smem + 2 * (size_t)KS::kElems * sizeof(T));

  int chunk, g, layer;
  score_item(a, &chunk, &g, &layer);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const T* kg = group_k<T>(a, layer, g);
  const int t_begin = chunk * a.chunk;
  const int t_end = min(t_begin + a.chunk, a.Lp);
  const int n_part = SUB ? a.n_part : 1;
  float* srow = SUB ? a.sraw + ((size_t)layer * a.Ns + (size_t)g * a.n_out) * a.Lp
                    : a.sraw + (size_t)(layer * a.G + g) * a.Lp;

  __shared__ __align__(16) float cs[NRB * 32];
  i32x4 sr[KS::kPerThread];
  stage_fetch<KS>(sr, kg, a.ts, t_begin, a.Lp, t_begin + KS::kRows <= a.Lp);
  typename M::frag qf[NK];
  load_q_frags<T, D>(group_q<T, D>(a, layer, g), a.R, wave, qf);
  {
    const float2* part = a.part + (size_t)(layer * a.G + g) * a.n_chunks_max * a.Rpad;
    for (int r = threadIdx.x; r < NRB * 32; r += NRB * 64) cs[r] = merge_row(a, part, r);
  }
  stage_store<KS>(sr, kbuf);
  __syncthreads();
  // c of the rows this lane receives: wave*32 + 8i + 4*half + j
  float c[16];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const f32x4 c4 = *reinterpret_cast<const f32x4*>(cs + wave * 32 + 4 * half + 8 * i);
#pragma unroll
    for (int j = 0; j < 4; ++j) c[4 * i + j] = c4[j];
  }

  int buf = 0;
  for (int t0 = t_begin; t0 < t_end; t0 += KS::kRows) {
    const bool more = t0 + KS::kRows < t_end;
    if (more) stage_fetch<KS>(sr, kg, a.ts, t0 + KS::kRows, a.Lp, t0 + 2 * KS::kRows <= a.Lp);
    const T* tile = kbuf + buf * KS::kElems;
    float* rs = red + buf * (NRB * n_part * KS::kRows);
#pragma unroll
    for (int b = 0; b < KS::kRows / 32; ++b) {
      const T* krow = tile + (32 * b + l32) * KS::kStride;
      f32x16 acc = {};
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) acc = M::mma(qf[kk], M::load(krow, kk, half), acc);
      // the other lane half's rows are added through a VALU lane swap (a
      // shuffle would round-trip through LDS and wait on the fragment
      // reads); both halves then hold the same sum and store it to the same
      // address
      if (n_part == 1) {
        float v = __builtin_amdgcn_exp2f(fmaf(acc[0], a.scale, -c[0]));
#pragma unroll
        for (int e = 1; e < 16; ++e) v += __builtin_amdgcn_exp2f(fmaf(acc[e], a.scale, -c[e]));
        v += other_half(v, half);
        rs[wave * KS::kRows + 32 * b + l32] = v;
      } else {
        // one partial per 8-row group: rows 8i + 4*half + (0..3) here
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = __builtin_amdgcn_exp2f(fmaf(acc[4 * i], a.scale, -c[4 * i]));
#pragma unroll
          for (int j = 1; j < 4; ++j)
            v += __builtin_amdgcn_exp2f(fmaf(acc[4 * i + j], a.scale, -c[4 * i + j]));
          rs[(wave * 4 + i) * KS::kRows + 32 * b + l32] = v + other_half(v, half);
        }
      }
    }
    if (more) stage_store<KS>(sr, kbuf + (buf ^ 1) * KS::kElems);
    __syncthreads();
    if (!SUB) {           // one subspace per group: all NRB wave sums
      for (int i = threadIdx.x; i < KS::kRows; i += NRB * 64) {
        if (t0 + i < t_end) {
          float sum = 0.f;
#pragma unroll
          for (int w = 0; w < NRB; ++w) sum += rs[w * KS::kRows + i];
          srow[t0 + i] = sum;
        }
      }
    } else {              // per head: upo consecutive partials per head
      for (int it = threadIdx.x; it < a.n_out * KS::kRows; it += NRB * 64) {
        const int o = it / KS::kRows, i = it % KS::kRows;
        if (t0 + i < t_end) {
          float sum = 0.f;
          for (int u = o * a.upo; u < (o + 1) * a.upo; ++u) sum += rs[u * KS::kRows + i];
          srow[(size_t)o * a.Lp + t0 + i] = sum;
        }
      }
    }
    buf ^= 1;
  }
}

template <typename T, int D, int NRB>
int run_passes(const ScoreArgs& a, int n_layers, hipStream_t st) {
  using KS = KStage<T, D, NRB * 64>;
  const int items = a.n_chunks * a.G * n_layers;
  const size_t lds1 = 2 * (size_t)KS::kElems * sizeof(T);
  const size_t lds2 = lds1 + 2 * (size_t)NRB * a.n_part * KS::kRows * sizeof(float);
  score_pass1<T, D, NRB><<<items, NRB * 64, lds1, st>>>(a);
  if (a.n_out > 1)
    score_pass2<T, D, NRB, true><<<items, NRB * 64, lds2, st>>>(a);
  else
    score_pass2<T, D, NRB, false><<<items, NRB * 64, lds2, st>>>(a);
  return (int)hipGetLastError();
}

template <typename T, int D>
int run_nrb(const ScoreArgs& a, int n_layers, hipStream_t st) {
  switch (a.Rpad / 32) {
#define STARKV_NRB(n) \
  case n: return run_passes<T, D, n>(a, n_layers, st);
    STARKV_NRB(1) STARKV_NRB(2) STARKV_NRB(3) STARKV_NRB(4) STARKV_NRB(5) STARKV_NRB(6)
    STARKV_NRB(7) STARKV_NRB(8) STARKV_NRB(9) STARKV_NRB(10) STARKV_NRB(11)
    STARKV_NRB(12) STARKV_NRB(13) STARKV_NRB(14) STARKV_NRB(15) STARKV_NRB(16)
#undef STARKV_NRB
  }
  return (int)hipErrorInvalidValue;
}

template <typename T, int D>
int run_nrb_small(const ScoreArgs& a, int n_layers, hipStream_t st) {
  switch (a.Rpad / 32) {
    case 1: return run_passes<T, D, 1>(a, n_layers, st);
    case 2: return run_passes<T, D, 2>(a, n_layers, st);
    case 3: return run_passes<T, D, 3>(a, n_layers, st);
    case 4: return run_passes<T, D, 4>(a, n_layers, st);
  }
  return (int)hipErrorInvalidValue;
}

}  // namespace

// Runners of the two passes, one translation unit per element type.
int run_score_bf16(const ScoreArgs& a, int d, int n_layers, hipStream_t st);
int run_score_f32(const ScoreArgs& a, int d, int n_layers, hipStream_t st);

}  // namespace starkv
