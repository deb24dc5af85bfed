// Pass 2 of the window scoring (sec. 3.3, Eq. A_raw) for bf16 keys with
// d = 128: for every past token t of a (layer, group), sum_r 2^(y_rt - c_r)
// over the group's R window rows, with y = q.k * log2(e)/sqrt(d) and c_r the
// row's log2-sum-exp from pass 1.  With one scoring subspace per KV group
// the sum runs over all R rows; with per-head subspaces (PH), when each
// head's W rows are whole 32-row blocks, over each head's own rows, one
// output per head.
//
// Persistent design: one 512-thread block per CU walks a contiguous range
// of the flattened (layer-group, 64-token slab) space.  For each group
// segment of its range the block stages the group's window rows in LDS
// (padded rows) together with c_r, merged once from the pass-1 chunk
// statistics.  Each wave then takes whole slabs: it loads the slab's 64 K
// rows straight from global memory into MFMA fragment registers (two
// 32-token blocks), and for every 32-row block of the group it reads each Q
// fragment once from LDS and feeds it to two v_mfma_f32_32x32x16_bf16, so
// every token's sum over all R rows is completed inside one wave (no
// cross-wave reduction, no barrier in the main loop).  The MFMAs of row
// block rb+1 are interleaved with the exponentials of row block rb.
#pragma once
#include "score_kernels.h"

namespace starkv {

struct SlabGrid {
  int S;      // 64-token slabs per (layer, group)
  int nlg;    // layers * groups
};

namespace {

template <int NRB>
struct SlabLds {
  static constexpr int kQS = 136;                           // padded Q row (272 B)
  static constexpr int kQBytes = NRB * 32 * kQS * 2;
  static constexpr int kBytes = kQBytes + NRB * 32 * 4;     // + c_r
};

// Blocks are dealt to the 8 XCDs round-robin by id; the id is permuted so
// that each XCD walks one contiguous part of the slab space (a bijection of
// [0, gridDim.x)).
__device__ inline int slab_block() {
  const int n = gridDim.x, b = blockIdx.x;
  const int xcd = b & 7, local = b >> 3, per = n >> 3, rem = n & 7;
  return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

template <int NRB, bool PH>
__global__ __launch_bounds__(512) void score_pass2_slab(ScoreArgs a, SlabGrid sg) {
  using T = __bf16;
  using M = Mfma<T>;
  constexpr int NW = 8, TB = 2, SLAB = 64;
  constexpr int QS = SlabLds<NRB>::kQS;
  extern __shared__ __align__(16) unsigned char smem[];
  T* qs = reinterpret_cast<T*>(smem);
  float* cs = reinterpret_cast<float*>(smem + SlabLds<NRB>::kQBytes);

  const int nb = gridDim.x, b = slab_block();
  const long total = (long)sg.S * sg.nlg;
  const long lo = (long)b * total / nb, hi = (long)(b + 1) * total / nb;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int half = lane >> 5, l32 = lane & 31;
  const T* qlane = qs + l32 * QS + half * 8;
  const float* clane = cs + 4 * half;

  for (long x = lo; x < hi;) {
    const int lg = (int)(x / sg.S);
    const int s0 = (int)(x % sg.S);
    const int s1 = (int)min((long)sg.S, s0 + (hi - x));
    const int layer = lg / a.G, g = lg % a.G;
    const T* kg = group_k<T>(a, layer, g);
    // the group's first output row: its only one, or its first head's
    float* srow = a.sraw + (size_t)lg * (PH ? a.n_out : 1) * a.Lp;

    // the group's window rows (rows R..NRB*32 zero), in batches of at most
    // seven 16-byte vectors per thread, each batch's loads issued before
    // its stores
    {
      const T* qg = group_q<T, 128>(a, layer, g);
      constexpr int NV = NRB * 32 * 16;
      constexpr int PER = (NV + NW * 64 - 1) / (NW * 64);
      constexpr int BATCH = PER < 7 ? PER : 7;
#pragma unroll
      for (int j0 = 0; j0 < PER; j0 += BATCH) {
        i32x4 v[BATCH];
#pragma unroll
        for (int j = 0; j < BATCH; ++j) {
          const int i = threadIdx.x + (j0 + j) * NW * 64, row = i >> 4, part = i & 15;
          v[j] = i32x4{0, 0, 0, 0};
          if (j0 + j < PER && i < NV && row < a.R)
            v[j] = *reinterpret_cast<const i32x4*>(qg + (size_t)row * 128 + part * 8);
        }
#pragma unroll
        for (int j = 0; j < BATCH; ++j) {
          const int i = threadIdx.x + (j0 + j) * NW * 64, row = i >> 4, part = i & 15;
          if (j0 + j < PER && i < NV) *reinterpret_cast<i32x4*>(qs + row * QS + part * 8) = v[j];
        }
      }
    }
    {
      const float2* part = a.part + (size_t)lg * a.n_chunks_max * a.Rpad;
      for (int r = threadIdx.x; r < NRB * 32; r += NW * 64) cs[r] = merge_row(a, part, r);
    }
    // K fragments of one slab: token block cb, row (token) l32, the 8
    // k-slices of this lane half; tokens past L_p re-read the last token
    // and are not stored
    bf16x8 kf[TB][8];
    auto load_slab = [&](int slab) {
#pragma unroll
      for (int cb = 0; cb < TB; ++cb) {
        const int tok = min(slab * SLAB + cb * 32 + l32, a.Lp - 1);
        const T* krow = kg + (int64_t)tok * a.ts + half * 8;
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) kf[cb][kk] = *reinterpret_cast<const bf16x8*>(krow + kk * 16);
      }
    };
    if (s0 + wave < s1) load_slab(s0 + wave);
    __syncthreads();

    for (int slab = s0 + wave; slab < s1; slab += NW) {
      // two partial sums per token block keep the add chains short
      float s[TB][2];
#pragma unroll
      for (int cb = 0; cb < TB; ++cb) { s[cb][0] = 0.f; s[cb][1] = 0.f; }
      f32x16 accA[TB], accB[TB];
      bf16x8 qf[8];
      // row block 0's chain; the fragments of row block 1 are read as
      // those of row block 0 are consumed
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) qf[kk] = *reinterpret_cast<const bf16x8*>(qlane + kk * 16);
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
#pragma unroll
        for (int cb = 0; cb < TB; ++cb) accA[cb] = M::mma(qf[kk], kf[cb][kk], kk ? accA[cb] : f32x16{});
        if (NRB > 1) qf[kk] = *reinterpret_cast<const bf16x8*>(qlane + 32 * QS + kk * 16);
      }
      __builtin_amdgcn_sched_barrier(0);
      // stage rb: MFMAs of row block rb+1 (reading the Q fragments of rb+2
      // behind them), interleaved with the exponentials of row block rb
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb) {
        f32x16 (&cur)[TB] = (rb & 1) ? accB : accA;
        f32x16 (&nxt)[TB] = (rb & 1) ? accA : accB;
        // c of the rows this lane receives: rb*32 + 8i + 4*half + j
        float c[16];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const f32x4 c4 = *reinterpret_cast<const f32x4*>(clane + rb * 32 + 8 * i);
#pragma unroll
          for (int j = 0; j < 4; ++j) c[4 * i + j] = c4[j];
        }
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) {
          if (rb + 1 < NRB) {
#pragma unroll
            for (int cb = 0; cb < TB; ++cb) nxt[cb] = M::mma(qf[kk], kf[cb][kk], kk ? nxt[cb] : f32x16{});
            if (rb + 2 < NRB) qf[kk] = *reinterpret_cast<const bf16x8*>(qlane + (rb + 2) * 32 * QS + kk * 16);
          }
#pragma unroll
          for (int cb = 0; cb < TB; ++cb)
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2)
              s[cb][h2] += __builtin_amdgcn_exp2f(fmaf(cur[cb][2 * kk + h2], a.scale, -c[2 * kk + h2]));
          if (rb + 1 < NRB) {
            // one MFMA, then the epilogue's share of six VALU operations
#pragma unroll
            for (int cb = 0; cb < TB; ++cb) {
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
              __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
            }
            if (rb + 2 < NRB) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
        }
        // pin the partial sums to this stage: the compiler would otherwise
        // sink every stage's exponentials to the end of the slab and keep
        // all accumulators alive
#pragma unroll
        for (int cb = 0; cb < TB; ++cb) {
          asm volatile("" : "+v"(s[cb][0]));
          asm volatile("" : "+v"(s[cb][1]));
        }
        if (PH && (rb + 1) % a.upo == 0) {
          // the last row block of head rb / upo: its output, then a fresh sum
          float* hrow = srow + (size_t)(rb / a.upo) * a.Lp;
#pragma unroll
          for (int cb = 0; cb < TB; ++cb) {
            const float sc = s[cb][0] + s[cb][1];
            const float v = sc + other_half(sc, half);
            const int tok = slab * SLAB + cb * 32 + l32;
            if ((cb & 1) == half && tok < a.Lp) hrow[tok] = v;
            s[cb][0] = 0.f;
            s[cb][1] = 0.f;
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      const int t0 = slab * SLAB;
      if (slab + NW < s1) load_slab(slab + NW);
      // lanes l and l ^ 32 hold the same token's two row halves; half h
      // stores token block h
      if (!PH) {
#pragma unroll
        for (int cb = 0; cb < TB; ++cb) {
          const float sc = s[cb][0] + s[cb][1];
          const float v = sc + other_half(sc, half);
          const int tok = t0 + cb * 32 + l32;
          if ((cb & 1) == half && tok < a.Lp) srow[tok] = v;
        }
      }
    }
    x += s1 - s0;
    // the next segment overwrites the rows and c in LDS
    __syncthreads();
  }
}

}  // namespace

// Pass 2 on the slab kernel: R = NRB*32-padded rows, NRB <= kSlabMaxNrb;
// per-head subspaces need each head's rows to be whole row blocks (n_part
// 1, upo row blocks per head).
constexpr int kSlabMaxNrb = 14;
int run_pass2_slab(const ScoreArgs& a, int n_layers, int n_cu, hipStream_t st);

}  // namespace starkv
