// Device-side helpers shared by the gfx950 kernels: MFMA fragment access,
// wavefront/block reductions and order-preserving float keys.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace starkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// 32x32 MFMA tiles.  For v_mfma_f32_32x32x16_bf16 / _32x32x2f32, lane l
// supplies row (l % 32) of A and column (l % 32) of B with the k-slice of
// half h = l / 32, and receives the 16 accumulators
//   acc[4*i + j]  at  row 8*i + 4*h + j,  column l % 32   (i, j in 0..3).
template <typename T>
struct Mfma;

template <>
struct Mfma<__bf16> {
  using frag = bf16x8;
  static constexpr int kStep = 16;   // k elements per instruction
  // 8 consecutive elements of a row: k = kk*16 + half*8 .. +8
  __device__ static inline frag load(const __bf16* row, int kk, int half) {
    return *reinterpret_cast<const frag*>(row + kk * 16 + half * 8);
  }
  __device__ static inline f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

template <>
struct Mfma<float> {
  using frag = float;
  static constexpr int kStep = 2;
  __device__ static inline frag load(const float* row, int kk, int half) {
    return row[kk * 2 + half];
  }
  __device__ static inline f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

__device__ inline double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Deterministic block-wide sum of doubles (fixed combination order).
// `red` must hold blockDim.x / 64 doubles.  All threads get the result.
__device__ inline double block_sum_d(double v, double* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  v = wave_sum_d(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  double t = 0.0;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

// Order-preserving map of float bits to uint32 (larger float -> larger key).
__device__ inline uint32_t fkey(float x) {
  uint32_t b = __float_as_uint(x);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Exclusive prefix count of a per-thread flag over the block, in thread
// order, plus the block total.  `sh` holds blockDim.x / 64 ints.
__device__ inline int block_excl_count(bool flag, int* sh, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const uint64_t mask = __ballot(flag);
  const int in_wave = __popcll(mask & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
  __syncthreads();
  if (lane == 0) sh[w] = __popcll(mask);
  __syncthreads();
  int before = 0, tot = 0;
  for (int i = 0; i < nw; ++i) {
    const int c = sh[i];
    if (i < w) before += c;
    tot += c;
  }
  *total = tot;
  return before + in_wave;
}


// Inclusive prefix sum of an int across the 64 lanes of a wave.
__device__ inline int wave_incl_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(v, o);
    if (lane >= o) v += t;
  }
  return v;
}

__device__ inline uint32_t wave_min_u32(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = min(v, (uint32_t)__shfl_xor((int)v, o));
  return v;
}

__device__ inline uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o));
  return v;
}

// Exclusive prefix sum of an int over the block in thread order; all threads
// get the block total.  `sh` holds blockDim.x / 64 ints.
__device__ inline int block_excl_scan(int v, int* sh, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const int inc = wave_incl_scan(v);
  __syncthreads();
  if (lane == 63) sh[w] = inc;
  __syncthreads();
  int before = 0, tot = 0;
  for (int i = 0; i < nw; ++i) {
    const int c = sh[i];
    if (i < w) before += c;
    tot += c;
  }
  *total = tot;
  return before + inc - v;
}

// One wave: in the histogram h[0..nb) (nb <= 256), the bin d whose running
// count range [before, before + h[d]) contains `rank` (rank < sum of h).
__device__ inline void wave_find_bin(const int* h, int nb, int rank, int* d_out,
                                     int* before_out, int* cnt_out) {
  const int lane = threadIdx.x & 63;
  int c[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) c[j] = (4 * lane + j < nb) ? h[4 * lane + j] : 0;
  const int sum = c[0] + c[1] + c[2] + c[3];
  const int inc = wave_incl_scan(sum);
  const int exc = inc - sum;
  const uint64_t hit = __ballot(exc <= rank && rank < inc);
  const int src = hit ? __ffsll((unsigned long long)hit) - 1 : 0;
  int d = 0, before = 0, cnt = 0;
  if (lane == src) {
    int run = exc;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (rank < run + c[j]) { d = 4 * lane + j; before = run; cnt = c[j]; break; }
      run += c[j];
    }
  }
  *d_out = __shfl(d, src);
  *before_out = __shfl(before, src);
  *cnt_out = __shfl(cnt, src);
}

// Bits [shift, 32) of a key, with shift = 32 giving 0.
__device__ inline uint32_t key_hi(uint32_t k, int shift) {
  return shift >= 32 ? 0u : (k >> shift);
}

}  // namespace starkv
