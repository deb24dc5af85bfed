// Gather-compaction (sec. 3.7): K'[g] = [K[g, idx]; K[g, L_p..L)], V' alike.
// A thread moves 16-byte vectors; VPR consecutive threads cover one row, so
// every row read and every row written is a contiguous burst.
#include "device_common.h"
#include "internal.h"

namespace starkv {
namespace {

struct CompactArgs {
  const char* k;
  const char* v;
  char* ko;
  char* vo;
  const int32_t* idx;
  int64_t ls, gs, ts;   // byte strides
  int B, W, Lp, G, rows_out;
  int64_t row_bytes;
};

template <int VPR>
__global__ __launch_bounds__(256) void compact_kernel(CompactArgs a) {
  // each thread moves kPer vectors a block-width apart, their loads all in
  // flight together; the outputs are written once and not read again here,
  // so they bypass the caches
  constexpr int kPer = 4;
  const int g = blockIdx.y, layer = blockIdx.z;
  const int64_t nvec = (int64_t)a.rows_out * VPR;
  const int64_t in_base = (int64_t)layer * a.ls + (int64_t)g * a.gs;
  const int64_t out_base = ((int64_t)layer * a.G + g) * a.rows_out * a.row_bytes;
  const int64_t step = (int64_t)gridDim.x * blockDim.x * kPer;
  for (int64_t v0 = (int64_t)blockIdx.x * blockDim.x * kPer + threadIdx.x; v0 < nvec; v0 += step) {
    i32x4 kv[kPer], vv[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int64_t vec = v0 + (int64_t)j * blockDim.x;
      kv[j] = i32x4{0, 0, 0, 0};
      vv[j] = i32x4{0, 0, 0, 0};
      if (vec < nvec) {
        const int row = (int)(vec / VPR), part = (int)(vec % VPR);
        int src;
        bool ok = true;
        if (row < a.B) {
          src = a.idx[(int64_t)layer * a.B + row];
          ok = src >= 0 && src < a.Lp;
        } else {
          src = a.Lp + (row - a.B);
        }
        if (ok) {
          const int64_t off = in_base + (int64_t)src * a.ts + part * 16;
          kv[j] = *reinterpret_cast<const i32x4*>(a.k + off);
          vv[j] = *reinterpret_cast<const i32x4*>(a.v + off);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int64_t vec = v0 + (int64_t)j * blockDim.x;
      if (vec < nvec) {
        const int row = (int)(vec / VPR), part = (int)(vec % VPR);
        const int64_t o = out_base + (int64_t)row * a.row_bytes + part * 16;
        __builtin_nontemporal_store(kv[j], reinterpret_cast<i32x4*>(a.ko + o));
        __builtin_nontemporal_store(vv[j], reinterpret_cast<i32x4*>(a.vo + o));
      }
    }
  }
}

}  // namespace

int launch_compact(const Geometry& g, const void* k, const void* v,
                   const starkv_kv_layout& lay, const int32_t* idx, int32_t B,
                   void* k_out, void* v_out, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  CompactArgs a;
  a.k = static_cast<const char*>(k);
  a.v = static_cast<const char*>(v);
  a.ko = static_cast<char*>(k_out);
  a.vo = static_cast<char*>(v_out);
  a.idx = idx;
  a.ls = lay.layer_stride * g.esz;
  a.gs = lay.group_stride * g.esz;
  a.ts = lay.token_stride * g.esz;
  a.B = B;
  a.W = g.W;
  a.Lp = g.Lp;
  a.G = g.G;
  a.rows_out = B + g.W;
  a.row_bytes = (int64_t)g.d * g.esz;
  const int vpr = (int)(a.row_bytes / 16);
  const int64_t nvec = (int64_t)a.rows_out * vpr;
  int bx = (int)((nvec + 4 * 256 - 1) / (4 * 256));
  if (bx > 65535) bx = 65535;
  dim3 grid(bx, g.G, g.n_layers);
  switch (vpr) {
    case 8: compact_kernel<8><<<grid, 256, 0, st>>>(a); break;
    case 16: compact_kernel<16><<<grid, 256, 0, st>>>(a); break;
    default: compact_kernel<32><<<grid, 256, 0, st>>>(a); break;
  }
  return (int)hipGetLastError();
}

}  // namespace starkv
