// Host driver for the C ABI's validation layer, built with the address and
// undefined-behaviour sanitizers: validate.cpp and api.cpp with the kernel
// launch functions replaced by stubs that record the call.  Every status
// code of starkv.h is produced at least once; the program prints one line
// per check and exits non-zero on the first mismatch.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "internal.h"

namespace starkv {
static int g_launches = 0;
static int g_fail_launch = 0;   // make the next launch report a HIP error
static int stub() { ++g_launches; if (g_fail_launch) { g_fail_launch = 0; return 1; } return 0; }
int launch_score(const Geometry&, const starkv_params&, const void*, const void*,
                 const starkv_kv_layout&, float*, float*, uint8_t*, void*, void*) { return stub(); }
int launch_update_state(const Geometry&, const starkv_params&, const float*, const float*,
                        const starkv_span*, int32_t, int32_t, void*, int32_t, float*, void*) {
  return stub();
}
int launch_select(const Geometry&, const starkv_params&, const float*, const uint8_t*,
                  const float*, const starkv_span*, int32_t, int32_t, int32_t, float*,
                  int32_t*, void*) { return stub(); }
int launch_update_state_select(const Geometry&, const starkv_params&, const float*, const float*,
                               const uint8_t*, const starkv_span*, int32_t, int32_t, void*,
                               int32_t, float*, int32_t, float*, int32_t*, void*) {
  return stub();
}
int launch_compact(const Geometry&, const void*, const void*, const starkv_kv_layout&,
                   const int32_t*, int32_t, void*, void*, void*) { return stub(); }
int launch_state_init(const Geometry&, void*, int32_t, void*) { return stub(); }
int launch_decode(const DecodeGeometry&, const void*, const void*, const void*,
                  const starkv_kv_layout&, float*, void*, void*) { return stub(); }
}  // namespace starkv

using namespace starkv;

static int n_checks = 0;
static void expect(const char* what, int got, int want) {
  ++n_checks;
  if (got != want) {
    std::printf("FAIL %s: got %d want %d\n", what, got, want);
    std::exit(1);
  }
  std::printf("ok %s -> %d\n", what, got);
}

int main() {
  // device-side pointers are never dereferenced on the host: any aligned
  // non-null address stands in for them
  void* P = reinterpret_cast<void*>(0x10000);
  float* F = reinterpret_cast<float*>(0x10000);
  uint8_t* U = reinterpret_cast<uint8_t*>(0x10000);
  int32_t* I = reinterpret_cast<int32_t*>(0x10000);
  void* odd = reinterpret_cast<void*>(0x10002);

  starkv_dims d{28, 28, 4, 128, 13711, 32, STARKV_BF16, 0};
  starkv_params p;
  starkv_params_default(&p);
  starkv_kv_layout lay{4LL * 13711 * 128, 13711LL * 128, 128};
  const size_t ws = starkv_workspace_bytes(&d);
  expect("workspace bytes nonzero", ws > 0, 1);
  const int nf = 69 * 39;
  std::vector<starkv_span> sp;
  for (int f = 0; f < 5; ++f) sp.push_back(starkv_span{f * nf, 39, 69, f + 1});

  // OK paths reach the (stub) launches
  expect("score ok", starkv_score(&d, &p, P, P, &lay, F, F, U, P, ws, nullptr), STARKV_OK);
  expect("update ok", starkv_update_state(&d, &p, F, F, sp.data(), 5, 5, P, nf, F, nullptr, 0,
                                           nullptr), STARKV_OK);
  expect("select ok", starkv_select(&d, &p, F, U, F, sp.data(), 5, 5, 2691, F, I, nullptr, 0,
                                     nullptr), STARKV_OK);
  expect("compact ok", starkv_compact(&d, P, P, &lay, I, 2691, P, P, nullptr), STARKV_OK);
  expect("state init ok", starkv_state_init(&d, P, nf, nullptr), STARKV_OK);
  expect("update+select ok", starkv_update_state_select(&d, &p, F, F, U, sp.data(), 5, 5, P, nf, F,
                                                       2691, F, I, nullptr, 0, nullptr), STARKV_OK);
  expect("launch count", g_launches, 6);

  // E_NULL
  expect("score null q", starkv_score(&d, &p, nullptr, P, &lay, F, F, U, P, ws, nullptr), STARKV_E_NULL);
  expect("score null dims", starkv_score(nullptr, &p, P, P, &lay, F, F, U, P, ws, nullptr), STARKV_E_NULL);
  expect("select null idx", starkv_select(&d, &p, F, U, F, sp.data(), 5, 5, 10, F, nullptr, nullptr,
                                          0, nullptr), STARKV_E_NULL);
  expect("update null spans", starkv_update_state(&d, &p, F, F, nullptr, 5, 5, P, nf, F, nullptr, 0,
                                                  nullptr), STARKV_E_NULL);
  expect("update+select null gstar", starkv_update_state_select(&d, &p, F, F, nullptr, sp.data(), 5, 5,
                                                              P, nf, F, 10, F, I, nullptr, 0, nullptr),
         STARKV_E_NULL);
  expect("update+select null idx", starkv_update_state_select(&d, &p, F, F, U, sp.data(), 5, 5, P, nf,
                                                             F, 10, F, nullptr, nullptr, 0, nullptr),
         STARKV_E_NULL);
  expect("update+select no idx at B = 0", starkv_update_state_select(&d, &p, F, F, U, sp.data(), 5, 5,
                                                                    P, nf, F, 0, F, nullptr, nullptr,
                                                                    0, nullptr), STARKV_OK);
  // E_SHAPE
  starkv_dims bad = d;
  bad.H = 30;
  expect("H not a multiple of G", starkv_score(&bad, &p, P, P, &lay, F, F, U, P, ws, nullptr), STARKV_E_SHAPE);
  bad = d;
  bad.d = 96;
  expect("d = 96", starkv_score(&bad, &p, P, P, &lay, F, F, U, P, ws, nullptr), STARKV_E_SHAPE);
  bad = d;
  bad.W = bad.L;
  expect("W = L", starkv_score(&bad, &p, P, P, &lay, F, F, U, P, ws, nullptr), STARKV_E_SHAPE);
  bad = d;
  bad.G = 65;
  bad.H = 65;
  expect("G > max", starkv_score(&bad, &p, P, P, &lay, F, F, U, P, ws, nullptr), STARKV_E_SHAPE);
  starkv_kv_layout short_tok{lay.layer_stride, lay.group_stride, 64};
  expect("token stride < d", starkv_score(&d, &p, P, P, &short_tok, F, F, U, P, ws, nullptr), STARKV_E_SHAPE);
  // E_BUDGET
  expect("B < 0", starkv_select(&d, &p, F, U, F, sp.data(), 5, 5, -1, F, I, nullptr, 0, nullptr), STARKV_E_BUDGET);
  expect("update+select B > L_p", starkv_update_state_select(&d, &p, F, F, U, sp.data(), 5, 5, P, nf,
                                                            F, 13680, F, I, nullptr, 0, nullptr),
         STARKV_E_BUDGET);
  expect("B > L_p", starkv_compact(&d, P, P, &lay, I, 13680, P, P, nullptr), STARKV_E_BUDGET);
  // E_SPANS
  std::vector<starkv_span> ov = sp;
  ov[1].start -= 1;
  expect("overlapping spans", starkv_update_state(&d, &p, F, F, ov.data(), 5, 5, P, nf, F, nullptr, 0,
                                                  nullptr), STARKV_E_SPANS);
  expect("frame not a span's", starkv_update_state(&d, &p, F, F, sp.data(), 5, 6, P, nf, F, nullptr, 0,
                                                   nullptr), STARKV_E_SPANS);
  std::vector<starkv_span> past = sp;
  past[4].start = 13679 - nf + 1;
  expect("span past L_p", starkv_select(&d, &p, F, U, F, past.data(), 5, 5, 10, F, I, nullptr, 0,
                                        nullptr), STARKV_E_SPANS);
  expect("too many spans", starkv_update_state(&d, &p, F, F, sp.data(), 65, 5, P, nf, F, nullptr, 0,
                                               nullptr), STARKV_E_SPANS);
  expect("update+select span past L_p",
         starkv_update_state_select(&d, &p, F, F, U, past.data(), 5, 5, P, nf, F, 10, F, I, nullptr, 0,
                                    nullptr), STARKV_E_SPANS);
  // E_PARAM
  starkv_params q = p;
  q.lam = 1.5f;
  expect("lambda > 1", starkv_update_state(&d, &q, F, F, sp.data(), 5, 5, P, nf, F, nullptr, 0, nullptr),
         STARKV_E_PARAM);
  q = p;
  q.pool_kernel = 4;
  expect("even pool width", starkv_score(&d, &q, P, P, &lay, F, F, U, P, ws, nullptr), STARKV_E_PARAM);
  q = p;
  q.t_max = 0.5f;
  expect("T_max < T_min", starkv_select(&d, &q, F, U, F, sp.data(), 5, 5, 10, F, I, nullptr, 0, nullptr),
         STARKV_E_PARAM);
  q = p;
  q.grid = 17;
  expect("grid > 16", starkv_update_state(&d, &q, F, F, sp.data(), 5, 5, P, nf, F, nullptr, 0, nullptr),
         STARKV_E_PARAM);
  // E_DTYPE
  bad = d;
  bad.dtype = 7;
  expect("dtype 7", starkv_score(&bad, &p, P, P, &lay, F, F, U, P, ws, nullptr), STARKV_E_DTYPE);
  // E_ALIGN
  expect("q misaligned", starkv_score(&d, &p, odd, P, &lay, F, F, U, P, ws, nullptr), STARKV_E_ALIGN);
  starkv_kv_layout odd_lay{lay.layer_stride, lay.group_stride, 132};
  expect("token stride not 16 B", starkv_compact(&d, P, P, &odd_lay, I, 10, P, P, nullptr), STARKV_E_ALIGN);
  // E_WORKSPACE
  expect("workspace too small", starkv_score(&d, &p, P, P, &lay, F, F, U, P, ws - 1, nullptr),
         STARKV_E_WORKSPACE);
  expect("workspace null", starkv_score(&d, &p, P, P, &lay, F, F, U, nullptr, ws, nullptr),
         STARKV_E_WORKSPACE);
  // E_STATE
  expect("frame above capacity", starkv_update_state(&d, &p, F, F, sp.data(), 5, 5, P, nf - 1, F,
                                                     nullptr, 0, nullptr), STARKV_E_STATE);
  expect("update+select frame above capacity",
         starkv_update_state_select(&d, &p, F, F, U, sp.data(), 5, 5, P, nf - 1, F, 10, F, I, nullptr,
                                    0, nullptr), STARKV_E_STATE);
  expect("negative capacity", starkv_state_init(&d, P, -1, nullptr), STARKV_E_STATE);
  // E_HIP: a launch that reports an error
  g_fail_launch = 1;
  expect("launch error", starkv_compact(&d, P, P, &lay, I, 10, P, P, nullptr), STARKV_E_HIP);
  // decode
  const size_t dws = starkv_decode_workspace_bytes(&d, 2723);
  expect("decode ok", starkv_decode(&d, P, P, P, &lay, 2723, F, P, dws, nullptr), STARKV_OK);
  bad = d;
  bad.dtype = STARKV_F32;
  expect("decode f32", starkv_decode(&bad, P, P, P, &lay, 2723, F, P, dws, nullptr), STARKV_E_DTYPE);
  expect("decode no tokens", starkv_decode(&d, P, P, P, &lay, 0, F, P, dws, nullptr), STARKV_E_SHAPE);
  // status strings and sizes
  for (int s = 0; s <= STARKV_E_HIP; ++s)
    expect("status string", std::strlen(starkv_status_str((starkv_status)s)) > 0, 1);
  expect("state bytes per layer", (int)(starkv_state_bytes(&d, nf) % 256), 0);
  expect("scalars count", (int)starkv_scalars_count(&d), 4 * 4 + 4);
  std::printf("%d checks passed\n", n_checks);
  return 0;
}
