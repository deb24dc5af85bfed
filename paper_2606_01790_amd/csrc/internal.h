// Internal declarations shared by the host entry points and the kernels'
// launch functions.  Deliberately free of HIP types so that the validation
// unit compiles with a plain C++ compiler.
#pragma once

#include <cstddef>
#include <cstdint>

#include "starkv.h"

namespace starkv {

// Largest window-row block per group kept in LDS by the scoring kernels.
constexpr int kMaxQBytes = 128 * 1024;
// Token chunk of one scoring workgroup: the smallest size sets the
// workspace bound, the launcher may pick larger chunks.
constexpr int kMinChunk = 256;
constexpr int kMaxL = 1 << 26;

struct Geometry {
  int n_layers, H, G, d, L, W, Lp;
  int R;        // window rows of one group, W*H/G
  int Rpad;     // R rounded up to the 32-row MFMA block
  int esz;      // element bytes
  int dtype;
  int Ns;       // scoring subspaces: G, or H when per_head
  int hps;      // query heads per subspace, H / Ns
};

struct WsLayout {
  size_t part_off;   // float2 [n_layers][G][n_chunks_max][Rpad]  row stats
  size_t sraw_off;   // float  [n_layers][Ns][Lp]                 S before pooling
  size_t total;
};

starkv_status check_dims(const starkv_dims* dims, Geometry* g);
starkv_status check_params(const starkv_params* p);
starkv_status check_pool(const starkv_params* p);
starkv_status check_spans(const starkv_span* spans, int32_t n_spans,
                          int32_t frame, int Lp);
starkv_status check_layout(const starkv_kv_layout* lay, const Geometry& g);
bool aligned(const void* p, size_t a);

int max_chunks(const Geometry& g);
WsLayout ws_layout(const Geometry& g);
size_t scalars_count(int G);

// Per-layer state block: a 64-byte header, MI_bar[G] (padded to 16 bytes)
// and m[G][frame_cap], all float32 after the header; the block is padded
// to 256 bytes.
struct StateHeader {
  int32_t magic;      // kStateMagic once initialised
  int32_t G;
  int32_t frame_cap;
  int32_t n;          // compression calls so far in this trajectory
  int32_t nf;         // token count of the frame m_g was built from
  int32_t arrive;     // blocks of the running update that have finished
  int32_t pad[10];
};
constexpr int32_t kStateMagic = 0x53544B56;  // "STKV"
size_t state_stride(int G, int frame_cap);
size_t state_mibar_off();
size_t state_m_off(int G);

// The one span of the current frame (index into spans), or -1.
int current_span(const starkv_span* spans, int32_t n_spans, int32_t frame);

// ---- launch functions (defined with the kernels); stream is a hipStream_t.
// Each returns 0 on success or the HIP error code of the launch.
int launch_score(const Geometry& g, const starkv_params& p, const void* q,
                 const void* k, const starkv_kv_layout& lay, float* S,
                 float* sbar, uint8_t* gstar, void* ws, void* stream);
int launch_update_state(const Geometry& g, const starkv_params& p,
                        const float* S, const float* sbar,
                        const starkv_span* spans, int32_t n_spans,
                        int32_t frame, void* state, int32_t frame_cap,
                        float* scalars, void* stream);
int launch_select(const Geometry& g, const starkv_params& p, const float* sbar,
                  const uint8_t* gstar, const float* scalars,
                  const starkv_span* spans, int32_t n_spans, int32_t frame,
                  int32_t B, float* s, int32_t* idx, void* stream);
// update_state then select in one launch where the statistics run their
// 1024-thread shape (else the two launches).
int launch_update_state_select(const Geometry& g, const starkv_params& p, const float* S,
                               const float* sbar, const uint8_t* gstar,
                               const starkv_span* spans, int32_t n_spans, int32_t frame,
                               void* state, int32_t frame_cap, float* scalars, int32_t B,
                               float* s, int32_t* idx, void* stream);
int launch_compact(const Geometry& g, const void* k, const void* v,
                   const starkv_kv_layout& lay, const int32_t* idx, int32_t B,
                   void* k_out, void* v_out, void* stream);
int launch_state_init(const Geometry& g, void* state, int32_t frame_cap,
                      void* stream);

// Decode attention over a cache of n_tok tokens per (layer, group).
struct DecodeGeometry {
  int n_layers, H, G, d, n_tok;
  int chunk;     // tokens per split block
  int n_split;   // token splits per (layer, group)
};
starkv_status check_decode(const starkv_dims* dims, int32_t n_tokens, DecodeGeometry* g);
size_t decode_ws_bytes(const DecodeGeometry& g);
int launch_decode(const DecodeGeometry& g, const void* q, const void* k, const void* v,
                  const starkv_kv_layout& lay, float* out, void* ws, void* stream);

}  // namespace starkv
