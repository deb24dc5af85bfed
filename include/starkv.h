/*
 * starkv.h -- C ABI of the STaR-KV compression stage on MI355X (gfx950).
 *
 * STaR-KV (arxiv 2606.01790) compresses each layer's KV cache at prefill.
 * It scores the cached tokens from a window of recent queries and
 * re-weights the score with a spatial mutual-information prior, a temporal
 * stability discount and an entropy-derived temperature.  It then keeps the
 * top-B tokens plus the recent window (sections 3.2-3.7, Algorithm 1).
 *
 * The stage is split into four calls, in pipeline order:
 *   starkv_score        window attention mass, pooling, group mean     (3.3)
 *   starkv_update_state spatial MI prior, stability, entropy, T        (3.4-3.6)
 *   starkv_select       fused final score and global top-B             (3.2, 3.7)
 *   starkv_compact      gather of the kept K/V rows plus the window    (3.7)
 *
 * Conventions shared by every call:
 *  - Every call handles `n_layers` independent layers (sec. 3.7: all
 *    modules operate per layer) and returns before the GPU work finishes.
 *    The work is queued on `stream` (a hipStream_t; NULL is the default
 *    stream).  No call synchronises, copies to the host or allocates memory.
 *  - Pointers named as device pointers must be device memory.  Host
 *    pointers (dims, params, layouts, spans) are read only during the call.
 *  - The caller owns every buffer.  The library keeps no pointer after a
 *    call returns and has no global mutable state, except the device array
 *    behind starkv_score_noalloc (see there).
 *  - All arguments are validated on the host before any GPU work is queued.
 *    On any error code nothing is written and nothing is launched.
 *  - Tokens are 0-based.  L is the cache length of the step, W the
 *    observation window (the W most recent tokens, which are also the
 *    recent window kept outside the budget), and L_p = L - W the past
 *    tokens that are scored and selected.
 *  - Results are bitwise deterministic for identical inputs on one device.
 */
#ifndef STARKV_H
#define STARKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define STARKV_ABI_VERSION 2
#define STARKV_MAX_SPANS 64   /* visual spans per call */
#define STARKV_MAX_GROUPS 64  /* KV groups G, and scoring subspaces */

typedef enum starkv_status {
  STARKV_OK = 0,
  STARKV_E_NULL = 1,      /* a required pointer is NULL */
  STARKV_E_SHAPE = 2,     /* inconsistent or unsupported dims/layout */
  STARKV_E_BUDGET = 3,    /* B < 0 or B > L_p */
  STARKV_E_SPANS = 4,     /* visual spans malformed (see starkv_span) */
  STARKV_E_PARAM = 5,     /* a hyper-parameter out of range */
  STARKV_E_DTYPE = 6,     /* unknown element type */
  STARKV_E_ALIGN = 7,     /* a pointer or stride breaks 16-byte alignment */
  STARKV_E_WORKSPACE = 8, /* workspace NULL or smaller than required */
  STARKV_E_STATE = 9,     /* state capacity too small for the frame */
  STARKV_E_HIP = 10       /* the HIP runtime reported a launch error */
} starkv_status;

typedef enum starkv_dtype {
  STARKV_F32 = 0,   /* float32 Q/K/V */
  STARKV_BF16 = 1   /* bfloat16 Q/K/V */
} starkv_dtype;

/* Problem dimensions of one call.  GQA as in sec. 3.1: H query heads share
 * G KV groups, query head h reads group floor(h*G/H).  Requirements:
 * n_layers >= 1; G >= 1, G <= STARKV_MAX_GROUPS, H % G == 0; d in {64, 128};
 * 1 <= W < L; L <= 2^26; the window rows of one group, R = W*H/G, must
 * satisfy R <= 512 and R*(d*elem_bytes + 16) <= 128 KiB (R rounded up to 32);
 * for STARKV_F32, R <= 128.
 *
 * Subspaces (sec. 3.1; granularity ablation in sec. 4.2): the unit that
 * gets its own score row, MI prior, stability mean and g* candidate.
 *   per_head = 0: one subspace per KV group, Ns = G (the GQA default);
 *   per_head = 1: one subspace per query head, Ns = H, the heads of a group
 *                 all reading that group's shared K (the paper's MHA-head
 *                 granularity on a GQA model: K/V replicated across the heads
 *                 of the group, here without copying them).  Requires
 *                 H <= STARKV_MAX_GROUPS and W % 8 == 0.
 * Under MHA (G == H) both settings give the same subspaces.  Every buffer
 * documented below as per subspace has Ns rows. */
typedef struct starkv_dims {
  int32_t n_layers;
  int32_t H;
  int32_t G;
  int32_t d;
  int32_t L;
  int32_t W;
  int32_t dtype;    /* starkv_dtype of q, k and v */
  int32_t per_head; /* 0: Ns = G subspaces (default), 1: Ns = H */
} starkv_dims;

/* Element strides of a K or V cache.  Element (layer, group, token, j) is
 * at base + layer*layer_stride + group*group_stride + token*token_stride
 * + j, with the d elements of a token contiguous.  Every stride times the
 * element size must be a multiple of 16 bytes.  Tokens [0, L) of every
 * (layer, group) must be addressable. */
typedef struct starkv_kv_layout {
  int64_t layer_stride;
  int64_t group_stride;
  int64_t token_stride;
} starkv_kv_layout;

/* Hyper-parameters (Appendix, implementation details and the dataset
 * hyper-parameter table).  starkv_params_default() fills the paper's values.
 * Where the paper is silent (n_bins, grid, pool_kernel, eps) it fills the
 * readings given beside each field. */
typedef struct starkv_params {
  float lam;          /* target MI prior strength lambda, [0, 1]          (0.5) */
  int32_t n_warmup;   /* profiling steps with lambda_eff = 0, >= 0          (5) */
  int32_t n_ramp;     /* steps of the linear lambda ramp, >= 0             (10) */
  float rho_mi;       /* MI EMA decay rho, [0, 1)                           (0.9) */
  float tau;          /* prior softmax temperature, > 0                     (1.0) */
  float rho_t;        /* stability EMA decay rho_t, [0, 1)                  (0.9) */
  float delta;        /* temporal decay rate, >= 0                          (0.2) */
  float d_min;        /* discount floor D_min, [0, 1]                       (0.1) */
  float t_min;        /* AEB temperature range, 0 < t_min <= t_max   (0.75, 1.25) */
  float t_max;
  int32_t n_bins;     /* K equal-frequency bins, [1, 64]                      (8) */
  int32_t grid;       /* M x M spatial grid, [1, 16]                          (8) */
  int32_t pool_kernel;/* odd AvgPool1D width, [1, 63]                         (5) */
  float eps;          /* the paper's epsilon, >= 0                         (1e-8) */
  /* Ablation variants (sec. 4.2); the paper does not write their formulas,
   * the readings are given with the enums. */
  int32_t tem_decay;  /* starkv_tem_decay of the temporal discount  (EXP) */
  int32_t aeb_mode;   /* starkv_aeb_mode of the AEB temperature  (ENTROPY) */
} starkv_params;

/* Temporal discount D_t of historical visual tokens (sec. 3.5), with
 * eta = delta * (F - f(t)) * phi_{g*(t)}:
 *   EXP     D_min + (1 - D_min) exp(-eta)                 (the paper's)
 *   LINEAR  D_min + (1 - D_min) max(0, 1 - eta)
 *   GAMMA   D_min + (1 - D_min) (1 + F - f(t))^(-delta * phi_{g*(t)})
 * All three are 1 at distance 0 or phi = 0, floor at D_min and share the
 * exponential's slope at distance 0; linear lies below it, gamma above. */
typedef enum starkv_tem_decay {
  STARKV_TEM_EXP = 0,
  STARKV_TEM_LINEAR = 1,
  STARKV_TEM_GAMMA = 2
} starkv_tem_decay;

/* Statistic u in [0, 1] behind the AEB temperature T = t_min + (t_max -
 * t_min) u (sec. 3.6), with p = sbar / (sum sbar + eps) over the L_p tokens:
 *   ENTROPY     u = H^ = -sum p ln(p + eps) / ln L_p, clamped   (the paper's)
 *   CONFIDENCE  u = 1 - c, c = (max p - 1/L_p) / (1 - 1/L_p) clamped to
 *               [0, 1] (c = 1 for L_p = 1): the peak-mass variant. */
typedef enum starkv_aeb_mode {
  STARKV_AEB_ENTROPY = 0,
  STARKV_AEB_CONFIDENCE = 1
} starkv_aeb_mode;

/* A visual span (sec. 3.1): rows*cols visual tokens of one screenshot, laid
 * out row-major from token `start` (token start + r*cols + c has screen
 * coordinate (r, c)).  Spans of one call must lie inside [0, L_p), be sorted
 * by start, not overlap, and carry distinct frame indices <= the current
 * frame.  Tokens outside every span are non-visual. */
typedef struct starkv_span {
  int32_t start;
  int32_t rows;
  int32_t cols;
  int32_t frame;
} starkv_span;

/* Per-layer scalar block written by starkv_update_state and read by
 * starkv_select: float32 array [n_layers][starkv_scalars_count(dims)].
 * Within one layer, for the Ns subspaces (written G here):
 *   [0, G)     MI_g of this step                  (Eq. MI)
 *   [G, 2G)    MI_bar_g after the EMA update
 *   [2G, 3G)   prior weights w_g                  (sec. 3.4)
 *   [3G, 4G)   stability phi_g                    (sec. 3.5)
 *   4G         lambda_eff of this step
 *   4G+1       AEB statistic u: H^, or 1 - c      (sec. 3.6, starkv_aeb_mode)
 *   4G+2       temperature T
 *   4G+3       step count n (as a float)                                    */
#define STARKV_SCAL_MI(G) 0
#define STARKV_SCAL_MIBAR(G) (G)
#define STARKV_SCAL_W(G) (2 * (G))
#define STARKV_SCAL_PHI(G) (3 * (G))
#define STARKV_SCAL_LAMBDA(G) (4 * (G))
#define STARKV_SCAL_HHAT(G) (4 * (G) + 1)
#define STARKV_SCAL_T(G) (4 * (G) + 2)
#define STARKV_SCAL_N(G) (4 * (G) + 3)

/* ------------------------------------------------------------------ */
/* helpers (host only, no GPU work)                                   */
/* ------------------------------------------------------------------ */

int32_t starkv_abi_version(void);
const char* starkv_status_str(starkv_status status);
void starkv_params_default(starkv_params* params);

/* Bytes of device workspace any call with these dims (at this L or a
 * smaller one) needs.  0 if dims are invalid. */
size_t starkv_workspace_bytes(const starkv_dims* dims);

/* Floats per layer of the scalar block. */
size_t starkv_scalars_count(const starkv_dims* dims);

/* Bytes of the per-layer online state for all n_layers (sec. 3.2: O(L)
 * per-layer statistics kept across the steps of one trajectory).  The state
 * holds MI_bar and the stability mean m_g of every subspace (m_g: one entry
 * per token of the current frame, up to frame_cap) and the step count.  It is a plain device
 * block the caller may copy out and back to checkpoint a trajectory. */
size_t starkv_state_bytes(const starkv_dims* dims, int32_t frame_cap);

/* Start a trajectory: zero EMAs, step count 0 (the reset per trajectory of
 * the appendix).  state: device, starkv_state_bytes(dims, frame_cap). */
starkv_status starkv_state_init(const starkv_dims* dims, void* state,
                                int32_t frame_cap, void* stream);

/* ------------------------------------------------------------------ */
/* the compression stage                                               */
/* ------------------------------------------------------------------ */

/* Window attention scoring (sec. 3.3, Eq. A_raw and Eq. base_score;
 * Algorithm 1, base-score lines).  For each layer and subspace g:
 *   A_raw[h,t] = sum_{i<W} softmax_t(Q[h,i] . K[g(h),t] / sqrt(d)), t < L_p,
 *   A = AvgPool1D(A_raw) (odd width, zero padding, divide by the width),
 *   S[g,t] = mean of A[h,t] over the heads of subspace g (the heads of KV
 *            group g, or head g alone when dims->per_head),
 *   sbar[t] = mean_g S[g,t],  gstar[t] = argmax_g S[g,t] (lowest g on ties).
 * q:     device, [n_layers][H][W][d] contiguous, dims->dtype.  Row i is the
 *        query of token L - W + i.
 * k:     device cache with layout *k_layout, dims->dtype (G KV groups).
 * S:     device out, float32 [n_layers][Ns][L_p].
 * sbar:  device out, float32 [n_layers][L_p].
 * gstar: device out, uint8 [n_layers][L_p].
 * ws:    device workspace of ws_bytes >= starkv_workspace_bytes(dims).
 * Errors: E_NULL, E_SHAPE, E_DTYPE, E_ALIGN, E_PARAM (pool_kernel),
 * E_WORKSPACE, E_HIP. */
starkv_status starkv_score(const starkv_dims* dims, const starkv_params* params,
                           const void* q, const void* k,
                           const starkv_kv_layout* k_layout,
                           float* S, float* sbar, uint8_t* gstar,
                           void* ws, size_t ws_bytes, void* stream);

/* starkv_score for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, computation and results as starkv_score, without ws: the
 * workspace is a library-owned device array of STARKV_NOALLOC_SCRATCH_BYTES
 * that every GPU the library runs on holds from module load until the
 * process ends (one copy per device).  The call allocates nothing; its
 * first call on a device looks up that device's copy (no allocation).
 * Calls that overlap on one GPU (other streams, other host threads) share
 * the array and race: order them, or use starkv_score with separate
 * workspaces.  The array keeps the last call's contents; the call needs no
 * clearing of it.
 * Errors: as starkv_score, with E_WORKSPACE when
 * starkv_workspace_bytes(dims) > STARKV_NOALLOC_SCRATCH_BYTES. */
#define STARKV_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
starkv_status starkv_score_noalloc(const starkv_dims* dims,
                                   const starkv_params* params,
                                   const void* q, const void* k,
                                   const starkv_kv_layout* k_layout,
                                   float* S, float* sbar, uint8_t* gstar,
                                   void* stream);

/* Online statistics of one step (sec. 3.4 online MI prior, sec. 3.5
 * stability, sec. 3.6 entropy and temperature; Algorithm 1, MI and AEB
 * lines).  Per layer:
 *   MI_g    = plug-in MI between RankBin(S[g, visual]) (n_bins equal-frequency
 *             bins, ranks by value then token index) and SpatialBin(visual)
 *             (each frame's rows x cols mapped onto a grid x grid raster);
 *   MI_bar  = rho_mi * MI_bar + (1 - rho_mi) * MI;
 *   w       = softmax(minmax(MI_bar) / tau);
 *   n += 1, lambda_eff = 0 for n <= n_warmup, then lam*min(1,(n-n_warmup)/n_ramp);
 *   phi_g   = cos(S[g, current frame], m_g) (eps in the denominator), then
 *             m_g = rho_t*m_g + (1-rho_t)*S[g, current frame]; m_g restarts
 *             from 0 when the current frame's token count changes;
 *   H^      = clamp(-sum p ln(p+eps) / ln L_p, 0, 1), p = sbar/(sum sbar + eps)
 *             (or the params->aeb_mode variant, see starkv_aeb_mode);
 *   T       = t_min + (t_max - t_min) * H^.
 * S, sbar: device, as written by starkv_score.
 * spans:   host, n_spans in [0, STARKV_MAX_SPANS]; frame: the current
 *          frame F (must be a span's frame when n_spans > 0).
 * state:   device, from starkv_state_init with the same dims and frame_cap;
 *          the current frame's rows*cols must be <= frame_cap (E_STATE).
 *          The state lives in device memory, so the host cannot check it: a
 *          layer whose state block was not initialised for the same
 *          subspace count and frame_cap is left untouched and gets NaN in
 *          all of its scalars.  (A frame_cap above the one the buffer was
 *          sized for addresses memory past the buffer; it is the caller's
 *          to match the allocation.)
 * scalars: device out, float32 [n_layers][starkv_scalars_count(dims)].
 * ws, ws_bytes: unused (reserved); may be NULL and 0.
 * Every per-group quantity above is per subspace (Ns of them).
 * Errors: E_NULL, E_SHAPE, E_SPANS, E_PARAM, E_STATE, E_ALIGN, E_HIP. */
starkv_status starkv_update_state(const starkv_dims* dims,
                                  const starkv_params* params,
                                  const float* S, const float* sbar,
                                  const starkv_span* spans, int32_t n_spans,
                                  int32_t frame, void* state, int32_t frame_cap,
                                  float* scalars, void* ws, size_t ws_bytes,
                                  void* stream);

/* Final score and global top-B (Eq. final_score in sec. 3.2, sec. 3.5
 * discount, sec. 3.7 selection; Algorithm 1, fusion and selection lines):
 *   beta_t = (1 - lambda_eff) + lambda_eff * Ns * w[gstar_t],
 *   D_t    = d_min + (1 - d_min) exp(-delta (F - f(t)) phi[gstar_t]) on visual
 *            tokens (or the params->tem_decay variant), 1 elsewhere,
 *   s_t    = max(sbar_t beta_t D_t, 0)^(1/T) (no power when 1/T == 1),
 *   idx    = the B tokens of largest s (lower index first on ties), ascending.
 * sbar, gstar: device, from starkv_score; scalars: device, from
 * starkv_update_state; spans/frame as for starkv_update_state.
 * s:   device out, float32 [n_layers][L_p].
 * idx: device out, int32 [n_layers][B] (may be NULL when B == 0).
 * ws, ws_bytes: unused (reserved); may be NULL and 0.
 * Errors: E_NULL, E_SHAPE, E_BUDGET, E_SPANS, E_PARAM, E_ALIGN, E_HIP. */
starkv_status starkv_select(const starkv_dims* dims, const starkv_params* params,
                            const float* sbar, const uint8_t* gstar,
                            const float* scalars,
                            const starkv_span* spans, int32_t n_spans,
                            int32_t frame, int32_t B, float* s, int32_t* idx,
                            void* ws, size_t ws_bytes, void* stream);

/* starkv_update_state followed by starkv_select, in one call (sec. 3.4-3.6,
 * then sec. 3.2 and 3.7; Algorithm 1, from the statistics through the
 * selection line): the arguments of both, with the same meaning, layout,
 * ownership and errors; the outputs (scalars, state, s, idx) are bit for bit
 * those of the two calls in a row.  Where the statistics run one block per
 * CU, the block that finishes a layer's statistics runs that layer's
 * selection next, so the selection needs no launch of its own; otherwise
 * the two launches are queued.
 * ws, ws_bytes: unused (reserved); may be NULL and 0.
 * Errors: E_NULL, E_SHAPE, E_BUDGET, E_SPANS, E_PARAM, E_STATE, E_ALIGN,
 * E_HIP. */
starkv_status starkv_update_state_select(const starkv_dims* dims,
                                         const starkv_params* params, const float* S,
                                         const float* sbar, const uint8_t* gstar,
                                         const starkv_span* spans, int32_t n_spans,
                                         int32_t frame, void* state, int32_t frame_cap,
                                         float* scalars, int32_t B, float* s, int32_t* idx,
                                         void* ws, size_t ws_bytes, void* stream);

/* Gather-compaction (sec. 3.7; Algorithm 1, return line), over the G KV
 * groups whatever the subspaces:
 *   K'[g] = [K[g, idx[0..B)]; K[g, L_p..L)],  V' likewise.
 * k, v:   device caches with layout *kv_layout (both use it), dims->dtype.
 * idx:    device, int32 [n_layers][B], every entry in [0, L_p); ascending
 *         order is what starkv_select writes but is not required.  The
 *         kernel never reads outside the cache: an entry outside [0, L_p)
 *         (a caller bug) produces an all-zero row in K' and V' instead of a
 *         copy, so check idx before relying on rows that come out zero.
 * k_out, v_out: device out, [n_layers][G][B + W][d] contiguous, bit copies.
 * Outputs must not overlap the inputs.
 * Errors: E_NULL, E_SHAPE, E_DTYPE, E_ALIGN, E_BUDGET, E_HIP. */
starkv_status starkv_compact(const starkv_dims* dims, const void* k,
                             const void* v, const starkv_kv_layout* kv_layout,
                             const int32_t* idx, int32_t B, void* k_out,
                             void* v_out, void* stream);

/* ------------------------------------------------------------------ */
/* after the stage: decode attention over the compressed cache          */
/* ------------------------------------------------------------------ */

/* Bytes of device workspace starkv_decode needs for these dims and token
 * count.  0 if they are invalid for it. */
size_t starkv_decode_workspace_bytes(const starkv_dims* dims, int32_t n_tokens);

/* Decode attention of one new token per query head over a cache of n_tokens
 * tokens per (layer, KV group), the step whose cost the compression lowers
 * (sec. 4.3, decode-time efficiency; sec. 3.1 for the GQA map):
 *   o[h] = sum_{t < n_tokens} softmax_t(q[h] . K[g(h),t] / sqrt(d)) V[g(h),t].
 * Run on K'/V' from starkv_compact (n_tokens = B + W, layout layer_stride =
 * G*(B+W)*d, group_stride = (B+W)*d, token_stride = d) it is decoding with
 * the compressed cache; run on the full cache (n_tokens = L) it is the
 * uncompressed baseline.  Only n_layers, H, G, d and dtype of dims are read:
 * STARKV_BF16 only (E_DTYPE otherwise), H/G <= 16, d in {64, 128},
 * 1 <= n_tokens <= 2^26.
 * q:      device, bf16 [n_layers][H][d] contiguous.
 * k, v:   device bf16 caches with layout *kv_layout (both use it).
 * out:    device out, float32 [n_layers][H][d].
 * ws:     device workspace of ws_bytes >= starkv_decode_workspace_bytes().
 * Softmax and accumulation are fp32; the result does not depend on the
 * launch split beyond the fixed order of its partial sums, and is bitwise
 * deterministic.  Errors: E_NULL, E_SHAPE, E_DTYPE, E_ALIGN, E_WORKSPACE,
 * E_HIP. */
starkv_status starkv_decode(const starkv_dims* dims, const void* q, const void* k,
                            const void* v, const starkv_kv_layout* kv_layout,
                            int32_t n_tokens, float* out, void* ws, size_t ws_bytes,
                            void* stream);

#ifdef __cplusplus
}
#endif

#endif /* STARKV_H */
