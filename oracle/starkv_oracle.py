"""STaR-KV compression stage, written step by step from the paper in fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Notation follows the paper: H query heads, G KV groups (subspaces), d head
dimension, W observation window, L cache length, L_p = L - W past tokens,
B the historical-token budget.  Tokens, heads and groups are 0-based here.

Section references are to arxiv 2606.01790:
  3.1  Preliminaries (GQA head->group map, token stream, frame distance)
  3.2  STaR-KV overview (Eq. final_score)
  3.3  Base score construction (Eq. A_raw, AvgPool1D, Eq. base_score)
  3.4  Online spatial profiling (Eq. MI, MI EMA, subspace prior, lambda)
  3.5  Cumulative temporal stability discount
  3.6  Adaptive entropy-based sharpening (AEB)
  3.7  Unified selection
  App. Implementation details (hyper-parameters), Algorithm 1 (pipeline).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np


@dataclass
class Params:
    """Hyper-parameters.  Defaults are the paper's (Appendix, implementation
    details and the dataset hyper-parameter table); the ones the paper leaves
    open carry the reading noted beside them."""

    lam: float = 0.5          # target MI prior strength lambda
    n_warmup: int = 5         # online profiling steps before the prior acts
    n_ramp: int = 10          # steps over which lambda_eff ramps up to lambda
    rho_mi: float = 0.9       # MI EMA decay rho
    tau: float = 1.0          # prior softmax temperature
    rho_t: float = 0.9        # stability EMA decay rho_t
    delta: float = 0.2        # temporal decay rate
    d_min: float = 0.1        # discount floor D_min
    t_min: float = 0.75       # AEB T range (UI-TARS single-image setting)
    t_max: float = 1.25
    n_bins: int = 8           # K equal-frequency bins (paper silent; reading)
    grid: int = 8             # M x M spatial grid (paper silent; reading)
    pool_kernel: int = 5      # AvgPool1D width (paper silent; reading)
    eps: float = 1e-8         # the paper's epsilon (value unstated; reading)
    tem_decay: str = "exp"    # TEM decay: "exp" (the paper's), "linear", "gamma"
    aeb_mode: str = "entropy"  # AEB statistic: "entropy" (the paper's), "confidence"


@dataclass
class LayerState:
    """Per-layer online state that persists across the steps of one
    trajectory (sec. 3.2: statistics are online, per layer, O(L) memory;
    reset per trajectory)."""

    G: int
    mi_bar: np.ndarray = field(default=None)   # [G] EMA of MI_g
    m: np.ndarray = field(default=None)        # [G, N_F] EMA of s_g^(c)
    n: int = 0                                 # calls so far (lambda schedule)

    def __post_init__(self):
        if self.mi_bar is None:
            self.mi_bar = np.zeros(self.G, dtype=np.float64)
        if self.m is None:
            self.m = np.zeros((self.G, 0), dtype=np.float64)

    def copy(self) -> "LayerState":
        return LayerState(self.G, self.mi_bar.copy(), self.m.copy(), self.n)


# --------------------------------------------------------------------------
# 3.3 Base score construction
# --------------------------------------------------------------------------

def window_attention_mass(Q: np.ndarray, K_past: np.ndarray) -> np.ndarray:
    """A_raw[h, t] = sum over the W window queries of softmax_t(Q_{-i} K_past^T / sqrt(d)).

    Eq. A_raw (sec. 3.3) with the GQA map of sec. 3.1: query head h reads KV
    group g(h) = floor(h G / H) (0-based form of 1 + floor((h-1) G / H)).
    Reading: the softmax runs over the L_p past keys only, as the equation
    writes it, so each window row sums to 1.

    Q: [H, W, d]; K_past: [G, L_p, d].  Returns [H, L_p] float64.
    """
    Q = np.asarray(Q, dtype=np.float64)
    K_past = np.asarray(K_past, dtype=np.float64)
    H, W, d = Q.shape
    G, L_p, _ = K_past.shape
    A_raw = np.zeros((H, L_p), dtype=np.float64)
    for h in range(H):
        g = (h * G) // H
        X = Q[h] @ K_past[g].T / math.sqrt(d)          # [W, L_p] logits
        X = X - X.max(axis=1, keepdims=True)           # stable softmax
        P = np.exp(X)
        P = P / P.sum(axis=1, keepdims=True)           # row softmax over t
        A_raw[h] = P.sum(axis=0)                       # sum over window i
    return A_raw


def avg_pool1d(A_raw: np.ndarray, k: int) -> np.ndarray:
    """A = AvgPool1D(A_raw) along the token axis (sec. 3.3).

    The paper gives no width or padding.  Reading: odd width k, stride 1,
    zero padding k//2 on both ends, every window divided by k (padding
    counted), so the output keeps length L_p and k = 1 is the identity.
    """
    A_raw = np.asarray(A_raw, dtype=np.float64)
    r = k // 2
    L_p = A_raw.shape[-1]
    padded = np.zeros(A_raw.shape[:-1] + (L_p + 2 * r,), dtype=np.float64)
    padded[..., r:r + L_p] = A_raw
    out = np.zeros_like(A_raw)
    for j in range(k):
        out += padded[..., j:j + L_p]
    return out / k


def group_scores(A: np.ndarray, G: int) -> np.ndarray:
    """S[g, t] = (G/H) * sum of A[h, t] over the H/G heads of group g.

    Eq. base_score (sec. 3.3); Algorithm 1 writes the same mean as
    1/|H_g| sum_{h in H_g}.  Reading of the mixed 1-/0-based bounds: group g
    owns the contiguous heads [g H/G, (g+1) H/G), consistent with g(h).
    """
    H, L_p = A.shape
    hpg = H // G
    S = np.zeros((G, L_p), dtype=np.float64)
    for g in range(G):
        S[g] = A[g * hpg:(g + 1) * hpg].sum(axis=0) * (G / H)
    return S


def per_head_cache(K: np.ndarray, H: int) -> np.ndarray:
    """The MHA-head granularity on a GQA model (sec. 4.2, subspace granularity
    ablation): each shared key (or value) group is replicated across the H/G
    query heads that read it, so the cache has H groups with g(h) = h and
    every head is its own subspace (sec. 3.1: G = H recovers MHA).

    K: [G, L, d] -> [H, L, d], group g's rows repeated for heads
    [g H/G, (g+1) H/G)."""
    G = K.shape[0]
    return np.repeat(np.asarray(K), H // G, axis=0)


def base_score(S: np.ndarray):
    """sbar_t = (1/G) sum_g S[g, t] (Eq. base_score) and the token binding
    g*(t) = argmax_g S[g, t] (sec. 3.4).  Reading: argmax ties go to the
    lowest group index."""
    G = S.shape[0]
    sbar = S.sum(axis=0) / G
    gstar = np.argmax(S, axis=0).astype(np.int64)      # first maximum
    return sbar, gstar


# --------------------------------------------------------------------------
# 3.4 Online spatial profiling
# --------------------------------------------------------------------------

def rank_bins(values: np.ndarray, K: int) -> np.ndarray:
    """Equal-frequency binning ("RankBin", Algorithm 1; sec. 3.4).

    Reading: tokens are ranked by (value ascending, token index ascending)
    and token of rank rho goes to bin floor(rho K / N), so bins hold
    floor(N/K) or ceil(N/K) tokens each.
    """
    values = np.asarray(values, dtype=np.float64)
    N = values.shape[0]
    order = np.lexsort((np.arange(N), values))          # value, then index
    rank = np.empty(N, dtype=np.int64)
    rank[order] = np.arange(N)
    return (rank * K) // N


def spatial_cells(r: np.ndarray, c: np.ndarray, rows: np.ndarray,
                  cols: np.ndarray, M: int) -> np.ndarray:
    """SpatialBin: the token's (row, column) on an M x M grid (sec. 3.4).

    Reading: each frame is mapped onto its own grid,
    cell = floor(r M / rows) * M + floor(c M / cols).
    """
    return (r * M // rows) * M + (c * M // cols)


def plugin_mi(b: np.ndarray, cell: np.ndarray, K: int, C: int) -> float:
    """Plug-in mutual information of the joint histogram (Eq. MI, sec. 3.4):
    MI = sum_{b,(r,c)} p(b,r,c) log[ p(b,r,c) / (p(b) p(r,c)) ], natural log,
    empty cells contribute 0, and an empty token set gives 0."""
    N = b.shape[0]
    if N == 0:
        return 0.0
    joint = np.zeros((K, C), dtype=np.int64)
    np.add.at(joint, (b, cell), 1)
    nb = joint.sum(axis=1)
    nc = joint.sum(axis=0)
    mi = 0.0
    for i in range(K):
        for j in range(C):
            n = joint[i, j]
            if n > 0:
                mi += (n / N) * math.log(n * N / (nb[i] * nc[j]))
    return mi


def mi_prior(mi_bar: np.ndarray, tau: float, eps: float) -> np.ndarray:
    """Subspace prior (sec. 3.4): min-max normalise the MI EMA,
    m~_g = (MI_bar_g - min_j MI_bar_j) / (max_j - min_j + eps), then
    w = softmax(m~ / tau)."""
    lo, hi = mi_bar.min(), mi_bar.max()
    m_tilde = (mi_bar - lo) / (hi - lo + eps)
    z = m_tilde / tau
    e = np.exp(z - z.max())
    return e / e.sum()


def lambda_schedule(n: int, lam: float, n_warmup: int, n_ramp: int) -> float:
    """Annealed prior strength lambda^(t) (sec. 3.4; Appendix).

    Reading: t is the 1-based count n of compression calls of this layer in
    the trajectory; lambda stays 0 for the first n_warmup profiling steps,
    then rises linearly to lam over n_ramp steps (n_ramp = 0: a step).
    """
    if n <= n_warmup:
        return 0.0
    if n_ramp <= 0:
        return lam
    return lam * min(1.0, (n - n_warmup) / n_ramp)


# --------------------------------------------------------------------------
# 3.5 Cumulative temporal stability discount
# --------------------------------------------------------------------------

def stability(s_cur: np.ndarray, m: np.ndarray, rho_t: float, eps: float):
    """phi_g = cos(s_g^(c), m_g), then m_g <- rho_t m_g + (1 - rho_t) s_g^(c)
    (sec. 3.5), phi from the old m as the equations are ordered.

    Reading: s_g^(c) is group g's score row restricted to the newest frame's
    tokens in raster order, so m_g has one entry per grid position; the cosine
    carries eps in its denominator, which makes phi = 0 while m_g is still 0.
    s_cur, m: [G, N_F].  Returns (phi [G], m_new [G, N_F]).
    """
    num = (s_cur * m).sum(axis=1)
    den = np.sqrt((s_cur * s_cur).sum(axis=1)) * np.sqrt((m * m).sum(axis=1)) + eps
    phi = num / den
    m_new = rho_t * m + (1.0 - rho_t) * s_cur
    return phi, m_new


def temporal_discount(is_vis: np.ndarray, frame: np.ndarray, F: int,
                      phi_of_token: np.ndarray, delta: float,
                      d_min: float, decay: str = "exp") -> np.ndarray:
    """D_t = D_min + (1 - D_min) exp(-eta_t), eta_t = delta * Delta_f(t) *
    phi_{g*(t)} for historical visual tokens, D_t = 1 otherwise (sec. 3.5),
    with the frame distance Delta_f(t) = F - f(t) of sec. 3.1.

    The decay ablation (sec. 4.2, temporal weighting functions) compares the
    exponential with a linear and a gamma decay but does not write them out.
    Readings, both with D = 1 at Delta_f = 0 or phi = 0, the floor D_min and
    the exponential's slope at the origin:
      linear: D_min + (1 - D_min) max(0, 1 - eta), reaching the floor at
              eta = 1 (it lies below the exponential: the paper finds it
              discards history too aggressively);
      gamma:  D_min + (1 - D_min) (1 + Delta_f)^(-delta phi), a power law of
              the frame distance (it lies above the exponential: the paper
              finds it keeps more long-range history)."""
    D = np.ones(is_vis.shape[0], dtype=np.float64)
    dist = (F - frame).astype(np.float64)
    eta = delta * dist * phi_of_token
    if decay == "exp":
        f = np.exp(-eta)
    elif decay == "linear":
        f = np.maximum(0.0, 1.0 - eta)
    elif decay == "gamma":
        f = np.power(1.0 + dist, -delta * phi_of_token)
    else:
        raise ValueError(decay)
    D_vis = d_min + (1.0 - d_min) * f
    D[is_vis] = D_vis[is_vis]
    return D


# --------------------------------------------------------------------------
# 3.6 Adaptive entropy-based sharpening
# --------------------------------------------------------------------------

def entropy_temperature(sbar: np.ndarray, t_min: float, t_max: float,
                        eps: float):
    """Normalised entropy of the base distribution and the temperature
    (sec. 3.6; Algorithm 1): p_t = sbar_t / (sum sbar + eps),
    H^ = -sum p_t log(p_t + eps) / log L, T = T_min + (T_max - T_min) H^.

    Reading: the sum and the normaliser run over the L_p scored tokens, and
    H^ is clamped to [0, 1] (eps can push it a hair outside); a single
    token has H^ = 0.
    """
    L_p = sbar.shape[0]
    Z = sbar.sum()
    p = sbar / (Z + eps)
    if L_p <= 1:
        h_hat = 0.0
    else:
        h_hat = float(-(p * np.log(p + eps)).sum() / math.log(L_p))
        h_hat = min(1.0, max(0.0, h_hat))
    T = t_min + (t_max - t_min) * h_hat
    return h_hat, T


def confidence_temperature(sbar: np.ndarray, t_min: float, t_max: float,
                           eps: float):
    """The confidence-based AEB of the ablation (sec. 4.2, entropy- vs
    confidence-based AEB): the temperature comes from the peak mass p_max of
    the base distribution instead of its entropy.  The paper gives no formula;
    reading: p_t = sbar_t / (sum sbar + eps), the confidence
    c = (p_max - 1/L_p) / (1 - 1/L_p) clamped to [0, 1] (0 for a uniform,
    1 for a one-hot distribution; 1 for a single token), and
    T = T_min + (T_max - T_min) (1 - c), so that both ends meet the entropy
    variant's.  Returns (1 - c, T): the statistic in the place of H^."""
    L_p = sbar.shape[0]
    p = sbar / (sbar.sum() + eps)
    if L_p <= 1:
        c = 1.0
    else:
        c = (float(p.max()) - 1.0 / L_p) / (1.0 - 1.0 / L_p)
        c = min(1.0, max(0.0, c))
    u = 1.0 - c
    return u, t_min + (t_max - t_min) * u


def aeb_temperature(sbar: np.ndarray, params: "Params"):
    """The AEB statistic in [0, 1] and T for the configured variant."""
    if params.aeb_mode == "confidence":
        return confidence_temperature(sbar, params.t_min, params.t_max, params.eps)
    if params.aeb_mode != "entropy":
        raise ValueError(params.aeb_mode)
    return entropy_temperature(sbar, params.t_min, params.t_max, params.eps)


# --------------------------------------------------------------------------
# 3.2 final score, 3.7 selection
# --------------------------------------------------------------------------

def final_score(sbar: np.ndarray, beta: np.ndarray, D: np.ndarray,
                T: float) -> tuple[np.ndarray, np.ndarray]:
    """Eq. final_score (sec. 3.2): s^f = sbar * beta * D (D is 1 off the
    visual tokens already), s = max(s^f, 0)^(1/T).  Reading: the power is
    skipped when 1/T is exactly 1, so unit temperature leaves s^f intact."""
    s_f = sbar * beta * D
    inv_t = 1.0 / T
    if inv_t == 1.0:
        return s_f, np.maximum(s_f, 0.0)
    return s_f, np.maximum(s_f, 0.0) ** inv_t


def topb_select(s: np.ndarray, B: int) -> np.ndarray:
    """I = Sort(TopK({s_t}, B)) (sec. 3.7; Algorithm 1): one global set for
    all groups.  Reading: ties at the cut keep the lower token index; the
    result is in ascending token order."""
    L_p = s.shape[0]
    order = np.lexsort((np.arange(L_p), -s))           # s desc, index asc
    return np.sort(order[:B]).astype(np.int64)


def gather_compact(K: np.ndarray, V: np.ndarray, I: np.ndarray, L: int,
                   W: int):
    """K' = [K_past[I]; K_rec], V' = [V_past[I]; V_rec] (sec. 3.7), with the
    W_rec = W most recent tokens kept unconditionally after the selected
    ones.  K, V: [G, >=L, d] (any dtype; rows are copied, not converted)."""
    L_p = L - W
    rec = np.arange(L_p, L)
    sel = np.concatenate([np.asarray(I, dtype=np.int64), rec])
    return K[:, sel], V[:, sel]


# --------------------------------------------------------------------------
# token metadata (sec. 3.1) and the per-layer pipeline (Algorithm 1)
# --------------------------------------------------------------------------

def visual_metadata(spans, L_p: int):
    """Per-token metadata of sec. 3.1 from the visual spans.

    A span is (start, rows, cols, frame): rows*cols visual tokens of one
    frame laid out row-major from token `start`.  Returns is_vis, frame,
    r, c, span_rows, span_cols (each [L_p]); zeros off the visual tokens.
    """
    is_vis = np.zeros(L_p, dtype=bool)
    frame = np.zeros(L_p, dtype=np.int64)
    r = np.zeros(L_p, dtype=np.int64)
    c = np.zeros(L_p, dtype=np.int64)
    rows = np.ones(L_p, dtype=np.int64)
    cols = np.ones(L_p, dtype=np.int64)
    for (start, nr, nc, f) in spans:
        t = np.arange(start, start + nr * nc)
        is_vis[t] = True
        frame[t] = f
        r[t] = (t - start) // nc
        c[t] = (t - start) % nc
        rows[t] = nr
        cols[t] = nc
    return is_vis, frame, r, c, rows, cols


def current_frame_span(spans, F: int):
    """The span of the current frame F, whose scores form the row s_g^(c)
    the stability EMA follows (sec. 3.5); None when no span has frame F."""
    for sp in spans:
        if sp[3] == F:
            return sp
    return None


def compress_layer(Q, K, V, L: int, W: int, spans, F: int, B: int,
                   params: Params, state: LayerState, copy_rows=None):
    """One layer of one trajectory step, in the order of Algorithm 1.

    Q: [H, W, d] window queries; K, V: [G, >=L, d] cache (token order), as
    real values; spans: visual spans inside the L_p past tokens; F: current
    frame; B: budget.  copy_rows: optional (K_rows, V_rows) arrays the compacted
    cache copies its rows from (e.g. the stored bf16 bit patterns); default
    (K, V).  Returns (out, new_state), out holding every intermediate.
    """
    p = params
    Qf = np.asarray(Q, dtype=np.float64)
    Kf = np.asarray(K[:, :L], dtype=np.float64)
    G = Kf.shape[0]
    L_p = L - W
    K_past = Kf[:, :L_p]

    # Base score (sec. 3.3)
    A_raw = window_attention_mass(Qf, K_past)
    A = avg_pool1d(A_raw, p.pool_kernel)
    S = group_scores(A, G)
    sbar, gstar = base_score(S)

    is_vis, frame, r, c, rows, cols = visual_metadata(spans, L_p)
    vis = np.nonzero(is_vis)[0]

    # Online MI prior (sec. 3.4)
    cells = spatial_cells(r[vis], c[vis], rows[vis], cols[vis], p.grid)
    mi = np.zeros(G, dtype=np.float64)
    for g in range(G):
        b = rank_bins(S[g, vis], p.n_bins)
        mi[g] = plugin_mi(b, cells, p.n_bins, p.grid * p.grid)
    mi_bar = p.rho_mi * state.mi_bar + (1.0 - p.rho_mi) * mi
    w = mi_prior(mi_bar, p.tau, p.eps)
    n = state.n + 1
    lam_eff = lambda_schedule(n, p.lam, p.n_warmup, p.n_ramp)
    beta = (1.0 - lam_eff) + lam_eff * G * w[gstar]

    # Temporal stability (sec. 3.5): newest frame's tokens, raster order.
    # Reading: a change of the frame's token count restarts m_g from 0; with
    # no visual span at all there is no current row, phi = 0 and m_g stays.
    span_f = current_frame_span(spans, F)
    if span_f is not None:
        start, nr, nc, _ = span_f
        n_f = nr * nc
        s_cur = S[:, start:start + n_f]
        m_old = state.m if state.m.shape[1] == n_f else np.zeros((G, n_f))
        phi, m_new = stability(s_cur, m_old, p.rho_t, p.eps)
    else:
        phi, m_new = np.zeros(G, dtype=np.float64), state.m.copy()
    D = temporal_discount(is_vis, frame, F, phi[gstar], p.delta, p.d_min, p.tem_decay)

    # AEB (sec. 3.6)
    h_hat, T = aeb_temperature(sbar, p)

    # Fusion and selection (sec. 3.2, 3.7)
    s_f, s = final_score(sbar, beta, D, T)
    I = topb_select(s, B)
    K_rows, V_rows = copy_rows if copy_rows is not None else (K, V)
    K_out, V_out = gather_compact(K_rows, V_rows, I, L, W)

    new_state = LayerState(G, mi_bar, m_new, n)
    out = dict(A_raw=A_raw, A=A, S=S, sbar=sbar, gstar=gstar, mi=mi,
               mi_bar=mi_bar, w=w, lam_eff=lam_eff, beta=beta, phi=phi,
               m=m_new, D=D, h_hat=h_hat, T=T, s_f=s_f, s=s, I=I,
               K_out=K_out, V_out=V_out)
    return out, new_state


# --------------------------------------------------------------------------
# after the stage: decode attention over the (compressed) cache
# --------------------------------------------------------------------------

def decode_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """One decoding step of attention, the cost the compression lowers
    (sec. 4.3, decode-time efficiency): each query head h attends to every
    cached token of its group g(h) = floor(h G / H) (sec. 3.1),
      o[h] = softmax_t(q[h] . K[g(h), t] / sqrt(d)) V[g(h), t].

    q: [H, d]; K, V: [G, n, d] (the compacted K', V' or a full cache).
    Returns o: [H, d] in fp64."""
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    H, d = q.shape
    G = K.shape[0]
    o = np.zeros((H, d), dtype=np.float64)
    for h in range(H):
        g = (h * G) // H
        x = K[g] @ q[h] / math.sqrt(d)
        p = np.exp(x - x.max())
        p /= p.sum()
        o[h] = p @ V[g]
    return o
