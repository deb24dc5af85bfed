"""Planted mistakes in the oracle, each of which some pin must catch.

Every case replaces one oracle function with a plausible wrong version (a
dropped term, a wrong sign or index, a transposed operand, an off-by-one)
and runs the pins of tests/test_oracle_pins.py that cover that function:
at least one of them must fail.  This checks the pins, not the oracle, so it
runs on the CPU only and touches nothing on the GPU path.
"""

import math

import numpy as np
import pytest

import test_oracle_pins as P
from oracle import starkv_oracle as O

ORIG = {name: getattr(O, name) for name in dir(O) if callable(getattr(O, name))}


def _wam(scale=True, axis=1, gmap=None, transpose=False):
    def f(Q, K_past):
        Q = np.asarray(Q, dtype=np.float64)
        K_past = np.asarray(K_past, dtype=np.float64)
        H, W, d = Q.shape
        G, L_p, _ = K_past.shape
        A = np.zeros((H, L_p))
        for h in range(H):
            g = gmap(h, H, G) if gmap else (h * G) // H
            X = Q[h] @ K_past[g].T
            if scale:
                X = X / math.sqrt(d)
            if transpose:      # softmax over the window queries instead of the keys
                X = X - X.max(axis=0, keepdims=True)
                P_ = np.exp(X)
                P_ = P_ / P_.sum(axis=0, keepdims=True)
            else:
                X = X - X.max(axis=1, keepdims=True)
                P_ = np.exp(X)
                P_ = P_ / P_.sum(axis=axis, keepdims=True)
            A[h] = P_.sum(axis=0)
        return A
    return f


def _pool_valid_count(A_raw, k):
    A_raw = np.asarray(A_raw, dtype=np.float64)
    r = k // 2
    L_p = A_raw.shape[-1]
    pad = np.zeros(A_raw.shape[:-1] + (L_p + 2 * r,))
    pad[..., r:r + L_p] = A_raw
    ones = np.zeros(L_p + 2 * r)
    ones[r:r + L_p] = 1
    out = sum(pad[..., j:j + L_p] for j in range(k))
    cnt = sum(ones[j:j + L_p] for j in range(k))
    return out / cnt


def _pool_shifted(A_raw, k):
    out = ORIG["avg_pool1d"](A_raw, k)
    return np.roll(out, 1, axis=-1)


def _group_sum(A, G):
    H, L_p = A.shape
    hpg = H // G
    return np.stack([A[g * hpg:(g + 1) * hpg].sum(axis=0) for g in range(G)])


def _group_interleaved(A, G):
    H, L_p = A.shape
    return np.stack([A[g::G].mean(axis=0) for g in range(G)])


def _base_last_max(S):
    G = S.shape[0]
    sbar = S.sum(axis=0) / G
    gstar = (G - 1 - np.argmax(S[::-1], axis=0)).astype(np.int64)
    return sbar, gstar


def _rank_index_desc(values, K):
    values = np.asarray(values, dtype=np.float64)
    N = values.shape[0]
    order = np.lexsort((-np.arange(N), values))
    rank = np.empty(N, dtype=np.int64)
    rank[order] = np.arange(N)
    return (rank * K) // N


def _rank_ceil(values, K):
    values = np.asarray(values, dtype=np.float64)
    N = values.shape[0]
    order = np.lexsort((np.arange(N), values))
    rank = np.empty(N, dtype=np.int64)
    rank[order] = np.arange(N)
    return np.minimum(-((-rank * K) // N), K - 1)


def _mi_log2(b, cell, K, C):
    return ORIG["plugin_mi"](b, cell, K, C) / math.log(2)


def _mi_swapped_marginals(b, cell, K, C):
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
            if n > 0:   # each cell's count paired with the next bin's total
                mi += (n / N) * math.log(n * N / (nb[(i + 1) % K] * nc[j]))
    return mi


def _cells_swapped(r, c, rows, cols, M):
    return (r * M // cols) * M + (c * M // rows)


def _metadata(transpose_shape=False, column_major=False):
    def f(spans, L_p):
        is_vis = np.zeros(L_p, dtype=bool)
        frame = np.zeros(L_p, dtype=np.int64)
        r = np.zeros(L_p, dtype=np.int64)
        c = np.zeros(L_p, dtype=np.int64)
        rows = np.ones(L_p, dtype=np.int64)
        cols = np.ones(L_p, dtype=np.int64)
        for (start, nr, nc, fr) in spans:
            if transpose_shape:      # the span's rows and columns swapped
                nr, nc = nc, nr
            t = np.arange(start, start + nr * nc)
            is_vis[t] = True
            frame[t] = fr
            if column_major:         # raster walks down the columns
                r[t] = (t - start) % nr
                c[t] = (t - start) // nr
            else:
                r[t] = (t - start) // nc
                c[t] = (t - start) % nc
            rows[t] = nr
            cols[t] = nc
        return is_vis, frame, r, c, rows, cols
    return f


def _first_span(spans, F):
    return spans[0] if spans else None


def _prior_raw(mi_bar, tau, eps):
    z = mi_bar / tau
    e = np.exp(z - z.max())
    return e / e.sum()


def _prior_negated(mi_bar, tau, eps):
    return ORIG["mi_prior"](-mi_bar, tau, eps)


def _lambda_early(n, lam, n_warmup, n_ramp):
    if n < n_warmup:
        return 0.0
    if n_ramp <= 0:
        return lam
    return lam * min(1.0, (n - n_warmup + 1) / n_ramp)


def _stability_new_mean(s_cur, m, rho_t, eps):
    m_new = rho_t * m + (1.0 - rho_t) * s_cur
    num = (s_cur * m_new).sum(axis=1)
    den = np.sqrt((s_cur ** 2).sum(axis=1)) * np.sqrt((m_new ** 2).sum(axis=1)) + eps
    return num / den, m_new


def _mi_ema_swapped(Q, K, V, L, W, spans, F, B, params, state, copy_rows=None):
    """compress_layer with the MI EMA weights swapped (rho on the new MI)."""
    out, st = ORIG["compress_layer"](Q, K, V, L, W, spans, F, B, params, state, copy_rows)
    rho = params.rho_mi
    mi_bar = (1.0 - rho) * state.mi_bar + rho * out["mi"]
    out["mi_bar"] = mi_bar
    return out, O.LayerState(st.G, mi_bar, st.m, st.n)


def _stability_swapped_ema(s_cur, m, rho_t, eps):
    phi, _ = ORIG["stability"](s_cur, m, rho_t, eps)
    return phi, rho_t * s_cur + (1.0 - rho_t) * m


def _discount_sign(is_vis, frame, F, phi, delta, d_min, decay="exp"):
    return ORIG["temporal_discount"](is_vis, 2 * F - frame, F, phi, delta, d_min, decay)


def _discount_all_tokens(is_vis, frame, F, phi, delta, d_min, decay="exp"):
    return ORIG["temporal_discount"](np.ones_like(is_vis), frame, F, phi, delta, d_min, decay)


def _entropy_log2(sbar, t_min, t_max, eps):
    L_p = sbar.shape[0]
    p = sbar / (sbar.sum() + eps)
    h = 0.0 if L_p <= 1 else float(-(p * np.log(p + eps)).sum() / math.log2(L_p))
    h = min(1.0, max(0.0, h))
    return h, t_min + (t_max - t_min) * h


def _entropy_reversed_t(sbar, t_min, t_max, eps):
    h, _ = ORIG["entropy_temperature"](sbar, t_min, t_max, eps)
    return h, t_max - (t_max - t_min) * h


def _final_power_t(sbar, beta, D, T):
    s_f = sbar * beta * D
    return s_f, np.maximum(s_f, 0.0) ** T


def _topb_high_index(s, B):
    L_p = s.shape[0]
    order = np.lexsort((-np.arange(L_p), -s))
    return np.sort(order[:B]).astype(np.int64)


def _topb_unsorted(s, B):
    L_p = s.shape[0]
    order = np.lexsort((np.arange(L_p), -s))
    return order[:B].astype(np.int64)


def _gather_no_window(K, V, I, L, W):
    sel = np.asarray(I, dtype=np.int64)
    return K[:, sel], V[:, sel]


def _decode_unscaled(q, K, V):
    q = np.asarray(q, np.float64)
    d = q.shape[1]
    return ORIG["decode_attention"](q * math.sqrt(d), K, V)


def _per_head_interleaved(K, H):
    K = np.asarray(K)
    return np.tile(K, (H // K.shape[0], 1, 1))     # head h reads group h % G


def _discount_variant(linear_unclamped=False, gamma_no_one=False):
    def f(is_vis, frame, F, phi_of_token, delta, d_min, decay="exp"):
        if not ((linear_unclamped and decay == "linear") or (gamma_no_one and decay == "gamma")):
            return ORIG["temporal_discount"](is_vis, frame, F, phi_of_token, delta, d_min, decay)
        D = np.ones(is_vis.shape[0], dtype=np.float64)
        dist = (F - frame).astype(np.float64)
        with np.errstate(divide="ignore"):
            if decay == "linear":
                f_ = 1.0 - delta * dist * phi_of_token
            else:
                f_ = np.power(dist, -delta * phi_of_token)
        D_vis = d_min + (1.0 - d_min) * f_
        D[is_vis] = D_vis[is_vis]
        return D
    return f


def _confidence_unshifted(sbar, t_min, t_max, eps):
    p = sbar / (sbar.sum() + eps)
    c = min(1.0, max(0.0, float(p.max())))
    return 1.0 - c, t_min + (t_max - t_min) * (1.0 - c)


def _confidence_reversed_t(sbar, t_min, t_max, eps):
    u, _ = ORIG["confidence_temperature"](sbar, t_min, t_max, eps)
    return u, t_min + (t_max - t_min) * (1.0 - u)


def _aeb_swapped(sbar, params):
    if params.aeb_mode == "entropy":
        return O.confidence_temperature(sbar, params.t_min, params.t_max, params.eps)
    return O.entropy_temperature(sbar, params.t_min, params.t_max, params.eps)


def _lambda_ramp_long(n, lam, n_warmup, n_ramp):
    if n <= n_warmup:
        return 0.0
    if n_ramp <= 0:
        return lam
    return lam * min(1.0, (n - n_warmup) / (n_ramp + 1))


def _gather_window_from_start(K, V, I, L, W):
    sel = np.concatenate([np.asarray(I, dtype=np.int64), np.arange(W)])
    return K[:, sel], V[:, sel]


def _compress_window_in_softmax(Q, K, V, L, W, spans, F, B, params, state, copy_rows=None):
    """The softmax runs over all L keys, the window's own included, and the
    past tokens keep their share."""
    K_all = np.asarray(K[:, :L], dtype=np.float64)
    L_p = L - W

    def wam(Q_, K_past):
        return ORIG["window_attention_mass"](Q_, K_all)[:, :L_p]

    saved = O.window_attention_mass
    O.window_attention_mass = wam
    try:
        return ORIG["compress_layer"](Q, K, V, L, W, spans, F, B, params, state, copy_rows)
    finally:
        O.window_attention_mass = saved


WAM = ["test_window_rows_sum_to_one", "test_two_key_closed_form_checks_sqrt_d_scaling",
       "test_gqa_head_to_group_map", "test_window_mass_brute_force_tiny",
       "test_zero_queries_give_uniform_mass"]
POOL = ["test_pool_impulse_response", "test_pool_constant_edges_count_padding",
        "test_pool_width_one_is_identity"]
GROUP = ["test_group_scores_reduce_to_mha", "test_group_scores_are_head_means",
         "test_group_scores_are_means_of_per_head_scores"]
RANK = ["test_rank_bins_match_ordinal_ranks_and_equal_frequency",
        "test_rank_bins_all_equal_follow_index", "test_rank_bins_invariant_to_monotone_transform"]
MI = ["test_mi_zero_for_factorised_construction", "test_mi_maximum_ln_k",
      ("test_mi_matches_sklearn_and_entropy_identity", 0), "test_mi_empty_token_set"]
PRIOR = ["test_prior_uniform_when_mi_equal", "test_prior_two_groups_closed_form",
         "test_prior_sums_to_one_and_is_order_preserving"]
STAB = ["test_stability_same_row_twice", "test_stability_uses_old_mean",
        "test_stability_ema_closed_form_and_range"]
ENT = ["test_entropy_uniform_and_one_hot", "test_entropy_matches_scipy",
       "test_entropy_single_token"]
TOPB = ["test_topb_brute_force_and_ties", "test_topb_invariant_under_temperature"]

MUTANTS = [
    ("window_attention_mass", _wam(scale=False), "no 1/sqrt(d)", WAM),
    ("window_attention_mass", _wam(axis=0), "softmax normalised over keys' columns", WAM),
    ("window_attention_mass", _wam(gmap=lambda h, H, G: h % G), "interleaved GQA map", WAM),
    ("window_attention_mass", _wam(transpose=True), "softmax over queries", WAM),
    ("avg_pool1d", _pool_valid_count, "pool divides by the valid count", POOL),
    ("avg_pool1d", _pool_shifted, "pool window shifted by one", POOL),
    ("group_scores", _group_sum, "head sum instead of mean", GROUP),
    ("group_scores", _group_interleaved, "heads dealt round-robin", GROUP),
    ("base_score", _base_last_max, "argmax ties to the last group",
     ["test_base_score_single_group_and_ties"]),
    ("rank_bins", _rank_index_desc, "ties ranked by index descending", RANK),
    ("rank_bins", _rank_ceil, "ceil instead of floor in the bin index", RANK),
    ("plugin_mi", _mi_log2, "log base 2", MI),
    ("plugin_mi", _mi_swapped_marginals, "wrong bin marginal", MI),
    ("spatial_cells", _cells_swapped, "rows and columns swapped", ["test_spatial_cells_per_frame_grid"]),
    ("visual_metadata", _metadata(transpose_shape=True), "span rows and columns swapped",
     ["test_visual_metadata_table"]),
    ("visual_metadata", _metadata(column_major=True), "column-major raster",
     ["test_visual_metadata_table"]),
    ("current_frame_span", _first_span, "stability row from the first span, not frame F's",
     ["test_stability_row_is_the_current_frame"]),
    ("mi_prior", _prior_raw, "no min-max normalisation", PRIOR),
    ("mi_prior", _prior_negated, "sign of the MI flipped", PRIOR),
    ("lambda_schedule", _lambda_early, "warm-up one step short", ["test_lambda_schedule_values"]),
    ("compress_layer", _mi_ema_swapped, "MI EMA weights swapped", ["test_mi_ema_closed_form"]),
    ("stability", _stability_new_mean, "phi from the updated mean", STAB),
    ("stability", _stability_swapped_ema, "EMA weights swapped", STAB),
    ("temporal_discount", _discount_sign, "frame distance sign flipped",
     ["test_discount_closed_form_and_special_cases"]),
    ("temporal_discount", _discount_all_tokens, "text tokens discounted too",
     ["test_discount_closed_form_and_special_cases"]),
    ("entropy_temperature", _entropy_log2, "entropy normalised by log2 L", ENT),
    ("entropy_temperature", _entropy_reversed_t, "temperature runs the wrong way", ENT),
    ("final_score", _final_power_t, "power T instead of 1/T",
     ["test_unit_temperature_leaves_scores_unchanged", "test_power_sharpening_closed_form"]),
    ("topb_select", _topb_high_index, "cut ties keep the higher index", TOPB),
    ("topb_select", _topb_unsorted, "indices not in token order", TOPB),
    ("gather_compact", _gather_no_window, "recent window dropped", ["test_gather_compact_is_row_copy"]),
    ("per_head_cache", _per_head_interleaved, "per-head cache dealt round-robin",
     ["test_per_head_cache_gives_each_head_its_own_attention",
      "test_group_scores_are_means_of_per_head_scores"]),
    ("temporal_discount", _discount_variant(linear_unclamped=True), "linear decay not floored",
     [("test_decay_variants_shared_properties", "linear"),
      "test_decay_variant_closed_forms_and_order"]),
    ("temporal_discount", _discount_variant(gamma_no_one=True), "gamma decay of the distance, not 1 + distance",
     [("test_decay_variants_shared_properties", "gamma"),
      "test_decay_variant_closed_forms_and_order"]),
    ("confidence_temperature", _confidence_unshifted, "confidence not rescaled from 1/L_p",
     ["test_confidence_temperature_ends_and_scale_invariance"]),
    ("confidence_temperature", _confidence_reversed_t, "confidence temperature runs the wrong way",
     ["test_confidence_temperature_ends_and_scale_invariance"]),
    ("lambda_schedule", _lambda_ramp_long, "ramp one step too long", ["test_lambda_schedule_values"]),
    ("aeb_temperature", _aeb_swapped, "AEB variants dispatched the wrong way round",
     ["test_aeb_temperature_closed_forms_per_variant"]),
    ("gather_compact", _gather_window_from_start, "window rows taken from the cache start",
     ["test_gather_compact_is_row_copy"]),
    ("compress_layer", _compress_window_in_softmax, "window keys inside the softmax",
     ["test_layer_scores_sum_to_the_window_rows"]),
    ("decode_attention", _decode_unscaled, "decode logits not scaled by 1/sqrt(d)",
     ["test_decode_two_tokens_closed_form", "test_decode_brute_force_and_token_permutation"]),
]


@pytest.mark.parametrize("name,mutant,what,pins", MUTANTS, ids=[m[2] for m in MUTANTS])
def test_pins_catch_planted_mistake(monkeypatch, name, mutant, what, pins):
    monkeypatch.setattr(O, name, mutant)
    caught = []
    for pin in pins:
        fn, args = (getattr(P, pin[0]), pin[1:]) if isinstance(pin, tuple) else (getattr(P, pin), ())
        try:
            fn(*args)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin)
    assert caught, f"no pin catches: {what} in {name}"


def test_the_same_pins_pass_on_the_oracle_itself():
    """Control: with nothing planted, every pin used above passes, so each
    catch comes from its mistake."""
    seen = []
    for _, _, _, pins in MUTANTS:
        for pin in pins:
            if pin in seen:
                continue
            seen.append(pin)
            fn, args = (getattr(P, pin[0]), pin[1:]) if isinstance(pin, tuple) else (getattr(P, pin), ())
            fn(*args)
    assert len(seen) >= 25
