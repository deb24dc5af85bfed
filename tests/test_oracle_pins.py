"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a closed
form, an invariant the paper states, a special case that reduces to a
library routine, or brute force on tiny inputs.
"""

import math

import numpy as np
import pytest
from scipy import stats
from sklearn.metrics import mutual_info_score

from oracle import starkv_oracle as O


def rng(seed):
    return np.random.default_rng(seed)


# ----------------------------------------------------------------- Eq. A_raw

def test_window_rows_sum_to_one():
    """Each window row is a softmax over the past keys, so summing A_raw over
    tokens gives W for every head (sec. 3.3)."""
    r = rng(1)
    Q = r.standard_normal((6, 5, 16))
    K = r.standard_normal((3, 40, 16)) * 3.0
    A = O.window_attention_mass(Q, K)
    assert A.shape == (6, 40)
    np.testing.assert_allclose(A.sum(axis=1), 5.0, rtol=1e-13)
    assert (A > 0).all()


def test_two_key_closed_form_checks_sqrt_d_scaling():
    """Two keys, one query: p = 1 / (1 + e^{-(x1 - x2)}) with x = q.k/sqrt(d)."""
    d = 4
    Q = np.zeros((1, 1, d))
    Q[0, 0, 0] = 2.0
    K = np.zeros((1, 2, d))
    K[0, 0, 0] = 1.0          # x1 = 2 * 1 / sqrt(4) = 1, x2 = 0
    A = O.window_attention_mass(Q, K)
    p1 = 1.0 / (1.0 + math.exp(-1.0))
    np.testing.assert_allclose(A[0], [p1, 1.0 - p1], rtol=1e-14)


def test_zero_queries_give_uniform_mass():
    Q = np.zeros((2, 7, 8))
    K = rng(2).standard_normal((1, 13, 8))
    A = O.window_attention_mass(Q, K)
    np.testing.assert_allclose(A, 7.0 / 13.0, rtol=1e-14)


def test_gqa_head_to_group_map():
    """g(h) = floor(h G / H): with H=6, G=3 heads {0,1}->0, {2,3}->1, {4,5}->2
    (sec. 3.1).  Changing group 1's keys moves heads 2 and 3 only."""
    r = rng(3)
    Q = r.standard_normal((6, 2, 8))
    K = r.standard_normal((3, 9, 8))
    A0 = O.window_attention_mass(Q, K)
    K2 = K.copy()
    K2[1] = r.standard_normal((9, 8))
    A1 = O.window_attention_mass(Q, K2)
    changed = [not np.allclose(A0[h], A1[h]) for h in range(6)]
    assert changed == [False, False, True, True, False, False]


def test_window_sum_decomposes_over_queries():
    r = rng(4)
    Q = r.standard_normal((2, 4, 8))
    K = r.standard_normal((1, 11, 8))
    A = O.window_attention_mass(Q, K)
    parts = sum(O.window_attention_mass(Q[:, i:i + 1], K) for i in range(4))
    np.testing.assert_allclose(A, parts, rtol=1e-13)


def test_window_mass_brute_force_tiny():
    """Scalar loops over a tiny case: H=2, G=1, W=2, L_p=3, d=2."""
    r = rng(5)
    Q = r.standard_normal((2, 2, 2))
    K = r.standard_normal((1, 3, 2))
    want = np.zeros((2, 3))
    for h in range(2):
        for i in range(2):
            logits = [sum(Q[h, i, j] * K[0, t, j] for j in range(2)) / math.sqrt(2)
                      for t in range(3)]
            z = sum(math.exp(x) for x in logits)
            for t in range(3):
                want[h, t] += math.exp(logits[t]) / z
    np.testing.assert_allclose(O.window_attention_mass(Q, K), want, rtol=1e-13)


# ------------------------------------------------------------ AvgPool1D

def test_pool_impulse_response():
    x = np.zeros((1, 20))
    x[0, 10] = 1.0
    y = O.avg_pool1d(x, 5)
    want = np.zeros(20)
    want[8:13] = 0.2
    np.testing.assert_allclose(y[0], want, atol=1e-16)
    assert y.sum() == pytest.approx(1.0, abs=1e-15)


def test_pool_constant_edges_count_padding():
    y = O.avg_pool1d(np.full((1, 10), 3.0), 5)
    np.testing.assert_allclose(y[0], [1.8, 2.4, 3, 3, 3, 3, 3, 3, 2.4, 1.8], rtol=1e-15)


def test_pool_width_one_is_identity():
    x = rng(6).random((3, 17))
    np.testing.assert_array_equal(O.avg_pool1d(x, 1), x)


# ------------------------------------------------------------ Eq. base_score

def test_group_scores_reduce_to_mha():
    """G = H recovers standard multi-head attention: S = A (sec. 3.1)."""
    A = rng(7).random((4, 9))
    np.testing.assert_allclose(O.group_scores(A, 4), A, rtol=1e-15)


def test_group_scores_are_head_means():
    A = np.repeat(np.array([[1.0], [2.0], [3.0], [4.0]]), 5, axis=1)
    S = O.group_scores(A, 2)
    np.testing.assert_allclose(S, [[1.5] * 5, [3.5] * 5], rtol=1e-15)


def test_per_head_cache_gives_each_head_its_own_attention():
    """MHA-head granularity on a GQA model (sec. 4.2 ablation): with K
    replicated per head, the per-head window mass equals the GQA model's own
    per-head mass (every head still reads its group's keys), and S = A."""
    r = rng(21)
    H, G, W, L, d = 6, 2, 3, 11, 8
    Q = r.standard_normal((H, W, d))
    K = r.standard_normal((G, L, d))
    Kh = O.per_head_cache(K, H)
    assert Kh.shape == (H, L, d)
    for h in range(H):
        np.testing.assert_array_equal(Kh[h], K[h * G // H])
    A_gqa = O.window_attention_mass(Q, K)        # heads read group h G / H
    A_mha = O.window_attention_mass(Q, Kh)       # head h reads its own copy
    np.testing.assert_allclose(A_mha, A_gqa, rtol=1e-14)
    S = O.group_scores(A_mha, H)
    np.testing.assert_allclose(S, A_gqa, rtol=1e-14)


def test_group_scores_are_means_of_per_head_scores():
    """The GQA-group score of a group is the mean of its heads' per-head
    scores (Eq. base_score is linear in A), pooled or not."""
    r = rng(22)
    H, G, W, L, d = 8, 2, 4, 40, 16
    Q = r.standard_normal((H, W, d))
    K = r.standard_normal((G, L, d))
    A = O.avg_pool1d(O.window_attention_mass(Q, K), 5)
    S_group = O.group_scores(A, G)
    S_head = O.group_scores(O.avg_pool1d(O.window_attention_mass(Q, O.per_head_cache(K, H)), 5), H)
    np.testing.assert_allclose(S_head.reshape(G, H // G, L).mean(axis=1), S_group, rtol=1e-13)


def test_base_score_single_group_and_ties():
    S = rng(8).random((1, 6))
    sbar, gstar = O.base_score(S)
    np.testing.assert_array_equal(sbar, S[0])
    assert (gstar == 0).all()
    S2 = np.array([[1.0, 2.0, 5.0], [3.0, 2.0, 1.0], [3.0, 1.0, 5.0]])
    sbar2, g2 = O.base_score(S2)
    np.testing.assert_allclose(sbar2, [7 / 3, 5 / 3, 11 / 3], rtol=1e-15)
    assert list(g2) == [1, 0, 0]      # ties keep the lowest group


# ------------------------------------------------------------ RankBin / MI

def test_rank_bins_match_ordinal_ranks_and_equal_frequency():
    r = rng(9)
    v = r.random(103)
    v[10] = v[20] = v[30]          # ties resolved by index
    b = O.rank_bins(v, 8)
    ordinal = stats.rankdata(v, method="ordinal") - 1
    np.testing.assert_array_equal(b, ordinal * 8 // 103)
    counts = np.bincount(b, minlength=8)
    assert set(counts) <= {103 // 8, 103 // 8 + 1}
    assert b[10] <= b[20] <= b[30]


def test_rank_bins_all_equal_follow_index():
    b = O.rank_bins(np.full(10, 0.5), 4)
    np.testing.assert_array_equal(b, (np.arange(10) * 4) // 10)


def test_rank_bins_invariant_to_monotone_transform():
    v = rng(10).random(50)
    np.testing.assert_array_equal(O.rank_bins(v, 5), O.rank_bins(np.exp(3 * v) + 7, 5))


def _grid(nr, nc):
    t = np.arange(nr * nc)
    return t // nc, t % nc


def test_mi_zero_for_factorised_construction():
    """16x16 tokens on an 8x8 grid: four tokens per cell, one per 2x2
    sub-position.  Values ordered by sub-position make every cell hold one
    token of each of the K=4 bins, so p(b,c) = p(b) p(c) and MI = 0."""
    r, c = _grid(16, 16)
    cell = O.spatial_cells(r, c, 16, 16, 8)
    sub = (r % 2) * 2 + (c % 2)
    values = sub * 1000.0 + cell
    b = O.rank_bins(values, 4)
    assert O.plugin_mi(b, cell, 4, 64) == 0.0


def test_constant_attention_is_not_mi_zero_under_index_ties():
    """Constant values rank by index, so bins follow raster order and share
    information with the rows: MI > 0 (the reason the zero case above is
    built from sub-positions)."""
    r, c = _grid(16, 16)
    cell = O.spatial_cells(r, c, 16, 16, 8)
    b = O.rank_bins(np.ones(256), 4)
    assert O.plugin_mi(b, cell, 4, 64) > 0.1


def test_mi_maximum_ln_k():
    """K = M^2 bins, equal cells, values increasing with the cell id: bins
    equal cells and MI = ln K."""
    r, c = _grid(4, 4)
    cell = O.spatial_cells(r, c, 4, 4, 2)
    values = cell * 10.0 + np.arange(16) * 0.01
    b = O.rank_bins(values, 4)
    assert O.plugin_mi(b, cell, 4, 4) == pytest.approx(math.log(4), rel=1e-14)


@pytest.mark.parametrize("seed", [11, 12, 13])
def test_mi_matches_sklearn_and_entropy_identity(seed):
    r = rng(seed)
    nr, nc = 13, 17
    rr, cc = _grid(nr, nc)
    cell = O.spatial_cells(rr, cc, nr, nc, 4)
    values = r.random(nr * nc) + 0.5 * (cc > nc // 2)
    b = O.rank_bins(values, 5)
    mi = O.plugin_mi(b, cell, 5, 16)
    assert mi == pytest.approx(mutual_info_score(b, cell), rel=1e-12, abs=1e-14)
    joint = np.zeros((5, 16))
    np.add.at(joint, (b, cell), 1)
    h_b = stats.entropy(joint.sum(1))
    h_c = stats.entropy(joint.sum(0))
    h_bc = stats.entropy(joint.ravel())
    assert mi == pytest.approx(h_b + h_c - h_bc, rel=1e-12, abs=1e-14)
    assert 0.0 <= mi <= min(math.log(5), h_c) + 1e-12


def test_spatial_cells_per_frame_grid():
    r, c = _grid(39, 69)
    cell = O.spatial_cells(r, c, 39, 69, 8)
    assert cell.min() == 0 and cell.max() == 63
    assert cell[0] == 0 and cell[68] == 7 and cell[-1] == 63
    assert cell[38 * 69] == 56


def test_visual_metadata_table():
    """Sec. 3.1: a frame's rows x cols patch tokens are one raster-ordered
    run from the span's first token, token start + r*cols + c at row r,
    column c.  Two non-square spans at non-zero starts (2 rows x 3 columns
    from token 3, frame 1; 3 rows x 2 columns from token 11, frame 2), with
    every entry written out by hand."""
    spans = [(3, 2, 3, 1), (11, 3, 2, 2)]
    is_vis, frame, r, c, rows, cols = O.visual_metadata(spans, 19)
    # token:           0  1  2  3  4  5  6  7  8  9 10 11 12 13 14 15 16 17 18
    want_vis = [0, 0, 0, 1, 1, 1, 1, 1, 1, 0, 0, 1, 1, 1, 1, 1, 1, 0, 0]
    want_frame = [0, 0, 0, 1, 1, 1, 1, 1, 1, 0, 0, 2, 2, 2, 2, 2, 2, 0, 0]
    want_r = [0, 0, 0, 0, 0, 0, 1, 1, 1, 0, 0, 0, 0, 1, 1, 2, 2, 0, 0]
    want_c = [0, 0, 0, 0, 1, 2, 0, 1, 2, 0, 0, 0, 1, 0, 1, 0, 1, 0, 0]
    want_rows = [1, 1, 1, 2, 2, 2, 2, 2, 2, 1, 1, 3, 3, 3, 3, 3, 3, 1, 1]
    want_cols = [1, 1, 1, 3, 3, 3, 3, 3, 3, 1, 1, 2, 2, 2, 2, 2, 2, 1, 1]
    assert is_vis.tolist() == [bool(v) for v in want_vis]
    assert frame.tolist() == want_frame
    assert r.tolist() == want_r
    assert c.tolist() == want_c
    assert rows.tolist() == want_rows
    assert cols.tolist() == want_cols
    # the map feeds the M x M cells of Eq. MI: at M = 2 the 2 x 3 frame's
    # columns split 0,0,1 (floor(c*2/3)) and its rows 0 | 1
    vis = np.nonzero(is_vis)[0]
    cells = O.spatial_cells(r[vis], c[vis], rows[vis], cols[vis], 2)
    # the 3 x 2 frame's rows split 0,0,1 (floor(r*2/3)) and its columns 0 | 1
    assert cells.tolist() == [0, 0, 1, 2, 2, 3, 0, 1, 0, 1, 2, 3]


def test_mi_empty_token_set():
    assert O.plugin_mi(np.zeros(0, dtype=int), np.zeros(0, dtype=int), 8, 64) == 0.0


# ------------------------------------------------------------ subspace prior

def test_prior_uniform_when_mi_equal():
    w = O.mi_prior(np.full(4, 0.3), 1.0, 1e-8)
    np.testing.assert_allclose(w, 0.25, rtol=1e-15)
    # G w_{g*} averages to one: beta = (1 - lam) + lam G w = 1 (sec. 3.4)
    lam = 0.5
    np.testing.assert_allclose((1 - lam) + lam * 4 * w, 1.0, rtol=1e-15)


def test_prior_two_groups_closed_form():
    eps = 1e-8
    w = O.mi_prior(np.array([0.2, 1.2]), 2.0, eps)
    m1 = 1.0 / (1.0 + eps)
    want1 = math.exp(m1 / 2) / (1 + math.exp(m1 / 2))
    np.testing.assert_allclose(w, [1 - want1, want1], rtol=1e-14)


def test_prior_sums_to_one_and_is_order_preserving():
    mi = rng(14).random(6)
    w = O.mi_prior(mi, 1.0, 1e-8)
    assert w.sum() == pytest.approx(1.0, abs=1e-15)
    assert list(np.argsort(w)) == list(np.argsort(mi))


def test_lambda_schedule_values():
    vals = [O.lambda_schedule(n, 0.5, 5, 10) for n in range(1, 21)]
    assert vals[:5] == [0.0] * 5
    assert vals[5] == pytest.approx(0.05)
    assert vals[9] == pytest.approx(0.25)
    assert vals[14:] == [0.5] * 6
    assert O.lambda_schedule(1, 0.5, 0, 0) == 0.5


def test_mi_ema_closed_form():
    """The same layer input on n steps from a fresh state gives the same MI
    every step, so the EMA from zero (sec. 3.4) closes to (1 - rho^n) MI."""
    Q, K, V, L, W, spans = _tiny_layer(31)
    p = O.Params(rho_mi=0.9)
    st = O.LayerState(2)
    for _ in range(7):
        out, st = O.compress_layer(Q, K, V, L, W, spans, 1, 5, p, st)
    assert (out["mi"] > 0).all()
    np.testing.assert_allclose(out["mi_bar"], (1 - 0.9 ** 7) * out["mi"], rtol=1e-13)
    assert st.n == 7


# ------------------------------------------------------------ stability

def test_stability_same_row_twice():
    s = rng(15).random((3, 20))
    phi1, m1 = O.stability(s, np.zeros((3, 20)), 0.9, 1e-8)
    np.testing.assert_array_equal(phi1, 0.0)
    np.testing.assert_allclose(m1, 0.1 * s, rtol=1e-15)
    phi2, _ = O.stability(s, m1, 0.9, 1e-8)
    np.testing.assert_allclose(phi2, 1.0, atol=1e-7)


def test_stability_uses_old_mean():
    """phi comes from m before the update: orthogonal rows give phi = 0."""
    s1 = np.array([[1.0, 0.0, 2.0, 0.0]])
    s2 = np.array([[0.0, 3.0, 0.0, 1.0]])
    _, m1 = O.stability(s1, np.zeros((1, 4)), 0.9, 1e-8)
    phi2, m2 = O.stability(s2, m1, 0.9, 1e-8)
    assert phi2[0] == 0.0
    np.testing.assert_allclose(m2, 0.09 * s1 + 0.1 * s2, rtol=1e-15)


def test_stability_ema_closed_form_and_range():
    s = rng(16).random((2, 8))
    m = np.zeros((2, 8))
    for _ in range(5):
        phi, m = O.stability(s, m, 0.8, 1e-8)
    np.testing.assert_allclose(m, (1 - 0.8 ** 5) * s, rtol=1e-14)
    assert ((phi >= 0) & (phi <= 1 + 1e-12)).all()


# ------------------------------------------------------------ discount

def test_discount_closed_form_and_special_cases():
    is_vis = np.array([True, True, True, False, True])
    frame = np.array([1, 2, 3, 0, 1])
    phi_t = np.array([0.5, 1.0, 0.3, 0.9, 0.0])
    D = O.temporal_discount(is_vis, frame, 3, phi_t, 0.2, 0.1)
    want0 = 0.1 + 0.9 * math.exp(-0.2 * 2 * 0.5)
    want1 = 0.1 + 0.9 * math.exp(-0.2 * 1 * 1.0)
    np.testing.assert_allclose(D, [want0, want1, 1.0, 1.0, 1.0], rtol=1e-15)
    # delta = 0 and a single frame both give D = 1
    np.testing.assert_array_equal(
        O.temporal_discount(is_vis, frame, 3, phi_t, 0.0, 0.1), 1.0)
    np.testing.assert_array_equal(
        O.temporal_discount(is_vis, np.full(5, 3), 3, phi_t, 0.2, 0.1), 1.0)
    far = O.temporal_discount(np.array([True]), np.array([0]), 10 ** 6,
                              np.array([1.0]), 0.2, 0.1)
    assert far[0] == pytest.approx(0.1, abs=1e-15)


# ------------------------------------------------------------ AEB

def test_entropy_uniform_and_one_hot():
    h, T = O.entropy_temperature(np.full(100, 0.37), 0.75, 1.25, 1e-8)
    assert h == pytest.approx(1.0, abs=1e-6)
    assert T == pytest.approx(1.25, abs=1e-6)
    one = np.zeros(100)
    one[17] = 2.0
    h0, T0 = O.entropy_temperature(one, 0.75, 1.25, 1e-8)
    assert h0 == pytest.approx(0.0, abs=1e-7)
    assert T0 == pytest.approx(0.75, abs=1e-7)


def test_entropy_matches_scipy():
    x = rng(17).random(3000) ** 3
    h0, _ = O.entropy_temperature(x, 0.75, 1.25, 0.0)
    assert h0 == pytest.approx(stats.entropy(x) / math.log(3000), rel=1e-12)
    h, _ = O.entropy_temperature(x, 0.75, 1.25, 1e-8)
    # eps inside the log moves H^ by at most L eps / ln L
    assert abs(h - h0) <= 3000 * 1e-8 / math.log(3000) + 1e-12
    assert 0.0 <= h <= 1.0


def test_entropy_single_token():
    assert O.entropy_temperature(np.array([1.0]), 0.5, 1.5, 1e-8) == (0.0, 0.5)


# ------------------------------------------------------------ final score

def test_unit_temperature_leaves_scores_unchanged():
    r = rng(18)
    sbar, beta, D = r.random(50), r.random(50) + 0.5, r.random(50)
    s_f, s = O.final_score(sbar, beta, D, 1.0)
    np.testing.assert_array_equal(s, s_f)
    np.testing.assert_array_equal(s_f, sbar * beta * D)


def test_power_sharpening_closed_form():
    s_f, s = O.final_score(np.array([0.25, 4.0, -1.0]), np.ones(3), np.ones(3), 2.0)
    np.testing.assert_allclose(s, [0.5, 2.0, 0.0], rtol=1e-15)
    _, s2 = O.final_score(np.array([0.25, 4.0]), np.ones(2), np.ones(2), 0.5)
    np.testing.assert_allclose(s2, [0.0625, 16.0], rtol=1e-15)


# ------------------------------------------------------------ selection

def test_topb_brute_force_and_ties():
    r = rng(19)
    s = np.round(r.random(30), 1)     # many ties
    for B in [0, 1, 7, 15, 29, 30]:
        I = O.topb_select(s, B)
        brute = sorted(sorted(range(30), key=lambda t: (-s[t], t))[:B])
        assert list(I) == brute
        assert len(I) == B
        assert all(I[i] < I[i + 1] for i in range(len(I) - 1))


def test_topb_invariant_under_temperature():
    """x^(1/T) is increasing, so the hard top-B set does not depend on T."""
    r = rng(20)
    s_f = r.random(200)
    _, s = O.final_score(s_f, np.ones(200), np.ones(200), 0.8)
    np.testing.assert_array_equal(O.topb_select(s, 40), O.topb_select(s_f, 40))


def test_gather_compact_is_row_copy():
    r = rng(21)
    K = r.integers(0, 65535, size=(2, 12, 4)).astype(np.uint16)
    V = r.integers(0, 65535, size=(2, 12, 4)).astype(np.uint16)
    I = np.array([1, 4, 5])
    Ko, Vo = O.gather_compact(K, V, I, 10, 3)
    np.testing.assert_array_equal(Ko, K[:, [1, 4, 5, 7, 8, 9]])
    np.testing.assert_array_equal(Vo, V[:, [1, 4, 5, 7, 8, 9]])
    assert Ko.dtype == np.uint16


# ------------------------------------------------------------ whole layer

def _tiny_layer(seed, n_frames=1, H=4, G=2, d=8, nr=4, nc=5, text=6, W=3):
    r = rng(seed)
    nf = nr * nc
    L = n_frames * nf + text
    spans = [((f - 1) * nf, nr, nc, f) for f in range(1, n_frames + 1)]
    Q = r.standard_normal((H, W, d))
    K = r.standard_normal((G, L, d))
    V = r.standard_normal((G, L, d))
    return Q, K, V, L, W, spans


def test_base_reduction():
    """lambda = 0, one frame and T_min = T_max = 1 reduce STaR-KV to the
    'Base' ablation row: s = sbar and a global top-B of the GQA-mean score."""
    Q, K, V, L, W, spans = _tiny_layer(22)
    p = O.Params(lam=0.0, t_min=1.0, t_max=1.0)
    out, _ = O.compress_layer(Q, K, V, L, W, spans, 1, 7, p, O.LayerState(2))
    np.testing.assert_array_equal(out["s"], out["sbar"])
    np.testing.assert_array_equal(out["D"], 1.0)
    np.testing.assert_array_equal(out["beta"], 1.0)
    assert list(out["I"]) == sorted(np.argsort(-out["sbar"], kind="stable")[:7])


def test_layer_scores_sum_to_the_window_rows():
    """Sec. 3.3 with the softmax over the L_p past keys: every window row's
    mass sums to 1 over the past tokens, so with one head per group and a
    pool of width 1, each group's score row S sums to W exactly (the window's
    own keys take no share of it)."""
    Q, K, V, L, W, spans = _tiny_layer(26, H=2, G=2)
    p = O.Params(pool_kernel=1)
    out, _ = O.compress_layer(Q, K, V, L, W, spans, 1, 5, p, O.LayerState(2))
    np.testing.assert_allclose(out["S"].sum(axis=1), [W, W], rtol=1e-12)


def test_layer_state_across_steps():
    """Two steps: the counter advances, MI_bar follows the EMA recursion from
    zero, phi is 0 on the first step, and frame-1 tokens get discounted."""
    p = O.Params(n_warmup=0, n_ramp=0)
    st = O.LayerState(2)
    Q, K, V, L, W, spans = _tiny_layer(23, n_frames=2)
    nf = 20
    spans1 = spans[:1]
    L1 = nf + 6
    K1 = np.concatenate([K[:, :nf], K[:, 2 * nf:]], axis=1)
    V1 = np.concatenate([V[:, :nf], V[:, 2 * nf:]], axis=1)
    o1, st = O.compress_layer(Q, K1, V1, L1, W, spans1, 1, 5, p, st)
    assert st.n == 1
    np.testing.assert_array_equal(o1["phi"], 0.0)
    np.testing.assert_allclose(o1["mi_bar"], 0.1 * o1["mi"], rtol=1e-15)
    o2, st = O.compress_layer(Q, K, V, L, W, spans, 2, 9, p, st)
    assert st.n == 2
    np.testing.assert_allclose(o2["mi_bar"], 0.09 * o1["mi"] + 0.1 * o2["mi"], rtol=1e-14)
    assert ((o2["phi"] > 0) & (o2["phi"] <= 1)).all()
    old = np.arange(nf)
    want = 0.1 + 0.9 * np.exp(-0.2 * 1 * o2["phi"][o2["gstar"][old]])
    np.testing.assert_allclose(o2["D"][old], want, rtol=1e-14)
    np.testing.assert_array_equal(o2["D"][nf:], 1.0)
    lam = 0.5
    np.testing.assert_allclose(
        o2["beta"], (1 - lam) + lam * 2 * o2["w"][o2["gstar"]], rtol=1e-15)
    assert len(o2["I"]) == 9
    assert o2["K_out"].shape == (2, 9 + W, 8)


def test_frame_size_change_resets_stability():
    p = O.Params()
    st = O.LayerState(2)
    Q, K, V, L, W, spans = _tiny_layer(24)
    _, st = O.compress_layer(Q, K, V, L, W, spans, 1, 4, p, st)
    Q2, K2, V2, L2, W2, spans2 = _tiny_layer(25, nr=3, nc=5)
    o, st = O.compress_layer(Q2, K2, V2, L2, W2, spans2, 1, 4, p, st)
    np.testing.assert_array_equal(o["phi"], 0.0)
    assert st.m.shape == (2, 15)


def test_stability_row_is_the_current_frame():
    """Sec. 3.5: s_g^(c) is the current frame F's score row.  One query per
    head and one head per group make S[g] = softmax of one logit row, so a
    frame whose keys repeat the previous step's frame has a score row
    proportional to that step's: phi = 1 exactly when the row is taken from
    frame F.  Step 1 caches frame A; step 2 caches [B (frame 1); A (frame 2)]
    with F = 2, where B is unrelated, so frame 1's row would give phi < 1."""
    r = rng(32)
    G = H = 2
    W, d, nr, nc, n_text = 1, 8, 2, 3, 4
    nf = nr * nc
    A_k = r.standard_normal((G, nf, d)) * 2.0
    B_k = r.standard_normal((G, nf, d)) * 2.0
    text = r.standard_normal((G, n_text, d))
    Q = r.standard_normal((H, W, d))
    # a negligible epsilon, so that the cosine of parallel rows is 1 to rounding
    p = O.Params(pool_kernel=1, n_warmup=0, n_ramp=0, eps=1e-30)
    K1 = np.concatenate([A_k, text], axis=1)
    o1, st = O.compress_layer(Q, K1, K1, nf + n_text, W, [(0, nr, nc, 1)], 1, 3, p,
                              O.LayerState(G))
    K2 = np.concatenate([B_k, A_k, text], axis=1)
    spans2 = [(0, nr, nc, 1), (nf, nr, nc, 2)]
    o2, st = O.compress_layer(Q, K2, K2, 2 * nf + n_text, W, spans2, 2, 3, p, st)
    np.testing.assert_allclose(o2["phi"], 1.0, rtol=0, atol=1e-12)
    # the rows themselves: frame A's scores scale by the softmax normaliser
    ratio = o2["S"][:, nf:2 * nf] / o1["S"][:, :nf]
    np.testing.assert_allclose(ratio, ratio[:, :1] * np.ones((1, nf)), rtol=1e-12)
    # the EMA from zero after two steps: 0.09 * step-1 row + 0.1 * step-2 row
    np.testing.assert_allclose(st.m, 0.09 * o1["S"][:, :nf] + 0.1 * o2["S"][:, nf:2 * nf],
                               rtol=1e-14)
    # frame 1's row at step 2 is not parallel to step 1's row
    b = o2["S"][:, :nf]
    a = o1["S"][:, :nf]
    cos = (a * b).sum(1) / np.sqrt((a * a).sum(1) * (b * b).sum(1))
    assert (cos < 0.999).all()


# ----------------------------------------------- decode over the cache (4.3)

def test_decode_zero_query_averages_values():
    """q = 0: every logit is 0, so each head returns the mean of its group's
    value rows."""
    r = rng(31)
    K, V = r.standard_normal((2, 9, 8)), r.standard_normal((2, 9, 8))
    o = O.decode_attention(np.zeros((4, 8)), K, V)
    np.testing.assert_allclose(o[:2], np.repeat(V[0].mean(0)[None], 2, 0), rtol=1e-14)
    np.testing.assert_allclose(o[2:], np.repeat(V[1].mean(0)[None], 2, 0), rtol=1e-14)


def test_decode_two_tokens_closed_form():
    """Two tokens: o = sigma(x1 - x2) v1 + (1 - sigma(x1 - x2)) v2 with
    x = q.k / sqrt(d)."""
    q = np.array([[1.0, 2.0, 0.0, -1.0]])
    K = np.array([[[0.5, 0.0, 1.0, 0.0], [0.0, -1.0, 0.0, 2.0]]])
    V = np.array([[[1.0, 2.0, 3.0, 4.0], [-4.0, 0.0, 1.0, 0.5]]])
    x1, x2 = 0.5 / 2.0, -4.0 / 2.0
    w = 1.0 / (1.0 + math.exp(-(x1 - x2)))
    np.testing.assert_allclose(O.decode_attention(q, K, V)[0], w * V[0, 0] + (1 - w) * V[0, 1],
                               rtol=1e-14)


def test_decode_brute_force_and_token_permutation():
    """Against scalar loops on a tiny GQA case; permuting the cached tokens
    (K and V rows together) leaves the output unchanged."""
    r = rng(32)
    H, G, n, d = 6, 3, 7, 5
    q, K, V = r.standard_normal((H, d)), r.standard_normal((G, n, d)), r.standard_normal((G, n, d))
    o = O.decode_attention(q, K, V)
    for h in range(H):
        g = h * G // H
        x = [sum(q[h, j] * K[g, t, j] for j in range(d)) / math.sqrt(d) for t in range(n)]
        e = [math.exp(xi) for xi in x]
        want = [sum(e[t] * V[g, t, j] for t in range(n)) / sum(e) for j in range(d)]
        np.testing.assert_allclose(o[h], want, rtol=1e-12)
    perm = r.permutation(n)
    np.testing.assert_allclose(O.decode_attention(q, K[:, perm], V[:, perm]), o, rtol=1e-13)


# --------------------------------- ablation variants (sec. 4.2, readings)

def _disc(decay, dist, phi, delta=0.2, d_min=0.1):
    n = len(dist)
    return O.temporal_discount(np.ones(n, bool), 10 - np.asarray(dist, float), 10,
                               np.asarray(phi, float), delta, d_min, decay)


@pytest.mark.parametrize("decay", ["exp", "linear", "gamma"])
def test_decay_variants_shared_properties(decay):
    """Every decay: D = 1 for the current frame or phi = 0, D in [D_min, 1],
    non-increasing in the frame distance, and the exponential's slope at 0."""
    assert np.all(_disc(decay, [0, 0], [0.7, 1.0]) == 1.0)
    assert np.all(_disc(decay, [3, 9], [0.0, 0.0]) == 1.0)
    D = _disc(decay, np.arange(0, 60), np.full(60, 0.9))
    assert np.all((D >= 0.1) & (D <= 1.0)) and np.all(np.diff(D) <= 0)
    h = 1e-6     # one-sided derivative in the frame distance at 0, phi = 0.5
    d1 = _disc(decay, np.array([h]), [0.5])[0]
    assert (1.0 - d1) / (h * 0.2 * 0.5) == pytest.approx(0.9, rel=1e-4)


def test_decay_variant_closed_forms_and_order():
    """Linear: D_min + (1 - D_min)(1 - eta), floored at D_min from eta = 1;
    gamma: D_min + (1 - D_min)(1 + dist)^(-delta phi).  For every distance
    linear <= exponential <= gamma (1 - x <= e^-x <= (1 + d)^(-c) with
    x = c d): the ablation's finding that linear drops history hardest and
    gamma keeps the most."""
    np.testing.assert_allclose(_disc("linear", [2], [1.0]), [0.1 + 0.9 * 0.6], rtol=1e-15)
    np.testing.assert_allclose(_disc("linear", [6], [1.0]), [0.1], rtol=1e-15)
    np.testing.assert_allclose(_disc("gamma", [3], [0.5]), [0.1 + 0.9 * 4 ** -0.1], rtol=1e-14)
    dist, phi = np.arange(1, 40), np.linspace(0.05, 1.0, 39)
    lin, ex, ga = (_disc(k, dist, phi) for k in ("linear", "exp", "gamma"))
    assert np.all(lin <= ex + 1e-15) and np.all(ex <= ga + 1e-15)


def test_confidence_temperature_ends_and_scale_invariance():
    """Uniform base scores: confidence 0, T = T_max (as the entropy variant);
    one-hot: confidence 1, T = T_min; a single token counts as one-hot; the
    statistic does not change when sbar is scaled."""
    u, T = O.confidence_temperature(np.full(50, 0.3), 0.75, 1.25, 0.0)
    assert u == pytest.approx(1.0, abs=1e-12) and T == pytest.approx(1.25, abs=1e-12)
    x = np.zeros(50)
    x[7] = 2.0
    u, T = O.confidence_temperature(x, 0.75, 1.25, 0.0)
    assert u == pytest.approx(0.0, abs=1e-12) and T == pytest.approx(0.75, abs=1e-12)
    assert O.confidence_temperature(np.array([3.0]), 0.75, 1.25, 1e-8) == (0.0, 0.75)
    r = rng(41).random(300)
    a, b = O.confidence_temperature(r, 0.9, 1.1, 0.0), O.confidence_temperature(r * 7.0, 0.9, 1.1, 0.0)
    assert a[0] == pytest.approx(b[0], rel=1e-12)
    p = r / r.sum()
    assert a[0] == pytest.approx(1.0 - (p.max() - 1 / 300) / (1 - 1 / 300), rel=1e-12)


def test_aeb_temperature_closed_forms_per_variant():
    """s̄ = (1, 1, 2): p = (1/4, 1/4, 1/2).  Entropy variant (sec. 3.6):
    H^ = (ln 4 / 2 + ln 2 / 2) / ln 3; confidence variant (sec. 4.2 ablation,
    the reading documented with it): c = (1/2 - 1/3) / (1 - 1/3) = 1/4, so the
    statistic is 3/4.  T = T_min + (T_max - T_min) x statistic in both; an
    unknown variant is rejected."""
    sbar = np.array([1.0, 1.0, 2.0])
    h = (0.5 * math.log(4.0) + 0.5 * math.log(2.0)) / math.log(3.0)
    for mode, stat in (("entropy", h), ("confidence", 0.75)):
        p = O.Params(t_min=0.8, t_max=1.3, eps=0.0, aeb_mode=mode)
        u, T = O.aeb_temperature(sbar, p)
        assert u == pytest.approx(stat, rel=1e-12), mode
        assert T == pytest.approx(0.8 + 0.5 * stat, rel=1e-12), mode
    with pytest.raises(ValueError):
        O.aeb_temperature(sbar, O.Params(aeb_mode="peak"))
