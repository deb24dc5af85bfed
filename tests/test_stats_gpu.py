"""GPU parity of the online statistics (sec. 3.4-3.6) on synthetic score rows.

starkv_update_state is fed score rows S built on the host, bypassing the
scoring stage, so that the equal-frequency bin edges land where the
selection has its harder paths: many distinct-but-close keys around an edge
(more than the kernel compacts into LDS), runs of exactly equal keys that
span frames (the tie rule orders them by token index), and more visual
tokens than the kernel caches in LDS.  The oracle bins the same float32
values, so both sides decide on identical numbers.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import starkv_oracle as O  # noqa: E402
from paper_2606_01790_amd import starkv as sk  # noqa: E402

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[stats] {msg}", flush=True)


def layout(n_frames, rows, cols, gap=37, head=50, tail=100):
    spans, t = [], head
    for f in range(1, n_frames + 1):
        spans.append((t, rows, cols, f))
        t += rows * cols + gap
    return spans, t - gap + tail


def cluster_row(rng, Lp, vis, n_below, n_cluster, base=1e-4):
    """Scores of one group: n_below visual tokens under `base`, n_cluster
    tokens whose float32 keys sit within 8 ulps of `base` (so they share
    every leading key bit but the last three, and repeat exactly), the rest
    above it; text tokens random."""
    row = rng.uniform(1e-3, 1e-2, Lp).astype(np.float32)
    perm = rng.permutation(vis)
    lo = perm[:n_below]
    cl = perm[n_below:n_below + n_cluster]
    hi = perm[n_below + n_cluster:]
    row[lo] = rng.uniform(1e-5, 5e-5, lo.size).astype(np.float32)
    bits = np.full(cl.size, np.float32(base).view(np.uint32), np.uint32)
    bits += rng.integers(0, 8, cl.size).astype(np.uint32)
    row[cl] = bits.view(np.float32)
    row[hi] = rng.uniform(2e-4, 1e-2, hi.size).astype(np.float32)
    return row


def run_stats(tag, S_steps, sbar, spans, frame, p, mi_tol=1e-5):
    """S_steps: list of [n_layers, G, Lp] float32 score tensors, one per call
    with the same spans; checks MI (within mi_tol), phi and H^ of every call."""
    n_layers, G, Lp = S_steps[0].shape
    W = 8
    dims = sk.make_dims(n_layers, 2 * G, G, 64, Lp + W, W, sk.BF16)
    op = O.Params(n_bins=int(p.n_bins), grid=int(p.grid), rho_t=float(p.rho_t),
                  eps=float(p.eps))
    is_vis, fr, r, c, rows, cols = O.visual_metadata(spans, Lp)
    vis = np.nonzero(is_vis)[0]
    cells = O.spatial_cells(r[vis], c[vis], rows[vis], cols[vis], op.grid)
    cur = [s for s in spans if s[3] == frame][0]
    cur_tok = np.arange(cur[0], cur[0] + cur[1] * cur[2])
    frame_cap = cur[1] * cur[2]
    dev = torch.device("cuda:0")
    state = torch.empty(sk.state_bytes(dims, frame_cap), dtype=torch.uint8, device=dev)
    scal = torch.empty(n_layers * sk.scalars_count(dims), dtype=torch.float32, device=dev)
    sbar_d = torch.from_numpy(np.repeat(sbar[None, :], n_layers, axis=0)).to(dev)
    say(f"{tag}: N={vis.size} G={G} layers={n_layers} steps={len(S_steps)}")
    sk.state_init(dims, state, frame_cap)
    m = np.zeros((n_layers, G, frame_cap))
    h_or, _ = O.entropy_temperature(sbar.astype(np.float64), 0.75, 1.25, op.eps)
    for step, S in enumerate(S_steps, 1):
        S_d = torch.from_numpy(S).to(dev)
        sk.update_state(dims, p, S_d, sbar_d, spans, frame, state, frame_cap, scal)
        torch.cuda.synchronize()
        sc = scal.cpu().numpy().reshape(n_layers, -1)
        for layer in range(n_layers):
            S64 = S[layer].astype(np.float64)
            mi = np.array([O.plugin_mi(O.rank_bins(S64[g, vis], op.n_bins), cells,
                                       op.n_bins, op.grid * op.grid) for g in range(G)])
            phi, m[layer] = O.stability(S64[:, cur_tok], m[layer], op.rho_t, op.eps)
            got_mi = sc[layer, 0:G]
            got_phi = sc[layer, 3 * G:4 * G]
            assert np.max(np.abs(got_mi - mi)) <= mi_tol, \
                f"{tag} step{step} L{layer}: MI {got_mi} vs {mi}"
            assert np.max(np.abs(got_phi - phi)) <= 1e-5, \
                f"{tag} step{step} L{layer}: phi {got_phi} vs {phi}"
            assert abs(sc[layer, 4 * G + 1] - h_or) <= 1e-5, f"{tag}: H^"
    say(f"{tag}: ok")


def test_edges_in_dense_key_clusters():
    """Five 69x39 frames (N = 13455).  Group 0: 3000 near-equal keys at the
    bottom hold the first edge (beyond the LDS candidate list); group 1: 1500
    of them hold the second edge (within it); group 2: exact ties only,
    every key one of two values; group 3: plain random scores."""
    rng = np.random.default_rng(7)
    spans, Lp = layout(5, 39, 69)
    is_vis = O.visual_metadata(spans, Lp)[0]
    vis = np.nonzero(is_vis)[0]
    steps = []
    for _ in range(2):
        S = np.empty((2, 4, Lp), np.float32)
        for layer in range(2):
            S[layer, 0] = cluster_row(rng, Lp, vis, 0, 3000)
            S[layer, 1] = cluster_row(rng, Lp, vis, 3000, 1500)
            S[layer, 2] = np.where(rng.random(Lp) < 0.5, 1e-3, 2e-3).astype(np.float32)
            S[layer, 3] = rng.lognormal(-7, 1.5, Lp).astype(np.float32)
        steps.append(S)
    sbar = rng.uniform(1e-4, 1e-2, Lp).astype(np.float32)
    run_stats("clusters", steps, sbar, spans, 5, sk.params_default())


def test_visual_tokens_beyond_lds_cache():
    """Six 51x69 frames (N = 21114, more keys than the LDS cache): keys are
    re-read from S for every pass, with and without compaction."""
    rng = np.random.default_rng(8)
    spans, Lp = layout(6, 51, 69)
    is_vis = O.visual_metadata(spans, Lp)[0]
    vis = np.nonzero(is_vis)[0]
    S = np.empty((1, 3, Lp), np.float32)
    S[0, 0] = cluster_row(rng, Lp, vis, 2000, 1000)
    S[0, 1] = cluster_row(rng, Lp, vis, 0, 4000)
    S[0, 2] = rng.lognormal(-7, 1.5, Lp).astype(np.float32)
    sbar = rng.uniform(1e-4, 1e-2, Lp).astype(np.float32)
    run_stats("uncached", [S, S * np.float32(1.5)], sbar, spans, 6, sk.params_default())


def test_many_bins_fine_grid():
    """K = 64 equal-frequency bins on a 16 x 16 grid (the largest joint
    histogram) with a dense cluster across several edges."""
    rng = np.random.default_rng(9)
    spans, Lp = layout(3, 40, 70)
    is_vis = O.visual_metadata(spans, Lp)[0]
    vis = np.nonzero(is_vis)[0]
    S = np.empty((1, 2, Lp), np.float32)
    S[0, 0] = cluster_row(rng, Lp, vis, 500, 2500)
    S[0, 1] = rng.lognormal(-7, 1.5, Lp).astype(np.float32)
    p = sk.params_default()
    p.n_bins, p.grid = 64, 16
    sbar = rng.uniform(1e-4, 1e-2, Lp).astype(np.float32)
    run_stats("K64 M16", [S], sbar, spans, 3, p)


def test_many_bins_fine_grid_uncached():
    """K = 64 bins on a 16 x 16 grid with eight 51x69 frames (N = 28152,
    more keys than the LDS cache): the unfused joint histogram on keys read
    from S, with equal keys at several edges split by visual index."""
    rng = np.random.default_rng(10)
    spans, Lp = layout(8, 51, 69)
    is_vis = O.visual_metadata(spans, Lp)[0]
    vis = np.nonzero(is_vis)[0]
    S = np.empty((1, 3, Lp), np.float32)
    S[0, 0] = cluster_row(rng, Lp, vis, 3000, 6000)
    S[0, 1] = np.where(rng.random(Lp) < 0.4, 1e-3, 4e-3).astype(np.float32)
    S[0, 2] = rng.lognormal(-7, 1.5, Lp).astype(np.float32)
    p = sk.params_default()
    p.n_bins, p.grid = 64, 16
    sbar = rng.uniform(1e-4, 1e-2, Lp).astype(np.float32)
    run_stats("K64 M16 uncached", [S, S[:, :, ::-1].copy()], sbar, spans, 8, p, mi_tol=1e-6)


@pytest.mark.parametrize("rows,cols,K,M", [(1, 1, 8, 8), (1, 2, 8, 8), (1, 7, 8, 8),
                                            (3, 3, 8, 8), (4, 5, 1, 8), (6, 7, 8, 1),
                                            (9, 11, 64, 16)])
def test_tiny_frames_and_degenerate_bins(rows, cols, K, M):
    """Fewer visual tokens than bins (empty bins, coinciding edges), a single
    bin, a 1x1 grid: the edge selection's small-candidate path."""
    rng = np.random.default_rng(rows * 100 + cols)
    spans, Lp = layout(3, rows, cols, gap=5, head=3, tail=40)
    S = rng.lognormal(-7, 1.0, (1, 2, Lp)).astype(np.float32)
    p = sk.params_default()
    p.n_bins, p.grid = K, M
    sbar = rng.uniform(1e-4, 1e-2, Lp).astype(np.float32)
    run_stats(f"tiny {rows}x{cols} K{K} M{M}", [S, S[:, ::-1].copy()], sbar, spans, 3, p)


def test_all_scores_equal_and_two_levels():
    """Every visual key equal (no radix digit at all), and two levels with
    the edges inside the runs of equal keys."""
    spans, Lp = layout(4, 20, 30)
    S = np.empty((1, 2, Lp), np.float32)
    S[0, 0] = 3e-3
    rng = np.random.default_rng(5)
    S[0, 1] = np.where(rng.random(Lp) < 0.3, 1e-3, 4e-3).astype(np.float32)
    sbar = np.full(Lp, 1e-3, np.float32)
    run_stats("equal keys", [S, S], sbar, spans, 4, sk.params_default())


def test_ties_at_edges_with_few_candidates():
    """Continuous scores (few keys share the edges' first-digit buckets) with
    exact three-way ties at every edge rank, scattered over the frames: the
    equal keys at an edge split by visual index."""
    rng = np.random.default_rng(12)
    spans, Lp = layout(3, 20, 30)
    is_vis = O.visual_metadata(spans, Lp)[0]
    vis = np.nonzero(is_vis)[0]
    N, K = vis.size, 8
    S = np.empty((1, 2, Lp), np.float32)
    for g in range(2):
        vals = np.sort(rng.uniform(1e-3, 2e-2, N).astype(np.float32))
        for b in range(1, K):
            r = -(-b * N // K)
            vals[r - 1:r + 2] = vals[r]        # three equal keys around the edge
        row = rng.uniform(1e-3, 2e-2, Lp).astype(np.float32)
        row[vis[rng.permutation(N)]] = vals
        S[0, g] = row
    sbar = rng.uniform(1e-4, 1e-2, Lp).astype(np.float32)
    run_stats("edge ties", [S, S], sbar, spans, 3, sk.params_default())


def test_frame_above_the_fused_path_limit():
    """One 4200 x 4200 frame, N = 17.64e6 > 2^24 visual tokens: the rank pass
    takes the unfused joint histogram at its largest.  Group 0 has eight score
    levels by row band, offset by 100 rows from the grid's cell rows, so every
    edge falls inside a run of equal keys spanning whole rows and the tie rule
    (visual order) decides the bins of 420,000 tokens per edge; group 1 has
    lognormal scores rising with the row, with about 2e6 exact float32 ties.
    MI is computed in double from exact counts, so it is held to 1e-6 (a few
    float32 ulps): a misranked run of equal keys would move it far more."""
    rng = np.random.default_rng(13)
    rows = cols = 4200
    spans, Lp = layout(1, rows, cols)
    is_vis, _, r, _, _, _ = O.visual_metadata(spans, Lp)
    vis = np.nonzero(is_vis)[0]
    assert vis.size > 2 ** 24
    S = np.empty((1, 2, Lp), np.float32)
    S[0, 0] = rng.uniform(1e-3, 1e-2, Lp).astype(np.float32)
    level = np.minimum(7, (r[vis] + 100) * 8 // rows)
    S[0, 0, vis] = (1e-3 * (1 + level)).astype(np.float32)
    S[0, 1] = (rng.lognormal(-7, 1.5, Lp) * (1.0 + r / rows)).astype(np.float32)
    S2 = S.copy()
    S2[0, 1] = rng.lognormal(-7, 1.5, Lp).astype(np.float32)
    sbar = rng.uniform(1e-4, 1e-2, Lp).astype(np.float32)
    say("above 2^24: inputs generated")
    run_stats("N > 2^24", [S, S2], sbar, spans, 1, sk.params_default(), mi_tol=1e-6)


@pytest.mark.parametrize("frames,K,M,n_layers", [
    (2, 8, 8, 48), (5, 8, 8, 48), (3, 17, 16, 48), (2, 18, 8, 48),
    (2, 8, 8, 96), (5, 9, 8, 96), (1, 2, 2, 96), (3, 10, 8, 96), (2, 8, 16, 96)])
def test_more_blocks_than_cus(frames, K, M, n_layers):
    """48 layers of 4 subspaces: 288 statistics blocks, more than the GPU's
    256 CUs, so the kernel takes its narrow block shape (512 threads, two
    blocks per CU) when K <= 17, and the wide one at K = 18.  96 layers: 576
    blocks, more than two per CU, so the small shape (256 threads, four per
    CU) when K <= 9 and M*M <= 64, else the narrow one (K = 10, or M = 16).
    One or two 39x69 frames keep the keys in the narrow shape's LDS cache
    (the small shape's 2K-key cache holds none of them), five do not; every
    layer mixes dense key clusters at the edges, two-level ties and plain
    random scores."""
    rng = np.random.default_rng(frames * 100 + K + n_layers)
    spans, Lp = layout(frames, 39, 69)
    is_vis = O.visual_metadata(spans, Lp)[0]
    vis = np.nonzero(is_vis)[0]
    G = 4
    steps = []
    for _ in range(2):
        S = np.empty((n_layers, G, Lp), np.float32)
        for layer in range(n_layers):
            S[layer, 0] = cluster_row(rng, Lp, vis, vis.size // 7, vis.size // 5)
            S[layer, 1] = np.where(rng.random(Lp) < 0.4, 1e-3, 4e-3).astype(np.float32)
            S[layer, 2] = rng.lognormal(-7, 1.5, Lp).astype(np.float32)
            S[layer, 3] = cluster_row(rng, Lp, vis, 0, 700)
        steps.append(S)
    p = sk.params_default()
    p.n_bins, p.grid = K, M
    sbar = rng.uniform(1e-4, 1e-2, Lp).astype(np.float32)
    run_stats(f"{n_layers} layers K{K} M{M} {frames} frames", steps, sbar, spans, frames, p)


@pytest.mark.parametrize("G", [8, 9, 17, 64])
def test_stability_blocks_over_many_subspaces(G):
    """A layer's stability means are split over ceil(G/8) blocks of eight
    subspaces: 8 (one block), 9 (the second block holds one subspace), 17
    and 64 (eight blocks).  Three layers, two steps (the second step's phi
    reads the means the first wrote), every subspace's MI and phi against
    the oracle."""
    rng = np.random.default_rng(900 + G)
    spans, Lp = layout(2, 23, 31)
    n_layers = 3
    steps = []
    for _ in range(2):
        S = rng.lognormal(-7, 1.5, (n_layers, G, Lp)).astype(np.float32)
        S[:, ::3, 1::4] = S[:, ::3, ::4][:, :, :S[:, ::3, 1::4].shape[2]]   # exact ties
        steps.append(S)
    sbar = rng.uniform(1e-4, 1e-2, Lp).astype(np.float32)
    run_stats(f"G={G} stability blocks", steps, sbar, spans, 2, sk.params_default())


@pytest.mark.parametrize("mixed", [False, True])
def test_sixty_four_spans(mixed):
    """The largest span count the boundary accepts (64): equal 7x9 frames,
    or frames of mixed shapes from 1x1 to 13x17 with gaps of 0 to 40 text
    tokens; the keys fit the wide shape's LDS cache, so the joint histogram
    walks them span by span."""
    rng = np.random.default_rng(64 + mixed)
    if mixed:
        spans, t = [], int(rng.integers(0, 30))
        for f in range(1, 65):
            rows, cols = int(rng.integers(1, 14)), int(rng.integers(1, 18))
            spans.append((t, rows, cols, f))
            t += rows * cols + int(rng.integers(0, 41))
        Lp = t + 17
    else:
        spans, Lp = layout(64, 7, 9, gap=5)
    G, n_layers = 4, 3
    steps = []
    for _ in range(2):
        S = rng.lognormal(-7, 1.5, (n_layers, G, Lp)).astype(np.float32)
        S[:, 1, 2::5] = S[:, 1, 1::5][:, :S[:, 1, 2::5].shape[1]]   # exact ties
        steps.append(S)
    sbar = rng.uniform(1e-4, 1e-2, Lp).astype(np.float32)
    for K, M in [(8, 8), (5, 3)]:
        p = sk.params_default()
        p.n_bins, p.grid = K, M
        run_stats(f"64 spans mixed={mixed} K{K} M{M}", steps, sbar, spans, 64, p)
