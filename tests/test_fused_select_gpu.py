"""starkv_update_state_select against starkv_update_state then starkv_select.

The fused call promises the two calls' outputs bit for bit: the scalars, the
state (MI_bar, the stability means, the counters), the final scores s and
the selected indices.  Each case runs both on twin states over several
steps of synthetic score rows and compares every output word.  The cases
cover the fused shape (one block per CU, the selection in the finalizing
block), its LDS key cache (a prefix of L_p that is smaller than the
selection kernel's own), budgets 0 and L_p, the narrow-shape and per-head
fallbacks (two launches), frames of changing size (the stability means
restart), a layer whose state block does not match (NaN scalars), and the
temporal-decay and AEB variants.  The
oracle parity of each half is covered by the statistics and selection
tests; this one pins the fusion.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2606_01790_amd import starkv as sk  # noqa: E402

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[fused] {msg}", flush=True)


def layout(n_frames, rows, cols, gap=37, head=50, tail=100):
    spans, t = [], head
    for f in range(1, n_frames + 1):
        spans.append((t, rows, cols, f))
        t += rows * cols + gap
    return spans, t - gap + tail


def bits(t):
    return t.contiguous().view(torch.int32).cpu().numpy()


def run_pair(tag, n_layers, H, G, steps, B, p=None, per_head=False, spoil_layer=None,
             seed=0):
    """steps: list of (spans, frame, Lp); Lp fixed over the steps.  Compares
    the fused call with the two separate calls after every step."""
    rng = np.random.default_rng(seed)
    Lp = steps[0][2]
    W = 8
    dims = sk.make_dims(n_layers, H, G, 64, Lp + W, W, sk.BF16, per_head=per_head)
    Ns = H if per_head else G
    p = p or sk.params_default()
    cap = max([s[1] * s[2] for spans, _, _ in steps for s in spans] + [1])
    dev = torch.device("cuda:0")
    states = [torch.empty(sk.state_bytes(dims, cap), dtype=torch.uint8, device=dev)
              for _ in range(2)]
    for st in states:
        sk.state_init(dims, st, cap)
    if spoil_layer is not None:
        stride = sk.state_bytes(dims, cap) // n_layers
        for st in states:   # the header's magic word: the layer no longer matches
            st[spoil_layer * stride:spoil_layer * stride + 4].zero_()
    nsc = n_layers * sk.scalars_count(dims)
    scal = [torch.empty(nsc, dtype=torch.float32, device=dev) for _ in range(2)]
    s_out = [torch.empty(n_layers * Lp, dtype=torch.float32, device=dev) for _ in range(2)]
    idx = [torch.empty(max(1, n_layers * B), dtype=torch.int32, device=dev) for _ in range(2)]
    say(f"{tag}: layers={n_layers} Ns={Ns} Lp={Lp} B={B} steps={len(steps)}")
    for k, (spans, frame, _) in enumerate(steps, 1):
        S = rng.lognormal(-7, 1.5, (n_layers, Ns, Lp)).astype(np.float32)
        S[:, :, 1::5] = S[:, :, ::5][:, :, :S[:, :, 1::5].shape[2]]   # exact ties
        sbar = rng.lognormal(-7, 1.2, (n_layers, Lp)).astype(np.float32)
        sbar[:, 3::7] = sbar[:, 2::7][:, :sbar[:, 3::7].shape[1]]
        gstar = rng.integers(0, Ns, (n_layers, Lp)).astype(np.uint8)
        S_d, sbar_d, g_d = (torch.from_numpy(x).to(dev) for x in (S, sbar, gstar))
        for x in scal + s_out + idx:
            x.fill_(-1.0 if x.dtype == torch.float32 else -1)
        sk.update_state(dims, p, S_d, sbar_d, spans, frame, states[0], cap, scal[0])
        sk.select(dims, p, sbar_d, g_d, scal[0], spans, frame, B, s_out[0],
                  idx[0] if B else None)
        sk.update_state_select(dims, p, S_d, sbar_d, g_d, spans, frame, states[1], cap,
                               scal[1], B, s_out[1], idx[1] if B else None)
        torch.cuda.synchronize()
        for name, a, b in (("scalars", scal[0], scal[1]), ("s", s_out[0], s_out[1]),
                           ("idx", idx[0], idx[1])):
            x, y = bits(a), bits(b)
            bad = np.nonzero(x != y)[0]
            assert bad.size == 0, f"{tag} step {k}: {name} differs at {bad[:8]} " \
                                  f"({x[bad[:4]]} vs {y[bad[:4]]})"
        assert torch.equal(states[0], states[1]), f"{tag} step {k}: state differs"
        if spoil_layer is not None:
            sc = scal[1].view(n_layers, -1)
            assert torch.isnan(sc[spoil_layer]).all(), f"{tag}: spoiled layer not NaN"
            others = torch.cat([sc[:spoil_layer], sc[spoil_layer + 1:]])
            assert not torch.isnan(others).any(), f"{tag}: NaN outside the spoiled layer"
    say(f"{tag}: ok")


def test_fused_matches_two_calls_five_frames():
    """28 layers, 4 groups, five 39x69 frames (the selection's keys all in
    the LDS cache), budget 20%, the current frame moving forward (a frame's
    span is given from the step it becomes current)."""
    spans, Lp = layout(5, 39, 69)
    steps = [(spans[:f], f, Lp) for f in (3, 4, 4, 5)]
    run_pair("five frames", 28, 28, 4, steps, B=int(0.2 * Lp))


@pytest.mark.parametrize("B", [0, 1, "all"])
def test_fused_budget_extremes(B):
    spans, Lp = layout(3, 23, 31)
    steps = [(spans, 3, Lp)] * 2
    run_pair(f"B={B}", 28, 28, 4, steps, B=Lp if B == "all" else B, seed=7)


def test_fused_keys_beyond_the_cache():
    """L_p above both key caches (the fused one is the smaller): the
    selection reads the keys it does not cache from s."""
    spans, Lp = layout(4, 96, 96)
    assert Lp > 28 * 1024
    steps = [(spans, 4, Lp)] * 2
    run_pair("Lp beyond cache", 6, 8, 2, steps, B=Lp // 10, seed=3)


def test_fused_frame_size_changes():
    """A frame of another size becomes current: the stability means restart
    in both paths alike."""
    a, Lp = layout(2, 30, 40)
    b = [(a[0][0], 30, 40, 1), (a[1][0], 20, 50, 2)]
    c = [(a[0][0], 30, 40, 1), (a[1][0], 24, 50, 2)]
    steps = [(a, 2, Lp), (b, 2, Lp), (c, 2, Lp), (c, 2, Lp)]
    run_pair("frame size changes", 12, 12, 4, steps, B=Lp // 3, seed=5)


def test_fused_narrow_fallback():
    """48 layers of 4 subspaces at K = 8: more statistics blocks than CUs,
    so the statistics take the 512-thread shape and the call queues the
    selection kernel after them."""
    spans, Lp = layout(2, 39, 69)
    p = sk.params_default()
    p.n_bins, p.grid = 8, 8
    run_pair("narrow", 48, 48, 4, [(spans, 2, Lp)] * 2, B=Lp // 5, p=p, seed=11)


def test_fused_per_head():
    """Per-head subspaces (Ns = H = 28) of 4 KV groups."""
    spans, Lp = layout(3, 39, 69)
    run_pair("per head", 28, 28, 4, [(spans, 3, Lp)] * 2, B=Lp // 5, per_head=True, seed=13)


def test_fused_mismatched_state_layer():
    """A layer whose state block fails the header check gets NaN scalars
    and its selection runs on them, in both paths alike."""
    spans, Lp = layout(2, 23, 31)
    run_pair("spoiled layer", 8, 8, 2, [(spans, 2, Lp)] * 2, B=Lp // 4, spoil_layer=3,
             seed=17)


@pytest.mark.parametrize("tem,aeb", [("linear", "entropy"), ("gamma", "confidence"),
                                     ("exp", "confidence")])
def test_fused_ablation_variants(tem, aeb):
    """The temporal-decay and AEB variants (the discount table and the
    temperature of the fused selection), with the prior active from the
    first step."""
    spans, Lp = layout(4, 39, 69)
    p = sk.params_default()
    p.tem_decay = sk.TEM_DECAY[tem]
    p.aeb_mode = sk.AEB_MODE[aeb]
    p.n_warmup, p.n_ramp = 0, 0
    steps = [(spans[:f], f, Lp) for f in (2, 3, 4)]
    run_pair(f"{tem}/{aeb}", 28, 28, 4, steps, B=Lp // 4, p=p, seed=19)


@pytest.mark.parametrize("seed", range(16))
def test_fused_random_configurations(seed):
    """Sixteen seeded draws of layers, subspaces, frames, budget, bins, grid
    and variants (the wide shape's fused path when the blocks fit one per
    CU, the queued kernels otherwise)."""
    rng = np.random.default_rng(500 + seed)
    G = int(rng.choice([1, 2, 4, 8]))
    hpg = int(rng.choice([1, 2, 7]))
    per_head = bool(rng.random() < 0.25) and G * hpg <= 64
    n_layers = int(rng.integers(1, 40))
    spans, t = [], int(rng.integers(0, 40))
    for f in range(1, int(rng.integers(1, 5)) + 1):
        rows, cols = int(rng.integers(2, 60)), int(rng.integers(2, 70))
        spans.append((t, rows, cols, f))
        t += rows * cols + int(rng.integers(0, 60))
    Lp = t + int(rng.integers(1, 80))
    p = sk.params_default()
    p.n_bins = int(rng.integers(1, 25))
    p.grid = int(rng.integers(1, 13))
    p.tem_decay = sk.TEM_DECAY[str(rng.choice(list(sk.TEM_DECAY)))]
    p.aeb_mode = sk.AEB_MODE[str(rng.choice(list(sk.AEB_MODE)))]
    if rng.random() < 0.5:
        p.n_warmup, p.n_ramp = 0, 0
    steps = [(spans[:f], f, Lp) for f in range(1, len(spans) + 1)]
    run_pair(f"random {seed}", n_layers, G * hpg, G, steps, B=int(rng.integers(0, Lp + 1)),
             p=p, per_head=per_head, seed=seed)


def test_fused_no_visual_tokens():
    """No spans (a text-only context): the statistics have no visual keys
    and no current frame; the selection applies no discount."""
    run_pair("no spans", 12, 12, 4, [([], 0, 3000)] * 2, B=600, seed=23)


@pytest.mark.parametrize("n_layers,H,G", [(10, 18, 9), (8, 32, 16)])
def test_fused_several_stability_blocks(n_layers, H, G):
    """9 and 16 subspaces: two stability blocks per layer, the layer's
    finalize (and then its selection) in whichever block arrives last, still
    the wide fused shape (120 and 152 blocks)."""
    spans, Lp = layout(3, 23, 31)
    steps = [(spans[:f], f, Lp) for f in (2, 3, 3)]
    run_pair(f"G={G} stability blocks", n_layers, H, G, steps, B=Lp // 5, seed=29 + G)


def test_fused_sixty_four_spans():
    """64 frames of 5x6 (the span limit): the selection's discount table
    holds 64 spans per subspace."""
    spans, Lp = layout(64, 5, 6, gap=3)
    steps = [(spans[:f], f, Lp) for f in (63, 64)]
    run_pair("64 spans", 12, 12, 4, steps, B=Lp // 5, seed=64)
