"""Synthetic workload generator and the traffic/flop counters (CPU)."""

import json
import math
import os

import numpy as np
import pytest

from oracle import starkv_oracle as O
from paper_2606_01790_amd import workload as WL

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_flop_counter_reproduces_paper_table():
    """tab:flops: QK^T = 2 H W L d and Gather+Concat = H L d at the
    inferred workload (H=28, W=8, L=2500, d=128)."""
    g = json.load(open(os.path.join(GOLDEN, "flops_table.json")))
    w = g["inferred_workload"]
    qk = WL.qk_flops(w["H"], w["W"], w["L"], w["d"])
    assert qk / 1e6 == pytest.approx(g["mflops"]["qk_t"], abs=5e-3)
    assert w["H"] * w["L"] * w["d"] / 1e6 == pytest.approx(g["mflops"]["gather_concat"], abs=5e-3)
    # head-wise top-k of SnapKV, H L log2 k
    assert w["H"] * w["L"] * math.log2(w["k"]) / 1e6 == pytest.approx(
        g["mflops"]["topk_headwise_snapkv"], abs=5e-3)


def test_oracle_defaults_are_the_papers():
    g = json.load(open(os.path.join(GOLDEN, "hparams.json")))
    p = O.Params()
    assert p.lam == g["lambda"]
    assert p.n_warmup == g["online_profiling_steps"]
    assert p.n_ramp == g["lambda_ramp_steps"]
    assert p.rho_mi == g["mi_ema_decay"]
    assert p.tau == g["prior_temperature_tau"]
    assert p.rho_t == g["temporal_ema_decay"]
    assert p.delta == g["temporal_delta"]
    assert p.d_min == g["temporal_d_min"]
    assert [p.t_min, p.t_max] == g["aeb_t_range"]["ScreenSpot-Pro/UI-TARS"]


def test_config_shapes_and_budgets():
    s3 = WL.SPECS[3]
    assert [s3.budgets(s)[0] for s in range(1, 6)] == [538, 1076, 1614, 2152, 2691]
    assert s3.L(5) == 13711 and s3.L_p(5) == 13679 and s3.n_vis(5) == 13455
    assert WL.SPECS[1].budgets(1) == [38]
    assert WL.SPECS[2].L_p(1) == 2915 and WL.SPECS[2].budgets(1) == [538]
    assert WL.SPECS[4].budgets(15) == [4036, 8073, 16146]
    s5 = WL.SPECS[5]
    assert (s5.L(30), s5.n_vis(30), s5.budgets(30)) == (140254, 139230, [13923])


def test_bytes_alg_config3_total():
    """Sum over the 28 layers and 5 steps of config 3."""
    s3 = WL.SPECS[3]
    tot = sum(WL.bytes_alg(s3, s, s3.budgets(s)[0]) * s3.n_layers for s in range(1, 6))
    assert tot == 2166471440


def test_bf16_rounding_ties_to_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5],
                 dtype=np.float32)
    back = WL.bf16_bits_to_f32(WL.f32_to_bf16_bits(x))
    np.testing.assert_array_equal(back, [1.0, 1.0, 1.0 + 2 ** -6, 1.0, -2.5])
    torch = pytest.importorskip("torch")
    r = np.random.default_rng(0).standard_normal(10 ** 5).astype(np.float32) * 100
    want = torch.from_numpy(r).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(WL.f32_to_bf16_bits(r), want)


def test_generator_is_deterministic_and_cache_grows_by_append():
    t1 = WL.Trajectory(WL.SPECS[3])
    t2 = WL.Trajectory(WL.SPECS[3])
    k1, v1 = t1.layer_cache(5, 2)
    k2, v2 = t2.layer_cache(5, 2)
    np.testing.assert_array_equal(k1, k2)
    np.testing.assert_array_equal(v1, v2)
    assert k1.dtype == np.uint16 and k1.shape == (4, 2 * 2691 + 256, 128)
    k3, _ = t1.layer_cache(5, 3)
    np.testing.assert_array_equal(k3[:, :2 * 2691], k1[:, :2 * 2691])
    q = t1.window_q(5, 2)
    assert q.shape == (28, 32, 128)


def test_bump_centres_repeat_across_frames():
    t = WL.Trajectory(WL.SPECS[3])
    same = 0
    for f in range(2, 40):
        same += np.allclose(t.centres(0, f)[0], t.centres(0, f - 1)[0])
    assert 15 <= same <= 37      # about 70% of frames keep their places


def test_image_slots_and_resolution_change_bookkeeping():
    """image_slots = 5 with a 1920x1080 -> 1280x720 switch at frame 7: the
    context holds the newest five frames, spans tile the visual prefix in
    frame order, and L, N_vis and B follow the frames actually present."""
    sp = WL.SPECS[6]
    assert sp.frames(3) == [1, 2, 3]
    assert sp.frames(6) == [2, 3, 4, 5, 6]
    assert sp.frames(10) == [6, 7, 8, 9, 10]
    assert sp.grid(6) == (69, 39) and sp.grid(7) == (46, 26)
    assert sp.n_frame == 2691 and not sp.appends
    for s in range(1, sp.steps + 1):
        spans = sp.spans(s)
        t = 0
        for (start, rows, cols, f), want in zip(spans, sp.frames(s)):
            assert start == t and f == want and (cols, rows) == sp.grid(f)
            t += rows * cols
        assert t == sp.n_vis(s) and sp.L(s) == t + sp.text
        assert sp.budgets(s) == [20 * t // 100]
    assert sp.L(10) == 2691 + 4 * 46 * 26 + 256
    assert sp.peak_step == 5        # steps 5 and 6 tie; the first is taken


def test_frames_keep_their_bytes_when_they_move():
    """A frame's K/V bytes depend only on (layer, frame): after the oldest
    frames leave the context, frame 7 sits at position 0 .. with its own
    bytes, and the single-resolution configurations are unchanged by the
    per-frame grid (frame 3 of config 3 starts at 2 * 2691)."""
    t6 = WL.Trajectory(WL.SPECS[6])
    k10, v10 = t6.layer_cache(2, 10)
    k7, v7 = t6.frame_kv(2, 7)
    n6 = 2691
    np.testing.assert_array_equal(k10[:, n6:n6 + 46 * 26], k7)
    np.testing.assert_array_equal(v10[:, n6:n6 + 46 * 26], v7)
    k6, _ = t6.frame_kv(2, 6)
    np.testing.assert_array_equal(k10[:, :n6], k6)
    t3 = WL.Trajectory(WL.SPECS[3])
    k, _ = t3.layer_cache(1, 4)
    np.testing.assert_array_equal(k[:, 2 * 2691:3 * 2691], t3.frame_kv(1, 3)[0])


def test_bench_roofline_bound_follows_intensity():
    """The scoring call is HBM-bound at W = 32 (224 flop per K byte, below
    the bf16 ridge of 312.5) and MFMA-bound at W = 64 (448); fp32 inputs take
    the fp32 peak, whose ridge is 19.7."""
    import bench
    cases = [(3, "hbm"), (5, "mfma"), (1, "hbm")]
    for cid, bound in cases:
        spec = WL.SPECS[cid]
        s = spec.steps
        b = bench.call_bytes(spec, s, "score")
        f = spec.n_layers * WL.qk_flops(spec.H, spec.W, spec.L_p(s), spec.d)
        r = bench.roofline_of(1e-3, b, f, spec.dtype)
        assert r["bound"] == bound, (cid, r)
        if bound == "mfma":
            assert r["peak"] == 2500.0 and r["unit"] == "TFLOP/s"
            assert abs(r["achieved"] - f / 1e-3 / 1e12) < 0.1
        else:
            assert r["unit"] == "GB/s" and abs(r["achieved"] - b / 1e-3 / 1e9) < 0.1
    assert bench.roofline_of(1.0, 1, 10 ** 6, "f32")["peak"] == 157.3


def test_bench_fused_call_bytes_and_traffic_guard(tmp_path, monkeypatch):
    """The fused statistics-and-selection call is credited with the bytes of
    the two calls it replaces; a traffic summary is used only while the
    scoring sources hash to the version it was taken on."""
    import bench
    spec = WL.SPECS[3]
    for s in range(1, spec.steps + 1):
        assert bench.call_bytes(spec, s, "update_state_select") == (
            bench.call_bytes(spec, s, "update_state") + bench.call_bytes(spec, s, "select"))
    wl = spec.name
    prof = tmp_path / "profiles"
    prof.mkdir()
    f = prof / f"starkv_score-{wl}.traffic.md"
    f.write_text("- traffic_bytes_per_launch: 123\n- sources_sha1: abc\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "sources_sha1", lambda call: "abc")
    assert bench.measured_traffic("starkv_score", wl) == 123
    f.write_text("- traffic_bytes_per_launch: 123\n- sources_sha1: 0000\n")
    assert bench.measured_traffic("starkv_score", wl) is None
    assert bench.measured_traffic("starkv_compact", wl) is None
