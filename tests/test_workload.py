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
