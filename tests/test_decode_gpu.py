"""GPU parity of decode attention over the cache (starkv_decode) against the
fp64 oracle (oracle.decode_attention).

Bar: per output element, |o_gpu - o_ref| <= 1e-3 * sum_t p_t |v_t| + 1e-6,
with p the oracle's softmax weights.  Logits are fp32 MFMA sums of exact
bf16 products, the softmax and the P.V sums run in fp32, so the error is a
small multiple of 2^-24 times the number of terms added, relative to the
weighted L1 mass of the value column.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import starkv_oracle as O  # noqa: E402
from paper_2606_01790_amd import starkv as sk  # noqa: E402
from paper_2606_01790_amd import workload as WL  # noqa: E402
from paper_2606_01790_amd.pipeline import TrajectoryRunner  # noqa: E402

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[decode] {msg}", flush=True)


def bound(q, K, V):
    """1e-3 * sum_t p_t |v_t| per output element, from the oracle's weights."""
    H, d = q.shape
    G = K.shape[0]
    out = np.zeros((H, d))
    for h in range(H):
        g = h * G // H
        x = K[g] @ q[h] / np.sqrt(d)
        p = np.exp(x - x.max())
        p /= p.sum()
        out[h] = p @ np.abs(V[g])
    return 1e-3 * out + 1e-6


def run_decode(tag, q_bits, k_bits, v_bits, n_tok, H, G, d, token_stride=None):
    """q_bits [nl, H, d], k_bits/v_bits [nl, G, n_cap, d] bf16 bit patterns."""
    nl = q_bits.shape[0]
    dev = torch.device("cuda:0")
    dims = sk.make_dims(nl, H, G, d, n_tok + 1, 1, sk.BF16)
    q = torch.from_numpy(q_bits.view(np.int16)).to(dev)
    k = torch.from_numpy(k_bits.view(np.int16)).to(dev)
    v = torch.from_numpy(v_bits.view(np.int16)).to(dev)
    n_cap = k_bits.shape[2]
    ts = token_stride or d
    if ts != d:     # a strided cache: rows padded to token_stride elements
        pad = torch.zeros((nl, G, n_cap, ts), dtype=torch.int16, device=dev)
        pad[..., :d] = k
        k = pad.clone()
        pad[..., :d] = v
        v = pad
    lay = sk.KVLayout(G * n_cap * ts, n_cap * ts, ts)
    out = torch.zeros(nl * H * d, dtype=torch.float32, device=dev)
    ws = torch.zeros(max(sk.decode_workspace_bytes(dims, n_tok), 16), dtype=torch.uint8,
                     device=dev)
    say(f"{tag}: layers={nl} H={H} G={G} d={d} n={n_tok} stride={ts}")
    sk.decode(dims, q, k, v, lay, n_tok, out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy().reshape(nl, H, d)
    worst = 0.0
    for layer in range(nl):
        qf = WL.to_float64(q_bits[layer], "bf16")
        Kf = WL.to_float64(k_bits[layer][:, :n_tok], "bf16")
        Vf = WL.to_float64(v_bits[layer][:, :n_tok], "bf16")
        want = O.decode_attention(qf, Kf, Vf)
        err = np.abs(got[layer] - want)
        tol = bound(qf, Kf, Vf)
        assert np.all(err <= tol), f"{tag} L{layer}: max err {err.max()} (tol {tol.min()})"
        worst = max(worst, float((err / tol).max()))
    say(f"{tag}: ok, worst err / bound {worst:.3f}")
    return got


def random_bits(seed, shape, scale=1.0):
    r = np.random.default_rng([seed, 91])
    return WL.f32_to_bf16_bits(r.standard_normal(shape, dtype=np.float32) * np.float32(scale))


@pytest.mark.parametrize("H,G,d,n", [(28, 4, 128, 2723), (28, 4, 128, 1), (8, 8, 64, 31),
                                     (16, 1, 128, 33), (14, 2, 64, 5000), (4, 2, 128, 1024)])
def test_decode_random_caches(H, G, d, n):
    """Token counts around the 32-token tiles, the 4-wave rounds and the
    split size; 1, 2, 7, 8 and 16 heads per group; d = 64 and 128."""
    nl = 2
    q = random_bits(H * 100 + n, (nl, H, d))
    k = random_bits(H * 100 + n + 1, (nl, G, n + 3, d))
    v = random_bits(H * 100 + n + 2, (nl, G, n + 3, d))
    run_decode(f"random H{H} G{G}", q, k, v, n, H, G, d)


def test_decode_strided_cache_and_peaked_attention():
    """Rows padded to 192 elements; queries scaled up so that a few tokens
    take nearly all the weight (large logits, the max subtraction matters)."""
    H, G, d, n, nl = 28, 4, 128, 3000, 1
    q = random_bits(7, (nl, H, d), scale=4.0)
    k = random_bits(8, (nl, G, n, d), scale=2.0)
    v = random_bits(9, (nl, G, n, d))
    run_decode("peaked strided", q, k, v, n, H, G, d, token_stride=192)


def test_decode_zero_query_is_the_value_mean():
    """q = 0: every weight is exactly 1/n on both sides, so the output is the
    mean of the value rows up to fp32 summation."""
    H, G, d, n = 8, 2, 128, 2000
    q = np.zeros((1, H, d), dtype=np.uint16)
    k = random_bits(11, (1, G, n, d))
    v = random_bits(12, (1, G, n, d))
    got = run_decode("zero query", q, k, v, n, H, G, d)
    mean = WL.to_float64(v[0], "bf16").mean(axis=1)
    for h in range(H):
        assert np.max(np.abs(got[0, h] - mean[h * G // H])) <= 1e-5


def test_decode_reuses_one_workspace():
    """Calls in a row on one workspace, left as the previous call wrote it,
    with token counts that change the number of splits (1, 11, 3 and 20
    splits, so each call's partials cover a different range)."""
    H, G, d, nl = 28, 4, 128, 2
    n_max = 5000
    dev = torch.device("cuda:0")
    q = random_bits(31, (nl, H, d))
    k = random_bits(32, (nl, G, n_max, d))
    v = random_bits(33, (nl, G, n_max, d))
    dims = sk.make_dims(nl, H, G, d, n_max + 1, 1, sk.BF16)
    ws = torch.zeros(sk.decode_workspace_bytes(dims, n_max), dtype=torch.uint8, device=dev)
    qd = torch.from_numpy(q.view(np.int16)).to(dev)
    kd = torch.from_numpy(k.view(np.int16)).to(dev)
    vd = torch.from_numpy(v.view(np.int16)).to(dev)
    lay = sk.KVLayout(G * n_max * d, n_max * d, d)
    for n in (200, 2723, 700, n_max):
        out = torch.zeros(nl * H * d, dtype=torch.float32, device=dev)
        sk.decode(dims, qd, kd, vd, lay, n, out, ws)
        torch.cuda.synchronize()
        got = out.cpu().numpy().reshape(nl, H, d)
        for layer in range(nl):
            qf = WL.to_float64(q[layer], "bf16")
            Kf = WL.to_float64(k[layer][:, :n], "bf16")
            Vf = WL.to_float64(v[layer][:, :n], "bf16")
            err = np.abs(got[layer] - O.decode_attention(qf, Kf, Vf))
            assert np.all(err <= bound(qf, Kf, Vf)), f"n={n} L{layer}: max err {err.max()}"
        say(f"reused workspace: n={n} ok")


def test_decode_on_compressed_cache_of_the_stage():
    """The stage's own K'/V' (one 1920x1080 frame, Qwen2.5-VL-7B shape, top
    20%): decode over the B + W kept rows against the oracle on the same
    rows; with B = L_p (everything kept) the compressed cache is the full
    cache, and decoding over either gives bit-identical outputs."""
    spec = WL.SPECS[2]
    p = sk.params_default()
    r = TrajectoryRunner(spec, p, max_budget=spec.L_p(1))
    r.reset()
    r.load_step(1)
    H, G, d, W = spec.H, spec.G, spec.d, spec.W
    q = random_bits(21, (1, H, d))
    qd = torch.from_numpy(q.view(np.int16)).to("cuda")
    dev = torch.device("cuda:0")
    for B in (spec.budgets(1)[0], spec.L_p(1)):
        r.run_step(1, B)
        torch.cuda.synchronize()
        out = r.outputs(1, B)
        n = B + W
        say(f"stage K'/V' with B={B}")
        run_decode(f"K'V' B={B}", q, out["k_out"], out["v_out"], n, H, G, d)
    # B = L_p: K' equals the cache; compare the two decodes bit for bit
    L = spec.L(1)
    dims = sk.make_dims(1, H, G, d, L, W, sk.BF16)
    ws = torch.zeros(sk.decode_workspace_bytes(dims, L), dtype=torch.uint8, device=dev)
    o_full = torch.zeros(H * d, dtype=torch.float32, device=dev)
    o_comp = torch.zeros_like(o_full)
    sk.decode(dims, qd, r.K, r.V, r.layout, L, o_full, ws)
    n_out = G * L * d
    lay_c = sk.KVLayout(G * L * d, L * d, d)
    sk.decode(dims, qd, r.k_out[:n_out], r.v_out[:n_out], lay_c, L, o_comp, ws)
    torch.cuda.synchronize()
    assert torch.equal(o_full, o_comp)
