"""starkv_score_noalloc against starkv_score through the C ABI.

The allocation-free entry point runs the same kernels with the library's own
device workspace, so on identical inputs its S, sbar and g* must equal
starkv_score's bit for bit.  Two calls in a row, the second on a smaller
problem, also show that a call does not depend on what the previous one
left in the shared array.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2606_01790_amd import starkv as sk  # noqa: E402
from paper_2606_01790_amd import workload as WL  # noqa: E402
from paper_2606_01790_amd.pipeline import to_device  # noqa: E402

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[no-alloc] {msg}", flush=True)


def both_paths(seed, n_layers, H, G, d, L, W, dtype):
    Q, K, _ = WL.random_case(seed, n_layers, H, G, d, L, W, dtype)
    dev = torch.device("cuda")
    q, k = to_device(Q, dtype, dev), to_device(K, dtype, dev)
    dt = sk.BF16 if dtype == "bf16" else sk.F32
    dims = sk.make_dims(n_layers, H, G, d, L, W, dt)
    lay = sk.contiguous_layout(k, dims)
    p = sk.params_default()
    Lp = L - W
    out = {}
    for name in ("ws", "noalloc"):
        S = torch.full((n_layers * G * Lp,), -1.0, dtype=torch.float32, device=dev)
        sbar = torch.full((n_layers * Lp,), -1.0, dtype=torch.float32, device=dev)
        gstar = torch.full((n_layers * Lp,), 255, dtype=torch.uint8, device=dev)
        if name == "ws":
            ws = torch.zeros(sk.workspace_bytes(dims), dtype=torch.uint8, device=dev)
            sk.score(dims, p, q, k, lay, S, sbar, gstar, ws)
        else:
            sk.score_noalloc(dims, p, q, k, lay, S, sbar, gstar)
        torch.cuda.synchronize()
        out[name] = (S.cpu().numpy(), sbar.cpu().numpy(), gstar.cpu().numpy())
    return out


def check_equal(out):
    for a, b, what in zip(out["ws"], out["noalloc"], ("S", "sbar", "gstar")):
        assert np.array_equal(a, b), f"{what} differs from starkv_score"
    assert (out["noalloc"][0] > 0).all()


def test_noalloc_matches_workspace_call_twice_shrinking():
    # a 28-layer, five-frame 1080p-sized step, then a smaller problem
    say("28 layers, L 2947, W 32, bf16 (slab pass 2)")
    check_equal(both_paths(11, 28, 28, 4, 128, 2947, 32, "bf16"))
    say("4 layers, L 777, W 32, bf16")
    check_equal(both_paths(12, 4, 28, 4, 128, 777, 32, "bf16"))


def test_noalloc_other_kernel_paths():
    # the tile passes (fp32, d = 64) through the same array
    say("1 layer fp32 d 64, L 256, W 8")
    check_equal(both_paths(13, 1, 4, 2, 64, 256, 8, "f32"))
    say("2 layers bf16 d 64, L 600, W 16")
    check_equal(both_paths(14, 2, 8, 2, 64, 600, 16, "bf16"))
