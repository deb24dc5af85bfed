"""The online state on the GPU: checkpoint and resume, and state blocks that
do not match the call.

The state is a caller-owned device block (sec. 3.2: per-layer statistics
kept across the steps of one trajectory, reset per trajectory), so a
trajectory can be checkpointed by copying it out and resumed by copying it
back.  Results are bitwise deterministic, so a resumed trajectory must
reproduce the uninterrupted one bit for bit.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2606_01790_amd import starkv as sk  # noqa: E402
from paper_2606_01790_amd import workload as WL  # noqa: E402
from paper_2606_01790_amd.pipeline import ArrayCase, TrajectoryRunner  # noqa: E402

pytestmark = pytest.mark.gpu

KEYS = ("S", "sbar", "gstar", "s", "idx", "scal", "k_out", "v_out")


def say(msg):
    print(f"[state] {msg}", flush=True)


def _params():
    p = sk.params_default()
    p.t_min, p.t_max = 0.95, 1.05
    p.n_warmup, p.n_ramp = 1, 2          # the prior switches on inside the run
    return p


def _run(runner, steps, spec):
    out = {}
    for step in steps:
        B = spec.budgets(step)[0]
        runner.load_step(step)
        runner.run_step(step, B)
        torch.cuda.synchronize()
        out[step] = runner.outputs(step, B)
    return out


def test_checkpoint_and_resume_is_bit_exact():
    spec = WL.SPECS[3]                   # 28 layers, five 1920x1080 frames
    p = _params()
    say("uninterrupted five-step trajectory")
    ref_runner = TrajectoryRunner(spec, p)
    ref_runner.reset()
    ref = _run(ref_runner, range(1, 6), spec)
    ref_state = ref_runner.state.cpu()
    del ref_runner

    say("steps 1-2, checkpoint, re-initialise, restore, steps 3-5")
    r = TrajectoryRunner(spec, p)
    r.reset()
    _run(r, range(1, 3), spec)
    snap = r.state.cpu().clone()         # checkpoint: a plain byte copy
    r.reset()                            # a fresh trajectory state ...
    torch.cuda.synchronize()
    assert not torch.equal(r.state.cpu(), snap)
    r.state.copy_(snap.to(r.device))     # ... overwritten by the checkpoint
    got = _run(r, range(3, 6), spec)
    for step in range(3, 6):
        for key in KEYS:
            assert np.array_equal(got[step][key], ref[step][key]), (step, key)
    # the state itself carried on identically
    say("state after step 5")
    assert torch.equal(r.state.cpu(), ref_state)


@pytest.mark.parametrize("kind", ["frame_cap", "uninitialised"])
def test_mismatched_state_is_left_untouched(kind):
    H, G, d, W, nl = 28, 4, 128, 32, 3
    nr, nc, text = 12, 20, 64
    nf = nr * nc
    L = nf + text
    Q, K, V = WL.random_case(31, nl, H, G, d, L, W, "bf16")
    p = sk.params_default()
    spans = [(0, nr, nc, 1)]
    cap = 2 * nf
    case = ArrayCase(H, G, d, W, nl, L, "bf16", p, frame_cap=cap)
    dims = case.dims(L)
    if kind == "frame_cap":
        say("state built for frame_cap 2*N_F, called with N_F")
        call_cap = nf                    # smaller: the call stays inside the buffer
    else:
        say("state never initialised (zero bytes)")
        case.state.zero_()
        call_cap = cap
    before = case.state.cpu().clone()
    out = case.run(Q, K, V, L, spans, 1, 40) if kind == "uninitialised" else None
    if kind == "frame_cap":
        # the same calls as ArrayCase.run, with the mismatched capacity
        from paper_2606_01790_amd.pipeline import to_device
        dev = case.device
        q, k = to_device(Q, "bf16", dev), to_device(K, "bf16", dev)
        lay = sk.contiguous_layout(k, dims)
        Lp = L - W
        S = torch.zeros(nl * G * Lp, dtype=torch.float32, device=dev)
        sbar = torch.zeros(nl * Lp, dtype=torch.float32, device=dev)
        gstar = torch.zeros(nl * Lp, dtype=torch.uint8, device=dev)
        ws = torch.zeros(sk.workspace_bytes(dims), dtype=torch.uint8, device=dev)
        sk.score(dims, p, q, k, lay, S, sbar, gstar, ws)
        sk.update_state(dims, p, S, sbar, spans, 1, case.state, call_cap, case.scal)
        torch.cuda.synchronize()
        scal = case.scal.view(nl, case.nscal).cpu().numpy()
    else:
        scal = out["scal"]
    assert np.isnan(scal).all(), scal
    assert torch.equal(case.state.cpu(), before), "state modified"
