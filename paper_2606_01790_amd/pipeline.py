"""Device buffers of one trajectory and the four calls of a compression step.

This module only allocates (through PyTorch) and marshals; every step of the
compression runs in libstarkv.so.  The K/V cache of all layers is one
device tensor [n_layers, G, L_cap, d] that grows by appending a screenshot
per step, as in a GUI agent's prefill; the window queries are [n_layers, H,
W, d].
"""

from __future__ import annotations

import numpy as np
import torch

from . import starkv as sk
from .workload import Trajectory, WorkloadSpec


def to_device(arr: np.ndarray, dtype: str, device) -> torch.Tensor:
    """Storage array (uint16 bf16 bits or float32) -> device tensor."""
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32))
    return t.to(device, non_blocking=False)


class LayerGroups:
    """The four calls of one step run as `n` contiguous layer groups on `n`
    HIP streams.  Group j's scoring starts when group j-1's scoring has
    finished, so the statistics, selection and gather of one group (few
    workgroups, latency-bound) overlap the scoring of the next; the caller's
    stream waits for every group at the end of the step.

    Each layer's slice of every buffer is contiguous, so a group's arguments
    are pointer offsets into the full tensors; every group has its own
    workspace.  Group 0 runs on the caller's current stream."""

    def __init__(self, n_layers: int, n_groups: int, ws_bytes: int, device):
        n_groups = max(1, min(n_groups, n_layers))
        b = [(i * n_layers) // n_groups for i in range(n_groups + 1)]
        self.ranges = [(b[i], b[i + 1]) for i in range(n_groups)]
        self.ws = [torch.zeros(max(ws_bytes, 16), dtype=torch.uint8, device=device)
                   for _ in self.ranges]
        self.streams = [None] + [torch.cuda.Stream(device=device)
                                 for _ in self.ranges[1:]]

    def run(self, make_dims, params, step, spans, B, Q, K, V, S, sbar, gstar, s, idx,
            k_out, v_out, scal, nscal, state, state_stride, frame_cap):
        """make_dims(n_layers) -> dims of this step for that many layers."""
        cur = torch.cuda.current_stream()
        prev_scored = None
        for j, (l0, l1) in enumerate(self.ranges):
            st = cur if j == 0 else self.streams[j]
            if prev_scored is not None:
                st.wait_event(prev_scored)
            dims = make_dims(l1 - l0)
            G, Ns, Lp, W, d = dims.G, dims.Ns, dims.L - dims.W, dims.W, dims.d
            kg, vg = K[l0:l1], V[l0:l1]
            lay = sk.contiguous_layout(kg, dims)
            n_out = G * (B + W) * d
            Sg = S[l0 * Ns * Lp:l1 * Ns * Lp]
            sb = sbar[l0 * Lp:l1 * Lp]
            gs = gstar[l0 * Lp:l1 * Lp]
            scg = scal[l0 * nscal:l1 * nscal]
            stg = state[l0 * state_stride:l1 * state_stride]
            ws = self.ws[j]
            sk.score(dims, params, Q[l0:l1], kg, lay, Sg, sb, gs, ws, st)
            if j + 1 < len(self.ranges):
                prev_scored = torch.cuda.Event()
                prev_scored.record(st)
            sk.update_state_select(dims, params, Sg, sb, gs, spans, step, stg, frame_cap, scg, B,
                                   s[l0 * Lp:l1 * Lp], idx[l0 * B:l1 * B] if B else idx, ws,
                                   st)
            sk.compact(dims, kg, vg, lay, idx[l0 * B:l1 * B] if B else idx, B,
                       k_out[l0 * n_out:l1 * n_out], v_out[l0 * n_out:l1 * n_out], st)
        for st in self.streams[1:]:
            cur.wait_stream(st)


class TrajectoryRunner:
    """Holds every device buffer of a trajectory of `spec` and runs its steps."""

    def __init__(self, spec: WorkloadSpec, params: sk.Params, device="cuda",
                 max_budget: int | None = None, per_head: bool = False):
        self.spec = spec
        self.params = params
        self.per_head = per_head
        self.Ns = spec.H if per_head else spec.G   # scoring subspaces
        self.device = torch.device(device)
        self.traj = Trajectory(spec)
        sp = spec
        self.tdtype = torch.bfloat16 if sp.dtype == "bf16" else torch.float32
        self.dt = sk.BF16 if sp.dtype == "bf16" else sk.F32
        self.L_cap = sp.L(sp.peak_step)
        Lp_max = sp.L_p(sp.peak_step)
        B_max = max_budget if max_budget is not None else max(
            max(sp.budgets(s)) for s in range(1, sp.steps + 1))
        self.B_max = B_max
        nl, G, H, d, W = sp.n_layers, sp.G, sp.H, sp.d, sp.W
        dev = self.device
        self.K = torch.zeros((nl, G, self.L_cap, d), dtype=self.tdtype, device=dev)
        self.V = torch.zeros((nl, G, self.L_cap, d), dtype=self.tdtype, device=dev)
        self.Q = torch.zeros((nl, H, W, d), dtype=self.tdtype, device=dev)
        self.layout = sk.contiguous_layout(self.K, self.dims(sp.peak_step))
        self.S = torch.zeros(nl * self.Ns * Lp_max, dtype=torch.float32, device=dev)
        self.sbar = torch.zeros(nl * Lp_max, dtype=torch.float32, device=dev)
        self.gstar = torch.zeros(nl * Lp_max, dtype=torch.uint8, device=dev)
        self.s = torch.zeros(nl * Lp_max, dtype=torch.float32, device=dev)
        self.idx = torch.zeros(nl * max(B_max, 1), dtype=torch.int32, device=dev)
        self.k_out = torch.zeros(nl * G * (B_max + W) * d, dtype=self.tdtype, device=dev)
        self.v_out = torch.zeros_like(self.k_out)
        dmax = self.dims(sp.peak_step)
        self.ws = torch.zeros(sk.workspace_bytes(dmax), dtype=torch.uint8, device=dev)
        self.frame_cap = sp.n_frame
        self.state = torch.zeros(sk.state_bytes(dmax, self.frame_cap), dtype=torch.uint8,
                                 device=dev)
        self.nscal = sk.scalars_count(dmax)
        self.scal = torch.zeros(nl * self.nscal, dtype=torch.float32, device=dev)

    def dims(self, step: int) -> sk.Dims:
        sp = self.spec
        return sk.make_dims(sp.n_layers, sp.H, sp.G, sp.d, sp.L(step), sp.W, self.dt,
                            self.per_head)

    def reset(self, stream=None):
        """Start a trajectory: fresh online state."""
        sk.state_init(self.dims(self.spec.peak_step), self.state, self.frame_cap, stream)

    def load_step(self, step: int):
        """Append screenshot `step` and write the step's text tokens and window
        queries for every layer (host -> device copies, outside timing)."""
        sp, tr = self.spec, self.traj
        if not sp.appends:
            # frames leave the context or change size: the whole cache moves
            L = sp.L(step)
            for layer in range(sp.n_layers):
                k, v = tr.layer_cache(layer, step)
                self.K[layer, :, :L] = to_device(k, sp.dtype, self.device)
                self.V[layer, :, :L] = to_device(v, sp.dtype, self.device)
                self.Q[layer] = to_device(tr.window_q(layer, step), sp.dtype, self.device)
            return
        nf = sp.n_frame
        f0 = (step - 1) * nf
        for layer in range(sp.n_layers):
            k, v = tr.frame_kv(layer, step)
            self.K[layer, :, f0:f0 + nf] = to_device(k, sp.dtype, self.device)
            self.V[layer, :, f0:f0 + nf] = to_device(v, sp.dtype, self.device)
            k, v = tr.text_kv(layer, step)
            t0 = step * nf
            self.K[layer, :, t0:t0 + sp.text] = to_device(k, sp.dtype, self.device)
            self.V[layer, :, t0:t0 + sp.text] = to_device(v, sp.dtype, self.device)
            self.Q[layer] = to_device(tr.window_q(layer, step), sp.dtype, self.device)

    def score_and_update(self, step: int, stream=None):
        """starkv_score and starkv_update_state of one step, all layers."""
        sp = self.spec
        dims = self.dims(step)
        spans = sp.spans(step)
        sk.score(dims, self.params, self.Q, self.K, self.layout, self.S, self.sbar,
                 self.gstar, self.ws, stream)
        sk.update_state(dims, self.params, self.S, self.sbar, spans, step, self.state,
                        self.frame_cap, self.scal, self.ws, stream)

    def select_and_compact(self, step: int, B: int, stream=None):
        """starkv_select and starkv_compact of one step for budget B."""
        sp = self.spec
        dims = self.dims(step)
        spans = sp.spans(step)
        sk.select(dims, self.params, self.sbar, self.gstar, self.scal, spans, step, B,
                  self.s, self.idx, self.ws, stream)
        sk.compact(dims, self.K, self.V, self.layout, self.idx, B, self.k_out,
                   self.v_out, stream)

    def run_step(self, step: int, B: int, stream=None, groups: int = 1, fused: bool = False):
        """The compression stage of one step for all layers: the four calls
        (three with `fused`: the statistics and the selection in one call),
        on the current stream, or as `groups` layer groups on as many streams
        (see LayerGroups)."""
        if groups <= 1 and fused:
            sp = self.spec
            dims = self.dims(step)
            spans = sp.spans(step)
            sk.score(dims, self.params, self.Q, self.K, self.layout, self.S, self.sbar,
                     self.gstar, self.ws, stream)
            sk.update_state_select(dims, self.params, self.S, self.sbar, self.gstar, spans, step,
                                   self.state, self.frame_cap, self.scal, B, self.s, self.idx,
                                   self.ws, stream)
            sk.compact(dims, self.K, self.V, self.layout, self.idx, B, self.k_out, self.v_out,
                       stream)
            return
        if groups <= 1:
            self.score_and_update(step, stream)
            self.select_and_compact(step, B, stream)
            return
        sp = self.spec
        if getattr(self, "_groups", None) is None or len(self._groups.ranges) != groups:
            self._groups = LayerGroups(sp.n_layers, groups, self.ws.numel(), self.device)
        d1 = sk.make_dims(1, sp.H, sp.G, sp.d, sp.L(sp.peak_step), sp.W, self.dt,
                          self.per_head)
        self._groups.run(
            lambda n: sk.make_dims(n, sp.H, sp.G, sp.d, sp.L(step), sp.W, self.dt,
                                   self.per_head),
            self.params, step, sp.spans(step), B, self.Q, self.K, self.V, self.S,
            self.sbar, self.gstar, self.s, self.idx, self.k_out, self.v_out, self.scal,
            self.nscal, self.state, sk.state_bytes(d1, self.frame_cap), self.frame_cap)

    # ---- views of the outputs of the last step (host copies)
    def outputs(self, step: int, B: int) -> dict:
        sp = self.spec
        nl, G, Lp, W, d = sp.n_layers, sp.G, sp.L_p(step), sp.W, sp.d
        n_out = nl * G * (B + W) * d
        out = dict(
            S=self.S[:nl * self.Ns * Lp].view(nl, self.Ns, Lp).cpu().numpy(),
            sbar=self.sbar[:nl * Lp].view(nl, Lp).cpu().numpy(),
            gstar=self.gstar[:nl * Lp].view(nl, Lp).cpu().numpy(),
            s=self.s[:nl * Lp].view(nl, Lp).cpu().numpy(),
            idx=self.idx[:nl * B].view(nl, B).cpu().numpy(),
            scal=self.scal.view(nl, self.nscal).cpu().numpy(),
        )
        ko = self.k_out[:n_out].view(nl, G, B + W, d)
        vo = self.v_out[:n_out].view(nl, G, B + W, d)
        if sp.dtype == "bf16":
            out["k_out"] = ko.view(torch.int16).cpu().numpy().view(np.uint16)
            out["v_out"] = vo.view(torch.int16).cpu().numpy().view(np.uint16)
        else:
            out["k_out"] = ko.cpu().numpy()
            out["v_out"] = vo.cpu().numpy()
        return out


class ArrayCase:
    """Runs the four calls on explicit host arrays (tests of edge cases).

    Q: [n_layers, H, W, d]; K, V: [n_layers, G, L_cap, d] storage arrays
    (uint16 bf16 bits or float32).  The state persists across run() calls
    until reset().
    """

    def __init__(self, H, G, d, W, n_layers, L_cap, dtype, params, frame_cap,
                 device="cuda", per_head=False):
        self.H, self.G, self.d, self.W, self.nl = H, G, d, W, n_layers
        self.per_head = per_head
        self.Ns = H if per_head else G
        self.L_cap, self.dtype, self.params = L_cap, dtype, params
        self.dt = sk.BF16 if dtype == "bf16" else sk.F32
        self.device = torch.device(device)
        self.frame_cap = frame_cap
        dmax = self.dims(L_cap)
        self.state = torch.zeros(sk.state_bytes(dmax, frame_cap), dtype=torch.uint8,
                                 device=self.device)
        self.nscal = sk.scalars_count(dmax)
        self.scal = torch.zeros(n_layers * self.nscal, dtype=torch.float32,
                                device=self.device)
        self.reset()

    def dims(self, L):
        return sk.make_dims(self.nl, self.H, self.G, self.d, L, self.W, self.dt,
                            self.per_head)

    def reset(self):
        sk.state_init(self.dims(self.L_cap), self.state, self.frame_cap)

    def run(self, Q, K, V, L, spans, F, B):
        dev, nl, G, W, d = self.device, self.nl, self.G, self.W, self.d
        dims = self.dims(L)
        Lp = L - W
        q = to_device(Q, self.dtype, dev)
        k = to_device(K, self.dtype, dev)
        v = to_device(V, self.dtype, dev)
        lay = sk.contiguous_layout(k, dims)
        S = torch.zeros(nl * self.Ns * Lp, dtype=torch.float32, device=dev)
        sbar = torch.zeros(nl * Lp, dtype=torch.float32, device=dev)
        gstar = torch.zeros(nl * Lp, dtype=torch.uint8, device=dev)
        s = torch.zeros(nl * Lp, dtype=torch.float32, device=dev)
        idx = torch.zeros(nl * max(B, 1), dtype=torch.int32, device=dev)
        tdt = k.dtype
        ko = torch.zeros(nl * G * (B + W) * d, dtype=tdt, device=dev)
        vo = torch.zeros_like(ko)
        ws = torch.zeros(max(sk.workspace_bytes(dims), 16), dtype=torch.uint8, device=dev)
        sk.score(dims, self.params, q, k, lay, S, sbar, gstar, ws)
        sk.update_state(dims, self.params, S, sbar, spans, F, self.state, self.frame_cap,
                        self.scal, ws)
        sk.select(dims, self.params, sbar, gstar, self.scal, spans, F, B, s, idx, ws)
        sk.compact(dims, k, v, lay, idx, B, ko, vo)
        torch.cuda.synchronize()
        out = dict(S=S.view(nl, self.Ns, Lp).cpu().numpy(), sbar=sbar.view(nl, Lp).cpu().numpy(),
                   gstar=gstar.view(nl, Lp).cpu().numpy(), s=s.view(nl, Lp).cpu().numpy(),
                   idx=idx[:nl * B].view(nl, B).cpu().numpy(),
                   scal=self.scal.view(nl, self.nscal).cpu().numpy())
        ko = ko.view(nl, G, B + W, d)
        vo = vo.view(nl, G, B + W, d)
        if self.dtype == "bf16":
            out["k_out"] = ko.view(torch.int16).cpu().numpy().view(np.uint16)
            out["v_out"] = vo.view(torch.int16).cpu().numpy().view(np.uint16)
        else:
            out["k_out"] = ko.cpu().numpy()
            out["v_out"] = vo.cpu().numpy()
        return out
