#!/usr/bin/env python3
"""Throughput of the STaR-KV compression stage on one MI355X.

One bench step is one whole pass of the hot path over the workload: every
trajectory step of the 28-layer, 5-screenshot trajectory (Qwen2.5-VL-7B
GQA shape, bf16), each running starkv_score, starkv_update_state_select
(the statistics and the selection in one call) and starkv_compact for all
layers.  The caches of every
trajectory step, the window queries and a fresh per-trajectory state are
resident in HBM before the timed region starts.

Prints one JSON line:
  value      compressed visual tokens per second per layer: the sum over
             trajectory steps and layers of N_vis, divided by the time;
  roofline   the dominant call's achieved algorithmic bandwidth against the
             8 TB/s HBM peak, or its algorithmic flops against the dense
             MFMA peak when its intensity is above the ridge (the W = 64
             trajectory), from HIP events on its stream;
  cpu_baseline  the fp64 CPU oracle on a bounded sample of the same work.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# dense MFMA peaks by input type (TFLOP/s)
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
METRIC = "compressed visual KV tokens/s per layer (score+select+gather); % HBM peak"


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="oracle time of the CPU sample: layers are added, each with its "
                         "whole trajectory, until this much oracle time has run")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--groups", type=int, default=1,
                    help="layer groups per step, each on its own HIP stream (1: one "
                         "launch of every call for all layers)")
    ap.add_argument("--eager", action="store_true",
                    help="launch every call from Python instead of replaying a HIP graph")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain elementwise kernel that reads 1 GiB and "
                         "writes 1 GiB (the calibration of the HBM byte counters)")
    ap.add_argument("--no-per-call", action="store_true",
                    help="skip the per-call timing (no roofline; for counter runs)")
    ap.add_argument("--decode", action="store_true",
                    help="instead of the stage: decode attention of one new token per head "
                         "over the stage's compressed cache and over the full cache, at the "
                         "trajectory's last step")
    ap.add_argument("--tem-decay", choices=["exp", "linear", "gamma"], default="exp",
                    help="temporal discount variant of the decay ablation (exp is the paper's)")
    ap.add_argument("--aeb", choices=["entropy", "confidence"], default="entropy",
                    help="AEB temperature variant of the ablation (entropy is the paper's)")
    ap.add_argument("--budget-pct", type=int, default=None,
                    help="run the workload at this one of its budget percentages "
                         "(default: the first)")
    ap.add_argument("--per-head", action="store_true",
                    help="a scoring subspace per query head (the MHA-head granularity "
                         "on the GQA model) instead of one per KV group")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class Workload:
    """Resident inputs and outputs of one trajectory of `spec`."""

    def __init__(self, spec, params, n_states, device="cuda", per_head=False):
        import torch
        from paper_2606_01790_amd import starkv as sk
        from paper_2606_01790_amd.pipeline import to_device
        from paper_2606_01790_amd.workload import Trajectory

        self.spec, self.params, self.sk = spec, params, sk
        self.per_head = per_head
        sp = spec
        Ns = sp.H if per_head else sp.G
        dt = torch.bfloat16 if sp.dtype == "bf16" else torch.float32
        self.dt = sk.BF16 if sp.dtype == "bf16" else sk.F32
        tr = Trajectory(sp)
        nl, G, H, d, W, nf = sp.n_layers, sp.G, sp.H, sp.d, sp.W, sp.n_frame
        frames_k, frames_v = {}, {}     # frame -> [n_layers, G, tokens, d]
        for f in range(1, sp.steps + 1):
            frames_k[f] = torch.empty((nl, G, sp.frame_tokens(f), d), dtype=dt, device=device)
            frames_v[f] = torch.empty_like(frames_k[f])
            for layer in range(nl):
                k, v = tr.frame_kv(layer, f)
                frames_k[f][layer] = to_device(k, sp.dtype, device)
                frames_v[f][layer] = to_device(v, sp.dtype, device)
        self.K, self.V, self.Q, self.layout = [], [], [], []
        for s in range(1, sp.steps + 1):
            tk = torch.empty((nl, G, sp.text, d), dtype=dt, device=device)
            tv = torch.empty_like(tk)
            q = torch.empty((nl, H, W, d), dtype=dt, device=device)
            for layer in range(nl):
                k, v = tr.text_kv(layer, s)
                tk[layer] = to_device(k, sp.dtype, device)
                tv[layer] = to_device(v, sp.dtype, device)
                q[layer] = to_device(tr.window_q(layer, s), sp.dtype, device)
            K = torch.cat([frames_k[f] for f in sp.frames(s)] + [tk], dim=2).contiguous()
            V = torch.cat([frames_v[f] for f in sp.frames(s)] + [tv], dim=2).contiguous()
            self.K.append(K)
            self.V.append(V)
            self.Q.append(q)
            self.layout.append(sk.contiguous_layout(K, self.dims(s)))
        del frames_k, frames_v
        Lp, B = sp.L_p(sp.peak_step), max(max(sp.budgets(s)) for s in range(1, sp.steps + 1))
        f32 = torch.float32
        self.S = torch.empty(nl * Ns * Lp, dtype=f32, device=device)
        self.sbar = torch.empty(nl * Lp, dtype=f32, device=device)
        self.gstar = torch.empty(nl * Lp, dtype=torch.uint8, device=device)
        self.s = torch.empty(nl * Lp, dtype=f32, device=device)
        self.idx = torch.empty(nl * B, dtype=torch.int32, device=device)
        self.k_out = torch.empty(nl * G * (B + W) * d, dtype=dt, device=device)
        self.v_out = torch.empty_like(self.k_out)
        dmax = self.dims(sp.peak_step)
        self.ws = torch.empty(sk.workspace_bytes(dmax), dtype=torch.uint8, device=device)
        self.nscal = sk.scalars_count(dmax)
        self.scal = torch.empty(nl * self.nscal, dtype=f32, device=device)
        self.frame_cap = nf
        self.states = [torch.empty(sk.state_bytes(dmax, nf), dtype=torch.uint8,
                                   device=device) for _ in range(n_states)]
        for st in self.states:
            sk.state_init(dmax, st, nf)
        torch.cuda.synchronize()

    def dims(self, s, n_layers=None):
        sp = self.spec
        return self.sk.make_dims(n_layers or sp.n_layers, sp.H, sp.G, sp.d, sp.L(s), sp.W,
                                 self.dt, self.per_head)

    def trajectory(self, state, groups=1):
        """The hot path over the whole trajectory: the four calls per step, for
        all layers at once or as `groups` layer groups on as many streams."""
        sk, sp, p = self.sk, self.spec, self.params
        if groups > 1:
            from paper_2606_01790_amd.pipeline import LayerGroups
            if getattr(self, "_lg", None) is None or len(self._lg.ranges) != groups:
                self._lg = LayerGroups(sp.n_layers, groups, self.ws.numel(), self.ws.device)
            stride = sk.state_bytes(self.dims(sp.peak_step, 1), self.frame_cap)
            for s in range(1, sp.steps + 1):
                i = s - 1
                self._lg.run(
                    lambda n, s=s: self.dims(s, n),
                    p, s, sp.spans(s), sp.budgets(s)[0], self.Q[i], self.K[i], self.V[i],
                    self.S, self.sbar, self.gstar, self.s, self.idx, self.k_out, self.v_out,
                    self.scal, self.nscal, state, stride, self.frame_cap)
            return
        for s in range(1, sp.steps + 1):
            i = s - 1
            dims = self.dims(s)
            spans = sp.spans(s)
            B = sp.budgets(s)[0]
            sk.score(dims, p, self.Q[i], self.K[i], self.layout[i], self.S, self.sbar,
                     self.gstar, self.ws)
            sk.update_state_select(dims, p, self.S, self.sbar, self.gstar, spans, s, state,
                                   self.frame_cap, self.scal, B, self.s, self.idx, self.ws)
            sk.compact(dims, self.K[i], self.V[i], self.layout[i], self.idx, B, self.k_out,
                       self.v_out)


def call_bytes(spec, s, name, per_head=False):
    """Algorithmic HBM bytes of one call at trajectory step s, all layers:
    inputs read once and outputs written once (Ns scoring subspaces)."""
    sp = spec
    e, nl, H, G, d, W = sp.elem_bytes, sp.n_layers, sp.H, sp.G, sp.d, sp.W
    Ns = H if per_head else G
    Lp, nv, nf, B = sp.L_p(s), sp.n_vis(s), sp.n_frame, sp.budgets(s)[0]
    if name == "score":        # Q and K_past read once (S, sbar, g* are intermediates)
        per = e * (H * W * d + G * Lp * d)
    elif name == "update_state":   # S of visual tokens, sbar, stability means
        per = 4 * Ns * nv + 4 * Lp + 4 * Ns * nf * 3
    elif name == "select":     # sbar, g* in; s, idx out
        per = 5 * Lp + 4 * Lp + 4 * B
    elif name == "update_state_select":
        return call_bytes(spec, s, "update_state", per_head) + call_bytes(spec, s, "select",
                                                                          per_head)
    else:                      # idx in; B+W rows of K and V in and out
        per = 4 * B + 4 * G * (B + W) * d * e
    return nl * per


def roofline_of(seconds, alg_bytes, alg_flops, dtype):
    """Roofline of one launch: the roof its algorithmic intensity meets first,
    HBM (GB/s against 8 TB/s) or the dense MFMA peak of its input type
    (TFLOP/s), with the achieved rate and its fraction of that peak."""
    mfma_peak = MFMA_PEAK_TFLOPS[dtype]
    if alg_bytes > 0 and alg_flops / alg_bytes > mfma_peak * 1e12 / (HBM_PEAK_GBS * 1e9):
        achieved = alg_flops / seconds / 1e12
        return {"bound": "mfma", "achieved": round(achieved, 1), "peak": mfma_peak,
                "unit": "TFLOP/s", "frac": round(achieved / mfma_peak, 4)}
    achieved = alg_bytes / seconds / 1e9
    return {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4)}


def per_call_timing(wl, spec, sk, torch, reps):
    """Average GPU time of each call, per trajectory step: `reps` launches of
    the call back to back, captured in a HIP graph and timed with HIP events
    on the replay stream.  update_state runs on a scratch state."""
    from paper_2606_01790_amd import workload as WL
    p = wl.params
    scratch = wl.states[-2]
    per = {}
    stream = torch.cuda.current_stream()
    for s in range(1, spec.steps + 1):
        i = s - 1
        dims, spans, B = wl.dims(s), spec.spans(s), spec.budgets(s)[0]
        calls = {
            "score": lambda: sk.score(dims, p, wl.Q[i], wl.K[i], wl.layout[i], wl.S,
                                      wl.sbar, wl.gstar, wl.ws),
            "update_state": lambda: sk.update_state(dims, p, wl.S, wl.sbar, spans, s,
                                                    scratch, wl.frame_cap, wl.scal, wl.ws),
            "select": lambda: sk.select(dims, p, wl.sbar, wl.gstar, wl.scal, spans, s, B,
                                        wl.s, wl.idx, wl.ws),
            "update_state_select": lambda: sk.update_state_select(
                dims, p, wl.S, wl.sbar, wl.gstar, spans, s, scratch, wl.frame_cap, wl.scal, B,
                wl.s, wl.idx, wl.ws),
            "compact": lambda: sk.compact(dims, wl.K[i], wl.V[i], wl.layout[i], wl.idx, B,
                                          wl.k_out, wl.v_out),
        }
        for name, fn in calls.items():
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for _ in range(reps):
                    fn()
            g.replay()
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            g.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            d = per.setdefault(name, {"time": 0.0, "launches": 0, "bytes": 0, "flops": 0})
            d["time"] += e0.elapsed_time(e1) * 1e-3
            d["launches"] += reps
            d["bytes"] += reps * call_bytes(spec, s, name, wl.per_head)
            if name == "score":   # the window-query/key contraction, counted once
                d["flops"] += reps * spec.n_layers * WL.qk_flops(spec.H, spec.W, spec.L_p(s),
                                                                 spec.d)
    return per


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: the compression stage runs on one GPU only; "
              "a multi-GPU run is not supported (use --gpus 1).", file=sys.stderr)
        sys.exit(2)
    if args.decode:
        return decode_bench(args)
    import numpy as np
    import torch

    from paper_2606_01790_amd import starkv as sk
    from paper_2606_01790_amd import workload as WL

    assert torch.cuda.is_available(), "no GPU visible"
    spec = pick_budget(WL.SPECS[args.config], args.budget_pct)
    params = sk.params_default()
    if args.config >= 3:
        params.t_min, params.t_max = 0.95, 1.05
    params.tem_decay, params.aeb_mode = sk.TEM_DECAY[args.tem_decay], sk.AEB_MODE[args.aeb]
    log(f"workload {spec.name}: building resident inputs")
    n_states = args.warmup + 3
    wl = Workload(spec, params, n_states, per_head=args.per_head)
    sweep = len(WL.SPECS[args.config].pcts) > 1
    workload = (spec.name + (f"-at-{spec.pcts[0]}pct" if sweep else "")
                + ("-per-head" if args.per_head else "")
                + ("" if args.tem_decay == "exp" else f"-tem-{args.tem_decay}")
                + ("" if args.aeb == "entropy" else f"-aeb-{args.aeb}"))
    layer_tokens = spec.n_layers * sum(spec.n_vis(s) for s in range(1, spec.steps + 1))
    bytes_alg = spec.n_layers * sum(WL.bytes_alg(spec, s, spec.budgets(s)[0])
                                    for s in range(1, spec.steps + 1))

    log(f"warmup {args.warmup}")
    k = 0
    for _ in range(args.warmup):
        wl.trajectory(wl.states[k], args.groups)
        k += 1
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    if args.eager:
        run = lambda: wl.trajectory(wl.states[0], args.groups)  # noqa: E731
    else:
        # One trajectory (a fresh state, then every step's four calls) captured
        # into a HIP graph: the timed region replays it, so the host's Python
        # launch cost does not starve the GPU.
        graph_state = wl.states[-1]
        dmax = wl.dims(spec.peak_step)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            sk.state_init(dmax, graph_state, wl.frame_cap)
            wl.trajectory(graph_state, args.groups)
        torch.cuda.synchronize()
        run = g.replay
        for _ in range(args.warmup):
            run()
        torch.cuda.synchronize()

    log(f"timed {args.steps} steps ({'eager' if args.eager else 'graph replay'})")
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = e0.elapsed_time(e1)
    ms_per_step = max(gpu_ms, wall * 1e3) / args.steps
    value = layer_tokens / (ms_per_step * 1e-3)

    roofline, per_call_us = None, None
    if not args.no_per_call:
        log("per-call timing: graphs of back-to-back launches of one call")
        per = per_call_timing(wl, spec, sk, torch, reps=10)
        dom = max(per, key=lambda n: per[n]["time"])
        dd = per[dom]
        avg_s = dd["time"] / dd["launches"]
        avg_b = dd["bytes"] / dd["launches"]
        avg_f = dd["flops"] / dd["launches"]
        roofline = roofline_of(avg_s, avg_b, avg_f, spec.dtype)
        roofline.update({"traffic": measured_traffic(f"starkv_{dom}", workload),
                         "kernel": f"starkv_{dom}",
                         "avg_launch_us": round(avg_s * 1e6, 2),
                         "alg_bytes_per_launch": int(avg_b),
                         "alg_flops_per_launch": int(avg_f),
                         # the contraction's rate against the dense MFMA peak of
                         # its input type, whichever roof binds
                         "mfma_frac": round(avg_f / avg_s / 1e12 / MFMA_PEAK_TFLOPS[spec.dtype], 4)})
        per_call_us = {n: round(per[n]["time"] / per[n]["launches"] * 1e6, 2) for n in per}

    copy_gbs = measure_copy_bandwidth(torch)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(spec, params, args.cpu_seconds, args.per_head, args.tem_decay,
                           args.aeb)

    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "layer-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic",
        "config": {"workload": workload, "n_layers": spec.n_layers, "H": spec.H,
                   "G": spec.G, "d": spec.d, "W": spec.W,
                   "subspaces": (f"per head ({spec.H})" if args.per_head
                                 else f"per KV group ({spec.G})"),
                   "trajectory_steps": spec.steps, "budget_pct": list(spec.pcts),
                   "layer_tokens_per_step": layer_tokens,
                   "bytes_alg_per_step": bytes_alg,
                   "launch": ("eager" if args.eager else "hipgraph")
                   + (f", {args.groups} layer groups on {args.groups} streams"
                      if args.groups > 1 else "")},
        "hbm_frac_path": round(bytes_alg / (ms_per_step * 1e-3) / (HBM_PEAK_GBS * 1e9), 4),
        "copy_gbs_measured": round(copy_gbs, 1),
        "copy_frac_path": round(bytes_alg / (ms_per_step * 1e-3) / (copy_gbs * 1e9), 4),
        "per_call_us": per_call_us,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    if args.copy_calibration:
        n = 1 << 28                       # float32: 1 GiB read, 1 GiB written
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        torch.neg(a, out=b)
        torch.cuda.synchronize()
        line["copy_calibration_bytes"] = 4 * n
    print(json.dumps(line), flush=True)


def decode_bench(args):
    """Decode attention (starkv_decode) of one new token per query head, all
    layers, at the trajectory's last step: over the K'/V' the stage keeps
    (B + W rows per group) and over the full cache (L rows).  Each is timed
    as a HIP graph of `reps` back-to-back launches with HIP events; `value`
    is decoded tokens per second over the compressed cache."""
    import numpy as np
    import torch

    from paper_2606_01790_amd import starkv as sk
    from paper_2606_01790_amd import workload as WL
    from paper_2606_01790_amd.pipeline import TrajectoryRunner

    spec = pick_budget(WL.SPECS[args.config], args.budget_pct)
    params = sk.params_default()
    if args.config >= 3:
        params.t_min, params.t_max = 0.95, 1.05
    s = spec.steps
    B = spec.budgets(s)[0]
    nl, H, G, d, W, L = spec.n_layers, spec.H, spec.G, spec.d, spec.W, spec.L(s)
    log(f"decode on {spec.name}: running the trajectory to step {s} for K'/V'")
    r = TrajectoryRunner(spec, params)
    r.reset()
    for step in range(1, s + 1):
        r.load_step(step)
        r.run_step(step, spec.budgets(step)[0])
    torch.cuda.synchronize()
    n_c = B + W
    rng = np.random.default_rng([spec.seed, 4242])
    q = torch.from_numpy(WL.f32_to_bf16_bits(
        rng.standard_normal((nl, H, d), dtype=np.float32)).view(np.int16)).to("cuda")
    out = torch.empty(nl * H * d, dtype=torch.float32, device="cuda")
    dims = sk.make_dims(nl, H, G, d, L, W, sk.BF16)
    kc = r.k_out[:nl * G * n_c * d]
    vc = r.v_out[:nl * G * n_c * d]
    lay_c = sk.KVLayout(G * n_c * d, n_c * d, d)
    cases = {"compressed": (kc, vc, lay_c, n_c), "full": (r.K, r.V, r.layout, L)}
    stream = torch.cuda.current_stream()
    reps = 20
    res = {}
    for name, (k, v, lay, n) in cases.items():
        ws = torch.empty(sk.decode_workspace_bytes(dims, n), dtype=torch.uint8, device="cuda")
        fn = lambda k=k, v=v, lay=lay, n=n, ws=ws: sk.decode(dims, q, k, v, lay, n, out, ws)  # noqa: E731
        for _ in range(args.warmup):
            fn()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                fn()
        g.replay()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) * 1e-3 / (args.steps * reps)
        # algorithmic bytes: every K and V row once, q, the output
        nbytes = nl * (2 * G * n * d * 2 + H * d * 2 + H * d * 4)
        res[name] = {"tokens": n, "us_per_token": round(t * 1e6, 2),
                     "achieved_GBs": round(nbytes / t / 1e9, 1),
                     "attention_mflops_per_token": round(nl * WL.decode_flops(H, n, d) / 1e6, 2)}
    comp, full = res["compressed"], res["full"]
    t_c = comp["us_per_token"] * 1e-6
    copy_gbs = measure_copy_bandwidth(torch)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = decode_cpu_baseline(spec, r, q, n_c, args.cpu_seconds)
    line = {
        "metric": "decode attention over the compressed cache: generated tokens/s, all layers",
        "value": round(1.0 / t_c, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_c * 1e3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": spec.name + "-decode", "n_layers": nl, "H": H, "G": G, "d": d,
                   "W": W, "step": s, "B": B, "cache_tokens_full": L,
                   "cache_tokens_compressed": n_c, "launch": f"hipgraph x{reps}"},
        "compressed": comp,
        "full": full,
        "speedup_vs_full": round(full["us_per_token"] / comp["us_per_token"], 2),
        "attention_flops_saving": round(1.0 - comp["attention_mflops_per_token"]
                                        / full["attention_mflops_per_token"], 4),
        "roofline": {"bound": "hbm", "achieved": comp["achieved_GBs"], "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(comp["achieved_GBs"] / HBM_PEAK_GBS, 4),
                     "traffic": None, "kernel": "starkv_decode",
                     "avg_launch_us": comp["us_per_token"]},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def decode_cpu_baseline(spec, runner, q, n_c, seconds):
    """The oracle's decode attention on the host, over the same compressed
    caches, layer after layer until `seconds` of oracle time have run."""
    import numpy as np

    from oracle import starkv_oracle as O
    from paper_2606_01790_amd import workload as WL

    nl, H, G, d = spec.n_layers, spec.H, spec.G, spec.d
    qh = q.cpu().numpy().view(np.uint16).reshape(nl, H, d)
    import torch
    kh = runner.k_out[:nl * G * n_c * d].view(torch.int16).cpu().numpy().view(np.uint16)
    vh = runner.v_out[:nl * G * n_c * d].view(torch.int16).cpu().numpy().view(np.uint16)
    kh = kh.reshape(nl, G, n_c, d)
    vh = vh.reshape(nl, G, n_c, d)
    spent, layers = 0.0, 0
    while spent < seconds:
        layer = layers % nl
        qf = WL.to_float64(qh[layer], "bf16")
        kf = WL.to_float64(kh[layer], "bf16")
        vf = WL.to_float64(vh[layer], "bf16")
        t0 = time.perf_counter()
        O.decode_attention(qf, kf, vf)
        spent += time.perf_counter() - t0
        layers += 1
    return {"value": round(layers / nl / spent, 1), "unit": "tokens/s", "cores": blas_threads(),
            **host_info(),
            "kind": "oracle",
            "sample": f"{layers} layer decodes over the compressed caches of {spec.name} "
                      f"(step {spec.steps}, {n_c} tokens per group; {spent:.1f} s of oracle "
                      f"time, numpy fp64, BLAS threads {blas_threads()}), scaled to all {nl} layers"}


# Sources whose kernels the committed traffic figure was measured on.
TRAFFIC_SOURCES = {
    "starkv_score": ["score_kernels.h", "score_slab.h", "score.hip", "score_bf16.hip",
                     "device_common.h"],
}


def sources_sha1(call):
    import hashlib
    h = hashlib.sha1()
    for f in TRAFFIC_SOURCES.get(call, []):
        with open(os.path.join(ROOT, "paper_2606_01790_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(call, workload):
    """HBM bytes per launch of `call` from the committed rocprofv3 FETCH_SIZE
    and WRITE_SIZE summary of this workload, or None when there is none or
    the call's kernel sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{call}-{workload}.traffic.md")
    if call not in TRAFFIC_SOURCES or not os.path.exists(path):
        return None
    vals = {}
    with open(path) as fh:
        for ln in fh:
            if ln.startswith("- ") and ":" in ln:
                k, v = ln[2:].split(":", 1)
                vals[k.strip()] = v.strip().strip("`")
    if vals.get("sources_sha1") != sources_sha1(call):
        return None
    try:
        return int(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def measure_copy_bandwidth(torch, reps=5):
    """Device-to-device copy rate of this GPU (GB/s, bytes read plus bytes
    written): 1 GiB copied with torch's copy kernel, best of `reps`, timed
    with HIP events on the current stream."""
    n = 1 << 28
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    best = float("inf")
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        b.copy_(a)
        e1.record(stream)
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1) * 1e-3)
    del a, b
    return 2 * 4 * n / best / 1e9


def host_info():
    """Cores this process may run on, the CPU model, and the BLAS threads."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for ln in fh:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"affinity_cores": len(os.sched_getaffinity(0)), "cpu_model": model,
            "blas_threads": blas_threads()}


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        blas = [i.get("num_threads", 1) for i in threadpool_info()
                if i.get("user_api") == "blas"]
        return max(blas) if blas else 1
    except Exception:
        return 1


def pick_budget(spec, pct):
    """The workload at one of its budget percentages (the first by default);
    the inputs do not depend on the budget."""
    import dataclasses
    if pct is None:
        pct = spec.pcts[0]
    if pct not in spec.pcts:
        sys.exit(f"bench: {spec.name} runs at budgets {list(spec.pcts)} percent, not {pct}")
    return dataclasses.replace(spec, pcts=(pct,))


def cpu_baseline(spec, params, seconds, per_head=False, tem_decay="exp", aeb="entropy"):
    """The fp64 oracle, untuned, on the host cores: whole trajectories (every
    step, fresh state) of layers 0, 1, 2, ... of the same workload, cycling
    through the layers again if needed, until `seconds` of oracle time have
    run.  Input generation is outside the timed part.  Reported as
    layer-tokens/s, like the metric."""
    from oracle import starkv_oracle as O
    from paper_2606_01790_amd import workload as WL

    threads = blas_threads()
    op = O.Params(lam=params.lam, n_warmup=params.n_warmup, n_ramp=params.n_ramp,
                  rho_mi=params.rho_mi, tau=params.tau, rho_t=params.rho_t,
                  delta=params.delta, d_min=params.d_min, t_min=params.t_min,
                  t_max=params.t_max, n_bins=params.n_bins, grid=params.grid,
                  pool_kernel=params.pool_kernel, eps=params.eps, tem_decay=tem_decay,
                  aeb_mode=aeb)
    tr = WL.Trajectory(spec)
    log(f"cpu baseline: oracle trajectories until {seconds:.0f} s of oracle time")
    spent, tokens, runs, layer = 0.0, 0, 0, 0
    while spent < seconds:
        steps = []
        for s in range(1, spec.steps + 1):
            K, V = tr.layer_cache(layer, s)
            steps.append((s, WL.to_float64(tr.window_q(layer, s), spec.dtype),
                          WL.to_float64(K, spec.dtype), K, V))
        state = O.LayerState(spec.H if per_head else spec.G)
        t0 = time.perf_counter()
        for s, Q, K64, K, V in steps:
            if per_head:
                K64 = O.per_head_cache(K64, spec.H)
            _, state = O.compress_layer(Q, K64, None, spec.L(s), spec.W, spec.spans(s), s,
                                        spec.budgets(s)[0], op, state, copy_rows=(K, V))
            tokens += spec.n_vis(s)
        spent += time.perf_counter() - t0
        runs += 1
        layer = (layer + 1) % spec.n_layers
    return {"value": round(tokens / spent, 1), "unit": "layer-tokens/s", "cores": threads,
            "kind": "oracle", **host_info(),
            "sample": f"{runs} whole {spec.steps}-step layer trajectories of {spec.name} "
                      + ("with per-head subspaces " if per_head else "")
                      + f"(layers 0-{min(runs, spec.n_layers) - 1}; {tokens} layer-tokens, "
                      f"{spent:.1f} s of oracle time; numpy fp64, BLAS threads {threads})"}


if __name__ == "__main__":
    main()
