"""Seeded synthetic GUI-trajectory KV caches (input generation only).

This module holds none of the compression method's arithmetic: it draws the
caches, window queries, visual spans and budgets that both the GPU library
and the CPU oracle consume, so that both sides see the same input bytes.

The shapes stand in for the paper's workloads (Qwen2.5-VL-7B-shaped GQA
attention, sec. 3.1; single-screenshot grounding and multi-step trajectories
with one screenshot appended per step, Appendix dataset settings).  None of
the paper's benchmark data is used or reproduced.

Token layout at trajectory step s (1-based): the frames in the context (1..s,
or with `slots` image slots only the newest `slots` of them; each a
rows x cols raster of visual tokens, row-major, at the frame's own
resolution), then the step's text tokens; the last W text tokens are the
observation window.  K, V and Q are standard normal;
each K group carries Gaussian "bumps" over screen regions along a random
sign vector u, and window queries lean toward their group's u, so attention
concentrates spatially and the spatial MI is non-zero.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class WorkloadSpec:
    name: str
    n_layers: int
    H: int
    G: int
    d: int
    dtype: str                 # "f32" or "bf16": storage type of Q, K, V
    cols: int                  # visual grid of one screenshot
    rows: int
    steps: int                 # trajectory steps (one screenshot per step)
    text: int                  # text tokens after the frames, per step
    W: int                     # observation window (also the recent window)
    pcts: tuple                # budgets, percent of visual tokens
    amp: float                 # bump amplitude added to K
    sigma: float               # bump width, tokens
    regions: int               # bumps per bumped group
    migrate: bool              # only group (layer mod G) carries bumps
    repeat_p: float            # chance a bump keeps its place next frame
    q_align: float             # window-query lean toward the group's u
    q_scale_range: tuple = None  # per-step Q scale, U[lo, hi], all layers
    seed: int = 0
    slots: int = 0             # image slots: frames kept in context (0: all)
    res_change: tuple = ()     # (first_frame, cols, rows): resolution from then on

    def grid(self, f: int):
        """(cols, rows) of frame f."""
        cols, rows = self.cols, self.rows
        for f0, c, r in self.res_change:
            if f >= f0:
                cols, rows = c, r
        return cols, rows

    def frame_tokens(self, f: int) -> int:
        c, r = self.grid(f)
        return c * r

    @property
    def n_frame(self) -> int:
        """The largest frame's token count (capacity of per-frame state)."""
        return max([self.rows * self.cols] + [c * r for _, c, r in self.res_change])

    def frames(self, s: int):
        """Frames in the context at step s, oldest first."""
        first = max(1, s - self.slots + 1) if self.slots else 1
        return list(range(first, s + 1))

    def L(self, s: int) -> int:
        return self.n_vis(s) + self.text

    def L_p(self, s: int) -> int:
        return self.L(s) - self.W

    def n_vis(self, s: int) -> int:
        return sum(self.frame_tokens(f) for f in self.frames(s))

    def spans(self, s: int):
        """Visual spans (start, rows, cols, frame) at step s, in context order."""
        out, t = [], 0
        for f in self.frames(s):
            c, r = self.grid(f)
            out.append((t, r, c, f))
            t += r * c
        return out

    @property
    def appends(self) -> bool:
        """Each step's cache is the previous one plus a frame of the same size
        (old tokens keep their positions)."""
        return self.slots == 0 and not self.res_change

    @property
    def peak_step(self) -> int:
        """The step with the longest cache (buffer sizes are taken there)."""
        return max(range(1, self.steps + 1), key=lambda s: (self.L(s), -s))

    def budgets(self, s: int):
        """B = floor(pct * N_vis / 100) for each budget percentage."""
        return [int(p) * self.n_vis(s) // 100 for p in self.pcts]

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


SPECS = {
    1: WorkloadSpec("tiny-f32-1L-H4G2d64-16x12", 1, 4, 2, 64, "f32", 16, 12,
                    1, 64, 8, (20,), 1.0, 2.0, 1, False, 0.0, 0.25,
                    seed=1001),
    2: WorkloadSpec("qwen25vl7b-1L-1920x1080-1step", 1, 28, 4, 128, "bf16",
                    69, 39, 1, 256, 32, (20,), 0.5, 6.0, 1, False, 0.0,
                    0.35, seed=1002),
    3: WorkloadSpec("qwen25vl7b-28L-5step-1920x1080", 28, 28, 4, 128, "bf16",
                    69, 39, 5, 256, 32, (20,), 0.5, 6.0, 1, True, 0.7, 0.35,
                    seed=1003),
    4: WorkloadSpec("qwen25vl7b-28L-15step-budget-sweep", 28, 28, 4, 128,
                    "bf16", 69, 39, 15, 512, 32, (10, 20, 40), 0.5, 6.0, 1,
                    True, 0.7, 0.35, q_scale_range=(0.5, 2.0), seed=1004),
    5: WorkloadSpec("qwen25vl7b-28L-30step-2560x1440", 28, 28, 4, 128, "bf16",
                    91, 51, 30, 1024, 64, (10,), 0.5, 6.0, 3, False, 0.7,
                    0.35, seed=1005),
    # image_slots = 5 (the multi-step setting of the paper's trajectory
    # benchmark): from step 6 on the oldest screenshot leaves the context;
    # from frame 7 on the screen is 1280x720 (46x26 tokens)
    6: WorkloadSpec("qwen25vl7b-28L-10step-slots5-1080p-720p", 28, 28, 4, 128,
                    "bf16", 69, 39, 10, 256, 32, (20,), 0.5, 6.0, 1, True, 0.7,
                    0.35, seed=1006, slots=5, res_change=((7, 46, 26),)),
}


# --------------------------------------------------------------------------
# storage helpers
# --------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round to nearest, ties to even); returns
    the 16-bit patterns as uint16."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    return ((b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


def to_float64(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 value of stored elements (bf16 bits or float32)."""
    if dtype == "bf16":
        return bf16_bits_to_f32(arr).astype(np.float64)
    return np.asarray(arr, dtype=np.float64)


# --------------------------------------------------------------------------
# the generator
# --------------------------------------------------------------------------

@dataclass
class Trajectory:
    """Deterministic source of one trajectory's inputs.

    Every array is a pure function of (spec.seed, layer, what, index), drawn
    with numpy's PCG64 from np.random.default_rng([seed, layer, key, id]).
    Arrays come back in storage form: uint16 bf16 bit patterns or float32.
    """

    spec: WorkloadSpec
    _centres: dict = field(default_factory=dict)

    def _rng(self, layer: int, key: int, tid: int):
        return np.random.default_rng([self.spec.seed, layer, key, tid])

    def _store(self, x32: np.ndarray) -> np.ndarray:
        if self.spec.dtype == "bf16":
            return f32_to_bf16_bits(x32)
        return np.ascontiguousarray(x32, dtype=np.float32)

    def _u(self, layer: int) -> np.ndarray:
        """Per-group random sign vectors u in {-1, +1}^d."""
        sp = self.spec
        r = self._rng(layer, 0, 4)
        return np.where(r.random((sp.G, sp.d)) < 0.5, -1.0, 1.0).astype(np.float32)

    def _bumped(self, layer: int, g: int) -> bool:
        return (not self.spec.migrate) or (g == layer % self.spec.G)

    def centres(self, layer: int, frame: int):
        """Bump centres [G][regions] of (x, y) for a frame; each keeps the
        previous frame's place with probability repeat_p."""
        sp = self.spec
        key = (layer, frame)
        if key in self._centres:
            return self._centres[key]
        r = self._rng(layer, frame, 3)
        cols, rows = sp.grid(frame)
        fresh = np.stack([r.random((sp.G, sp.regions)) * cols,
                          r.random((sp.G, sp.regions)) * rows], axis=-1)
        keep = r.random((sp.G, sp.regions)) < sp.repeat_p
        if frame > 1:
            prev = self.centres(layer, frame - 1)
            pc, pr = sp.grid(frame - 1)
            if (pc, pr) != (cols, rows):    # same screen place at the new resolution
                prev = prev * np.array([cols / pc, rows / pr])
            fresh = np.where(keep[..., None], prev, fresh)
        self._centres[key] = fresh
        return fresh

    def _bump_profile(self, layer: int, frame: int) -> np.ndarray:
        """[G, N_F] bump amplitude per visual token (float32)."""
        sp = self.spec
        cols, rows = sp.grid(frame)
        rr, cc = np.divmod(np.arange(cols * rows), cols)
        prof = np.zeros((sp.G, cols * rows), dtype=np.float64)
        cen = self.centres(layer, frame)
        for g in range(sp.G):
            if not self._bumped(layer, g):
                continue
            for k in range(sp.regions):
                x, y = cen[g, k]
                prof[g] += sp.amp * np.exp(-((cc - x) ** 2 + (rr - y) ** 2)
                                           / (2.0 * sp.sigma ** 2))
        return prof.astype(np.float32)

    def frame_kv(self, layer: int, frame: int):
        """K, V [G, N_F, d] of one screenshot in one layer."""
        sp = self.spec
        nf = sp.frame_tokens(frame)
        K = self._rng(layer, frame, 0).standard_normal(
            (sp.G, nf, sp.d), dtype=np.float32)
        V = self._rng(layer, frame, 1).standard_normal(
            (sp.G, nf, sp.d), dtype=np.float32)
        prof = self._bump_profile(layer, frame)
        u = self._u(layer)
        K = K + prof[:, :, None] * u[:, None, :]
        return self._store(K), self._store(V)

    def text_kv(self, layer: int, step: int):
        """K, V [G, text, d] of the text tokens at a step."""
        sp = self.spec
        K = self._rng(layer, 10000 + step, 0).standard_normal(
            (sp.G, sp.text, sp.d), dtype=np.float32)
        V = self._rng(layer, 10000 + step, 1).standard_normal(
            (sp.G, sp.text, sp.d), dtype=np.float32)
        return self._store(K), self._store(V)

    def q_scale(self, step: int) -> float:
        sp = self.spec
        if sp.q_scale_range is None:
            return 1.0
        lo, hi = sp.q_scale_range
        return float(self._rng(0, 30000 + step, 5).uniform(lo, hi))

    def window_q(self, layer: int, step: int) -> np.ndarray:
        """Window queries Q [H, W, d] at a step."""
        sp = self.spec
        Q = self._rng(layer, 20000 + step, 2).standard_normal(
            (sp.H, sp.W, sp.d), dtype=np.float32)
        u = self._u(layer)
        grp = (np.arange(sp.H) * sp.G) // sp.H
        Q = Q + np.float32(sp.q_align) * u[grp][:, None, :]
        Q = Q * np.float32(self.q_scale(step))
        return self._store(Q)

    def layer_cache(self, layer: int, step: int):
        """The assembled cache K, V [G, L, d] of a layer at a step."""
        sp = self.spec
        ks, vs = [], []
        for f in sp.frames(step):
            k, v = self.frame_kv(layer, f)
            ks.append(k)
            vs.append(v)
        k, v = self.text_kv(layer, step)
        ks.append(k)
        vs.append(v)
        return np.concatenate(ks, axis=1), np.concatenate(vs, axis=1)


def random_case(seed: int, n_layers: int, H: int, G: int, d: int, L_cap: int,
                W: int, dtype: str, scale: float = 1.0):
    """Plain seeded N(0, scale^2) Q [n_layers, H, W, d] and K, V
    [n_layers, G, L_cap, d] in storage form (edge-case tests)."""
    r = np.random.default_rng([seed, 77])
    Q = (r.standard_normal((n_layers, H, W, d), dtype=np.float32) * np.float32(scale))
    K = (r.standard_normal((n_layers, G, L_cap, d), dtype=np.float32) * np.float32(scale))
    V = r.standard_normal((n_layers, G, L_cap, d), dtype=np.float32)
    if dtype == "bf16":
        return f32_to_bf16_bits(Q), f32_to_bf16_bits(K), f32_to_bf16_bits(V)
    return Q, K, V


# --------------------------------------------------------------------------
# algorithmic traffic and flop counts (what the measurement credits)
# --------------------------------------------------------------------------

def bytes_alg(spec: WorkloadSpec, step: int, B: int) -> int:
    """Mandatory HBM bytes of one layer-call: Q, K_past read once, selected
    K/V rows read and written, window K/V rows read and written, idx."""
    e = spec.elem_bytes
    H, G, d, W = spec.H, spec.G, spec.d, spec.W
    L_p = spec.L_p(step)
    return e * (H * W * d + G * L_p * d + 4 * G * B * d + 4 * G * W * d) + 4 * B


def qk_flops(H: int, W: int, L_p: int, d: int) -> int:
    """Flops of the window-query/key contraction, counted once: 2 H W L_p d."""
    return 2 * H * W * L_p * d


def decode_flops(H: int, n: int, d: int) -> int:
    """Attention flops of one decoded token in one layer over n cached tokens:
    q.K and p.V, 2 H n d each."""
    return 4 * H * n * d
