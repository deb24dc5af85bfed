"""The C ABI on the CPU: the library loads, exports what include/starkv.h
declares, and rejects bad arguments on the host before any GPU work.

No test here launches a kernel: every call either only computes sizes or
fails validation, which happens before the first HIP call.
"""

import ctypes
import json
import os
import re

import pytest

from paper_2606_01790_amd import starkv as sk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "starkv.h")

pytestmark = pytest.mark.skipif(not os.path.exists(sk.LIB_PATH),
                                reason="libstarkv.so not built")

FAKE = 0x10000          # an aligned non-null address; never dereferenced here


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(starkv_[a-z_]+)\s*\(", text)))


def test_header_symbols_are_exported():
    L = sk.lib()
    names = declared_functions()
    assert len(names) == 15
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(sk.SIGNATURES)


def test_abi_version_and_status_strings():
    L = sk.lib()
    assert L.starkv_abi_version() == 2
    assert L.starkv_status_str(0) == b"ok"
    assert b"budget" in L.starkv_status_str(3)


def test_defaults_match_paper_table():
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "hparams.json")))
    p = sk.params_default()
    assert p.lam == pytest.approx(g["lambda"])
    assert (p.n_warmup, p.n_ramp) == (g["online_profiling_steps"], g["lambda_ramp_steps"])
    assert p.rho_mi == pytest.approx(g["mi_ema_decay"])
    assert p.tau == pytest.approx(g["prior_temperature_tau"])
    assert p.rho_t == pytest.approx(g["temporal_ema_decay"])
    assert p.delta == pytest.approx(g["temporal_delta"])
    assert p.d_min == pytest.approx(g["temporal_d_min"])
    assert [p.t_min, p.t_max] == pytest.approx(g["aeb_t_range"]["ScreenSpot-Pro/UI-TARS"])
    assert (p.n_bins, p.grid, p.pool_kernel) == (8, 8, 5)


def dims(**kw):
    base = dict(n_layers=28, H=28, G=4, d=128, L=13711, W=32, dtype=sk.BF16)
    base.update(kw)
    return sk.make_dims(**base)


def test_sizes():
    d = dims()
    assert sk.scalars_count(d) == 4 * 4 + 4
    # state: 64-byte header, MI_bar, m[G][cap], padded to 256 per layer
    per = (64 + 16 + 4 * 2691 * 4 + 255) // 256 * 256
    assert sk.state_bytes(d, 2691) == 28 * per
    ws = sk.workspace_bytes(d)
    Lp = 13711 - 32
    chunks = (Lp + 255) // 256
    up = lambda x: (x + 255) // 256 * 256  # noqa: E731
    part = up(28 * 4 * chunks * 224 * 8)    # per-chunk row statistics
    assert ws == part + up(28 * 4 * Lp * 4)
    assert sk.workspace_bytes(dims(G=3)) == 0          # H % G != 0


def test_sizes_per_head():
    """Per-head subspaces (Ns = H): S, the scalar block and the state have a
    row per head; the pass-1 row statistics stay per KV group."""
    d = dims(per_head=True)
    assert d.Ns == 28
    assert sk.scalars_count(d) == 4 * 28 + 4
    per = (64 + 28 * 4 + 28 * 2691 * 4 + 255) // 256 * 256
    assert sk.state_bytes(d, 2691) == 28 * per
    Lp = 13711 - 32
    chunks = (Lp + 255) // 256
    up = lambda x: (x + 255) // 256 * 256  # noqa: E731
    assert sk.workspace_bytes(d) == up(28 * 4 * chunks * 224 * 8) + up(28 * 28 * Lp * 4)
    # MHA: both settings describe the same subspaces
    m0, m1 = dims(G=28, W=8), dims(G=28, W=8, per_head=True)
    assert (sk.workspace_bytes(m0), sk.scalars_count(m0)) == \
        (sk.workspace_bytes(m1), sk.scalars_count(m1))


@pytest.mark.parametrize("kw,code", [
    (dict(G=3), "E_SHAPE"),
    (dict(d=96), "E_SHAPE"),
    (dict(W=13711), "E_SHAPE"),
    (dict(W=0), "E_SHAPE"),
    (dict(n_layers=0), "E_SHAPE"),
    (dict(dtype=7), "E_DTYPE"),
    (dict(W=80), "E_SHAPE"),       # 80*7 = 560 window rows > 512
    (dict(W=12, per_head=True), "E_SHAPE"),    # a head's rows not whole 8-row groups
    (dict(H=72, G=4, W=8, per_head=True), "E_SHAPE"),   # 72 subspaces > 64
])
def test_score_rejects_bad_dims(kw, code):
    d = dims(**kw)
    p = sk.params_default()
    lay = sk.KVLayout(4 * 13711 * 128, 13711 * 128, 128)
    rc = sk.lib().starkv_score(ctypes.byref(d), ctypes.byref(p), FAKE, FAKE,
                               ctypes.byref(lay), FAKE, FAKE, FAKE, FAKE, 1 << 40, None)
    assert sk.STATUS[rc] == code


def test_score_rejects_unknown_subspace_mode():
    d = dims()
    d.per_head = 2
    assert _score(d) == "E_SHAPE"
    assert sk.workspace_bytes(d) == 0


def _score(d, p=None, lay=None, q=FAKE, k=FAKE, ws=FAKE, ws_bytes=1 << 40):
    p = p or sk.params_default()
    lay = lay or sk.KVLayout(4 * 13711 * 128, 13711 * 128, 128)
    return sk.STATUS[sk.lib().starkv_score(ctypes.byref(d), ctypes.byref(p), q, k,
                                           ctypes.byref(lay), FAKE, FAKE, FAKE, ws,
                                           ws_bytes, None)]


def test_score_rejects_bad_arguments():
    d = dims()
    assert _score(d, q=None) == "E_NULL"
    assert _score(d, q=FAKE + 8) == "E_ALIGN"
    assert _score(d, lay=sk.KVLayout(0, 0, 100)) == "E_SHAPE"
    assert _score(d, lay=sk.KVLayout(0, 0, 132)) == "E_ALIGN"
    assert _score(d, ws_bytes=sk.workspace_bytes(d) - 1) == "E_WORKSPACE"
    assert _score(d, ws=None) == "E_WORKSPACE"
    p = sk.params_default()
    p.pool_kernel = 4
    assert _score(d, p=p) == "E_PARAM"


def _update(d, spans, frame, p=None, cap=2691):
    p = p or sk.params_default()
    arr, n = sk.spans_array(spans)
    return sk.STATUS[sk.lib().starkv_update_state(
        ctypes.byref(d), ctypes.byref(p), FAKE, FAKE, arr, n, frame, FAKE, cap,
        FAKE, None, 0, None)]


def test_variant_params_are_validated():
    d = dims()
    for field, bad in (("tem_decay", 3), ("tem_decay", -1), ("aeb_mode", 2)):
        p = sk.params_default()
        assert (p.tem_decay, p.aeb_mode) == (0, 0)
        setattr(p, field, bad)
        assert _update(d, [(0, 39, 69, 1)], 1, p=p) == "E_PARAM"


def test_update_state_rejects_bad_spans_and_params():
    d = dims(L=2947)                         # L_p = 2915
    ok = [(0, 39, 69, 1)]
    assert _update(d, [(0, 39, 69, 1)], 2) == "E_SPANS"        # frame not present
    assert _update(d, [(300, 39, 69, 1)], 1) == "E_SPANS"      # runs past L_p
    assert _update(d, [(0, 3, 3, 1), (5, 2, 2, 2)], 2) == "E_SPANS"   # overlap
    assert _update(d, [(20, 3, 3, 1), (0, 2, 2, 2)], 2) == "E_SPANS"  # unsorted
    assert _update(d, [(0, 3, 3, 1), (9, 2, 2, 1)], 1) == "E_SPANS"   # same frame
    assert _update(d, [(0, 3, 3, 3), (9, 2, 2, 1)], 1) == "E_SPANS"   # frame > F
    assert _update(d, [(0, 0, 3, 1)], 1) == "E_SPANS"
    assert _update(d, ok, 1, cap=100) == "E_STATE"
    for field, val in [("lam", 1.5), ("rho_mi", 1.0), ("tau", 0.0), ("rho_t", -0.1),
                       ("delta", -1.0), ("d_min", 2.0), ("t_min", 0.0),
                       ("t_max", 0.5), ("n_bins", 0), ("grid", 17), ("eps", -1.0),
                       ("n_warmup", -1), ("pool_kernel", 0)]:
        p = sk.params_default()
        setattr(p, field, val)
        assert _update(d, ok, 1, p=p) == "E_PARAM", field
    assert _update(d, [(0, 1, 1, 0)] * 65, 0) == "E_SPANS"      # too many spans


def test_select_and_compact_reject_bad_budget():
    d = dims(L=2947)
    p = sk.params_default()
    arr, n = sk.spans_array([(0, 39, 69, 1)])
    L = sk.lib()
    for B in (-1, 2916):
        rc = L.starkv_select(ctypes.byref(d), ctypes.byref(p), FAKE, FAKE, FAKE, arr, n,
                             1, B, FAKE, FAKE, None, 0, None)
        assert sk.STATUS[rc] == "E_BUDGET"
        lay = sk.KVLayout(4 * 2947 * 128, 2947 * 128, 128)
        rc = L.starkv_compact(ctypes.byref(d), FAKE, FAKE, ctypes.byref(lay), FAKE, B,
                              FAKE, FAKE, None)
        assert sk.STATUS[rc] == "E_BUDGET"
    rc = L.starkv_select(ctypes.byref(d), ctypes.byref(p), FAKE, FAKE, FAKE, arr, n,
                         1, 5, FAKE, None, None, 0, None)
    assert sk.STATUS[rc] == "E_NULL"
    lay = sk.KVLayout(4 * 2947 * 128, 2947 * 128, 128)
    rc = L.starkv_compact(ctypes.byref(d), FAKE, FAKE, ctypes.byref(lay), FAKE, 5,
                          FAKE + 4, FAKE, None)
    assert sk.STATUS[rc] == "E_ALIGN"


def _update_select(d, spans, frame, B=5, cap=2691, p=None, S=FAKE, gstar=FAKE, s=FAKE,
                   idx=FAKE):
    p = p or sk.params_default()
    arr, n = sk.spans_array(spans)
    return sk.STATUS[sk.lib().starkv_update_state_select(
        ctypes.byref(d), ctypes.byref(p), S, FAKE, gstar, arr, n, frame, FAKE, cap, FAKE, B,
        s, idx, None, 0, None)]


def test_update_state_select_validates_both_argument_lists():
    """The combined call rejects what either call rejects, before any launch."""
    d = dims(L=2947)                         # L_p = 2915
    ok = [(0, 39, 69, 1)]
    for B in (-1, 2916):
        assert _update_select(d, ok, 1, B=B) == "E_BUDGET"
    assert _update_select(d, ok, 1, B=5, idx=None) == "E_NULL"
    assert _update_select(d, ok, 1, S=None) == "E_NULL"
    assert _update_select(d, ok, 1, gstar=None) == "E_NULL"
    assert _update_select(d, ok, 1, s=None) == "E_NULL"
    assert _update_select(d, [(0, 39, 69, 1)], 2) == "E_SPANS"
    assert _update_select(d, [(300, 39, 69, 1)], 1) == "E_SPANS"
    assert _update_select(d, ok, 1, cap=100) == "E_STATE"
    assert _update_select(d, ok, 1, s=FAKE + 2) == "E_ALIGN"
    p = sk.params_default()
    p.tau = 0.0
    assert _update_select(d, ok, 1, p=p) == "E_PARAM"
    bad = dims(L=2947)
    bad.G = 3                                # H % G != 0
    assert _update_select(bad, ok, 1) == "E_SHAPE"


def test_state_init_rejects():
    d = dims()
    L = sk.lib()
    assert sk.STATUS[L.starkv_state_init(ctypes.byref(d), None, 10, None)] == "E_NULL"
    assert sk.STATUS[L.starkv_state_init(ctypes.byref(d), FAKE, -1, None)] == "E_STATE"
    assert sk.STATUS[L.starkv_state_init(ctypes.byref(d), FAKE + 4, 1, None)] == "E_ALIGN"


def _decode(d, n=1000, q=FAKE, k=FAKE, v=FAKE, out=FAKE, lay=None, ws=FAKE, ws_bytes=1 << 40):
    lay = lay or sk.KVLayout(4 * 1000 * 128, 1000 * 128, 128)
    return sk.STATUS[sk.lib().starkv_decode(ctypes.byref(d), q, k, v, ctypes.byref(lay), n,
                                            out, ws, ws_bytes, None)]


def test_decode_validation_and_workspace():
    d = dims()
    assert _decode(d, q=None) == "E_NULL"
    assert _decode(d, n=0) == "E_SHAPE"
    assert _decode(dims(dtype=sk.F32)) == "E_DTYPE"
    assert _decode(dims(H=34, G=2)) == "E_SHAPE"          # 17 heads per group > 16
    assert _decode(d, lay=sk.KVLayout(0, 0, 100)) == "E_SHAPE"
    assert _decode(d, lay=sk.KVLayout(0, 0, 132)) == "E_ALIGN"
    assert _decode(d, k=FAKE + 8) == "E_ALIGN"
    ws = sk.decode_workspace_bytes(d, 2723)
    # 28 layers x 4 groups, 11 splits of <= 256 tokens, 7 heads x (d + 2) floats
    assert ws == (28 * 4 * 11 * 7 * 130 * 4 + 255) // 256 * 256
    assert _decode(d, n=2723, ws_bytes=ws - 1) == "E_WORKSPACE"
    assert sk.decode_workspace_bytes(d, 0) == 0


def test_noalloc_rejects_workspace_beyond_its_array():
    """starkv_score_noalloc checks its workspace need against the library's
    array on the host: a 200000-token, W = 64 step needs more than 64 MiB."""
    dims = sk.make_dims(28, 28, 4, 128, 200000, 64, sk.BF16)
    assert sk.workspace_bytes(dims) > 64 << 20
    lay = sk.KVLayout(4 * 200000 * 128, 200000 * 128, 128)
    code = sk.lib().starkv_score_noalloc(
        ctypes.byref(dims), ctypes.byref(sk.params_default()), FAKE, FAKE,
        ctypes.byref(lay), FAKE, FAKE, FAKE, None)
    assert sk.STATUS[code] == "E_WORKSPACE"
    small = sk.make_dims(1, 4, 2, 64, 256, 8, sk.F32)
    code = sk.lib().starkv_score_noalloc(
        ctypes.byref(small), ctypes.byref(sk.params_default()), None, FAKE,
        ctypes.byref(sk.KVLayout(2 * 256 * 64, 256 * 64, 64)), FAKE, FAKE, FAKE, None)
    assert sk.STATUS[code] == "E_NULL"
