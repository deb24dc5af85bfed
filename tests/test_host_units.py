"""Host-side units built with the host compiler (no GPU, no HIP).

1. The C ABI's validation layer (validate.cpp, api.cpp) under the address
   and undefined-behaviour sanitizers, with stub kernel launches: every
   status code of include/starkv.h comes back where the header says.
2. The spatial-cell arithmetic of the statistics kernel (grid_cell.h, the
   same source the kernel compiles) against exact integer arithmetic, up to
   the largest frames the boundary accepts (rows * cols <= 2^26).
3. The statistics kernel's block-shape choice (stats_shape.h) on the
   workloads' shapes and around every threshold.
"""

import os
import random
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_01790_amd", "csrc")
INC = os.path.join(ROOT, "include")
HOST = os.path.join(ROOT, "tests", "host")

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="no host compiler")


def _build(tmp_path, name, sources, sanitize):
    exe = str(tmp_path / name)
    cmd = ["g++", "-std=c++17", "-g", "-O1", f"-I{INC}", f"-I{CSRC}", *sources, "-o", exe]
    if sanitize:
        cmd[1:1] = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-fno-omit-frame-pointer"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def test_abi_validation_under_sanitizers(tmp_path):
    exe = _build(tmp_path, "abi_driver",
                 [os.path.join(HOST, "abi_driver.cpp"), os.path.join(CSRC, "validate.cpp"),
                  os.path.join(CSRC, "api.cpp")], sanitize=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    assert "checks passed" in r.stdout
    codes = {int(line.rsplit("-> ", 1)[1]) for line in r.stdout.splitlines()
             if line.startswith("ok ") and "status string" not in line
             and "launch count" not in line and "bytes" not in line
             and "count" not in line}
    # every starkv_status value 0..10 occurs
    assert set(range(11)) <= codes, sorted(codes)


def _cells(exe, cases):
    inp = "".join(f"{p} {rows} {cols} {M}\n" for p, rows, cols, M in cases)
    r = subprocess.run([exe], input=inp, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    return [tuple(map(int, line.split())) for line in r.stdout.splitlines()]


def test_grid_cells_exact_at_large_positions(tmp_path):
    exe = _build(tmp_path, "grid_cell_driver", [os.path.join(HOST, "grid_cell_driver.cpp")],
                 sanitize=True)
    rnd = random.Random(5)
    cases = []
    big = 1 << 26                                   # largest span the boundary accepts
    small = 1 << 22                                 # the reciprocal-estimate path's limit
    for rows, cols in [(big, 1), (big // 2, 2), (big // 3, 3), (1, big), (8191, 8192),
                       (4096 * 4, 4096), (39, 69), (51, 91), (26, 46), (4000, 4000),
                       (3, big // 3), (7, 3), (1, 1), (1025, 1023), (2, 1024)]:
        n = rows * cols
        for M in (1, 7, 8, 16):
            pts = {0, n - 1, n // 2, n // 3, min(n - 1, 33554434), min(n - 1, (1 << 25) - 1),
                   min(n - 1, small - 1), min(n - 1, small), min(n - 1, 1023)}
            pts |= {rnd.randrange(n) for _ in range(40)}
            pts |= {rnd.randrange(min(n, 1024)) for _ in range(20)}
            cases += [(p, rows, cols, M) for p in sorted(pts)]
    got = _cells(exe, cases)
    assert len(got) == len(cases)
    for (p, rows, cols, M), (r, c, cell, ok) in zip(cases, got):
        assert (r, c) == divmod(p, cols), (p, rows, cols)
        want = (r * M // rows) * M + (c * M // cols)
        assert cell == want, (p, rows, cols, M, cell, want)
        assert 0 <= cell < M * M
        # the kernel's span-entry path: reciprocal estimates one ulp off
        assert ok == 1, (p, rows, cols, M)


def test_small_quotient_exact_near_every_multiple(tmp_path):
    exe = _build(tmp_path, "grid_cell_driver", [os.path.join(HOST, "grid_cell_driver.cpp")],
                 sanitize=False)
    r = subprocess.run([exe, "quot"], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    bad, checked = map(int, r.stdout.split())
    assert checked > 10**6 and bad == 0, (bad, checked)


def test_statistics_block_shape(tmp_path):
    """Wide (1024) when every block fits one per CU or the bins need it;
    small (256) when even two per CU leave a second round and K <= 9,
    M*M <= 64; narrow (512) otherwise."""
    exe = _build(tmp_path, "stats_shape", [os.path.join(HOST, "stats_shape_driver.cpp")],
                 sanitize=False)
    cases = [
        # (blocks, CUs, K, M) -> shape
        ((28 * 6, 256, 8, 8), 1024),      # 28 layers, 4 groups: the five-frame trajectory
        ((28 * 33, 256, 8, 8), 256),      # per-head subspaces
        ((28 * 33, 256, 12, 8), 512),     # per-head, more bins than the small shape holds
        ((28 * 33, 256, 8, 9), 512),      # per-head, more cells than the small shape holds
        ((28 * 33, 256, 18, 8), 1024),    # more bins than the narrow shape holds
        ((48 * 6, 256, 8, 8), 512),       # between one and two blocks per CU
        ((96 * 6, 256, 9, 8), 256),
        ((96 * 6, 256, 10, 8), 512),
        ((96 * 6, 256, 8, 16), 512),
        ((256, 256, 17, 16), 1024),       # exactly one per CU
        ((257, 256, 17, 16), 512),
        ((512, 256, 9, 8), 512),          # exactly two per CU
        ((513, 256, 9, 8), 256),
        ((513, 256, 1, 1), 256),
        ((1, 1, 64, 16), 1024),
    ]
    inp = "".join(f"{b} {c} {k} {m}\n" for (b, c, k, m), _ in cases)
    r = subprocess.run([exe], input=inp, capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    got = [int(x) for x in r.stdout.split()]
    assert got == [want for _, want in cases], list(zip(cases, got))
    # blocks per layer: one per subspace (MI), one AEB block, and one
    # stability block per eight subspaces (four groups: 6; 28 heads: 33)
    subs = [1, 4, 7, 8, 9, 16, 17, 28, 63, 64]
    r = subprocess.run([exe, "layer"], input="".join(f"{n}\n" for n in subs),
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    got = [tuple(map(int, line.split())) for line in r.stdout.splitlines()]
    assert got == [(-(-n // 8), n + 1 - (-n // 8)) for n in subs], list(zip(subs, got))
    assert got[1][1] == 6 and got[7][1] == 33
