"""The statistics and selection kernels launch with a fixed dynamic LDS size;
with their static LDS it must fit the 160 KiB a gfx950 workgroup can hold,
or every launch fails.  Checked on the CPU from a device-only compile of each
source with the library's own flags (hipcc cross-compiles without a GPU)."""

from __future__ import annotations

import math
import os
import re
import shutil
import subprocess

import pytest

from paper_2606_01790_amd import build as B

LDS_LIMIT = 160 * 1024


def _const(src: str, name: str) -> int:
    m = re.search(r"constexpr int %s = ([0-9* ]+);" % name, src)
    assert m, name
    return math.prod(int(f) for f in m.group(1).split("*"))


def _static_lds(source: str, kernel: str, tmp_path) -> int:
    out = tmp_path / (os.path.basename(source) + ".s")
    flags = [f for f in B.HIP_FLAGS if f != "-fPIC"]
    subprocess.run([B.HIPCC, *flags, "-I", B.INCLUDE, "--cuda-device-only", "-S",
                    "-o", str(out), source], check=True, capture_output=True)
    meta = out.read_text().split("amdhsa.kernels:", 1)[1]
    for blk in meta.split("\n  - ")[1:]:
        name = re.search(r"\.name:\s+(\S+)", blk)
        if name and kernel in name.group(1):
            return int(re.search(r"\.group_segment_fixed_size:\s+(\d+)", blk).group(1))
    raise AssertionError(f"{kernel} not found in {source}")


needs_hipcc = pytest.mark.skipif(not (os.path.exists(B.HIPCC) or shutil.which("hipcc")),
                                 reason="hipcc not available")


def _shape(src: str, nt: int) -> int:
    """Dynamic LDS bytes of the statistics kernel's block shape `nt`, from
    the StatsShape specialisation in the source (constants from the source
    and from stats_shape.h)."""
    consts = {m.group(1): int(m.group(2))
              for m in re.finditer(r"constexpr int (k\w+) = (\d+);",
                                   src + open(os.path.join(B.CSRC, "stats_shape.h")).read())}
    body = src.split("struct StatsShape<%d> {" % nt, 1)[1].split("};", 1)[0]

    def value(name):
        expr = re.search(name + r" = ([^,;]+)", body).group(1)
        for k, v in consts.items():
            expr = re.sub(r"\b%s\b" % k, str(v), expr)
        assert re.fullmatch(r"[0-9*+ ]+", expr), expr
        return eval(expr)

    return 4 * (value("kHistInts") + value("kKeyCache") + value("kCand"))


@needs_hipcc
def test_stats_kernel_lds_fits(tmp_path):
    """The wide shape fits one block per CU; the narrow one, launched when
    the blocks outnumber the CUs, must fit two, and the small one four."""
    path = os.path.join(B.CSRC, "state.hip")
    src = open(path).read()
    for fused in ("0", "1"):
        wide = _shape(src, 1024) + _static_lds(path, "stats_kernelILi1024ELb%sE" % fused,
                                               tmp_path)
        assert wide <= LDS_LIMIT, (fused, wide)
    narrow = _shape(src, 512) + _static_lds(path, "stats_kernelILi512", tmp_path)
    assert 2 * narrow <= LDS_LIMIT, narrow
    small = _shape(src, 256) + _static_lds(path, "stats_kernelILi256", tmp_path)
    assert 4 * small <= LDS_LIMIT, small


@needs_hipcc
def test_select_kernel_lds_fits(tmp_path):
    path = os.path.join(B.CSRC, "select.hip")
    src = open(os.path.join(B.CSRC, "select_body.h")).read()
    dynamic = 4 * _const(src, "kSelLdsKeys")
    static = _static_lds(path, "select_kernel", tmp_path)
    assert static + dynamic <= LDS_LIMIT, (static, dynamic)
