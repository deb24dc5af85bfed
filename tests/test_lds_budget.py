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


@needs_hipcc
def test_stats_kernel_lds_fits(tmp_path):
    path = os.path.join(B.CSRC, "state.hip")
    src = open(path).read()
    dynamic = 4 * (_const(src, "kHistInts") + _const(src, "kKeyCache") + _const(src, "kCand"))
    static = _static_lds(path, "stats_kernel", tmp_path)
    assert static + dynamic <= LDS_LIMIT, (static, dynamic)


@needs_hipcc
def test_select_kernel_lds_fits(tmp_path):
    path = os.path.join(B.CSRC, "select.hip")
    src = open(path).read()
    dynamic = 4 * _const(src, "kLdsKeys")
    static = _static_lds(path, "select_kernel", tmp_path)
    assert static + dynamic <= LDS_LIMIT, (static, dynamic)
