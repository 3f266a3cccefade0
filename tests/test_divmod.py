"""The kernels' multiply-high remainder (ring rows, source-pool entries),
checked on the host against the % operator: every divisor up to 4096 with
edge and random dividends, and random large divisors. The same header the
kernels include is compiled for the host with hipcc; no GPU is used."""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

from paper_2607_08973_amd import build as B

HERE = os.path.dirname(os.path.abspath(__file__))


def test_mod_u32_matches_the_remainder_operator(tmp_path):
    hipcc = shutil.which("hipcc") or ("/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc")
                                      else None)
    if hipcc is None:
        pytest.skip("hipcc not available")
    exe = tmp_path / "divmod_check"
    cmd = [hipcc, "-O2", "-std=c++17", "-I", B.CSRC, "-I", B.INCLUDE,
           os.path.join(HERE, "divmod_check.hip"), "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.startswith("ok"), out.stdout
