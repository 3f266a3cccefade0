"""Register budgets of the persistent step kernels, checked at compile time.

A persistent step needs every one of its waves resident at once. The payload
sweep's largest step (N = 8, T = 256, H = 8192: 4096 chunks) fills an MI355X
exactly: 8192 one-wave workgroups, i.e. 8 waves per SIMD, which gfx950 grants
only to kernels of at most 64 VGPRs. Compiling the
device code here (hipcc cross-compiles without a GPU) catches a change that
pushes those kernels past the budget before a GPU run skips or refuses the
step. No GPU is used.
"""
from __future__ import annotations

import os
import re
import shutil
import subprocess

import pytest

from paper_2607_08973_amd import build as B

VGPRS_FOR_8_WAVES_PER_SIMD = 64


def _hipcc():
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return None


@pytest.fixture(scope="module")
def kernel_resources(tmp_path_factory):
    """{mangled kernel name: {"vgpr": n, "spill": n}} from the device assembly."""
    hipcc = _hipcc()
    if hipcc is None:
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("isa") / "kernels.s"
    flags = [f for f in B.FLAGS if f not in ("-fPIC", "-shared")]
    cmd = [hipcc, *flags, "--cuda-device-only", "-S", "-I", B.INCLUDE, "-I", B.CSRC,
           os.path.join(B.CSRC, "kernels.hip"), "-o", str(out)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    text = out.read_text()
    found = {}
    # kernel metadata entries: ".name: <sym>" ... ".vgpr_count: n", ".vgpr_spill_count: n"
    for m in re.finditer(r"\.name:\s+(\S+)\n(.*?)(?=\n\s+- \.|\n\s+-\s|\Z)", text, re.S):
        body = m.group(2)
        v = re.search(r"\.vgpr_count:\s+(\d+)", body)
        if v:
            s = re.search(r"\.vgpr_spill_count:\s+(\d+)", body)
            found[m.group(1)] = {"vgpr": int(v.group(1)), "spill": int(s.group(1)) if s else 0}
    assert found, "no kernel metadata in the device assembly"
    return found


def _chain(n, epi, grouped, prefetch):
    b = lambda x: "1" if x else "0"
    return (f"_ZN5sifar12_GLOBAL__N_112chain_kernelILi{n}ELi1ELb{b(epi)}ELb{b(grouped)}"
            f"ELb{b(prefetch)}EEEvNS_9ChainArgsE")


def test_largest_steps_fit_eight_waves_per_simd(kernel_resources):
    """The non-prefetching one-wave kernel of a plain N = 8 step stays within
    64 VGPRs (the form init falls back to when a step needs every wave slot of
    the GPU). Plain steps have no grouped kernel: only epilogue steps group."""
    name = _chain(8, False, False, False)
    assert name in kernel_resources, name
    assert kernel_resources[name]["vgpr"] <= VGPRS_FOR_8_WAVES_PER_SIMD, (
        name, kernel_resources[name])
    assert _chain(8, False, True, False) not in kernel_resources


def test_prefetching_kernel_keeps_its_occupancy(kernel_resources):
    """The prefetching one-wave kernel (the llama8b decode step's) holds two
    epochs' sources. At most 80 VGPRs keeps 6 waves per SIMD, enough for
    one-wave steps of up to 3072 chunks (larger handles fall back to the
    non-prefetching form), and it does not spill. (A producer slot wait
    without its short sleep once took it to 109.)"""
    name = _chain(8, False, False, True)
    assert name in kernel_resources, name
    r = kernel_resources[name]
    assert r["vgpr"] <= 80 and r["spill"] == 0, (name, r)
