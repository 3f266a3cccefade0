"""GPU: a C11 client of the C ABI (tests/c_abi_client.c) -- no Python or
PyTorch between it and libsifar -- reduces seeded partials eagerly, in one
decode step and through the allocation-free entry point; its outputs are
checked bit for bit against the oracle."""
from __future__ import annotations

import ctypes
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2607_08973_amd as S
import synth

pytestmark = pytest.mark.gpu

CLIENT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libc_abi_client.so")


@pytest.fixture(scope="module")
def client():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    S.load()
    assert os.path.exists(CLIENT), "build() compiles the C client first"
    lib = ctypes.CDLL(CLIENT)
    lib.sifar_c_client.restype = ctypes.c_int
    lib.sifar_c_client.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_char_p)]
    yield lib
    torch.cuda.synchronize()


def run_client(lib, args):
    argv = (ctypes.c_char_p * len(args))(*[a.encode() for a in args])
    return lib.sifar_c_client(len(args), argv)


@pytest.mark.parametrize("persistent", [0, 1])
@pytest.mark.parametrize("N,T,H,L", [(8, 2, 4096, 8), (3, 5, 1000, 6)])
def test_c_client_matches_oracle(client, tmp_path, N, T, H, L, persistent):
    print(f"c client N={N} T={T} H={H} L={L} persistent={persistent}", flush=True)
    E = 5
    pool = synth.payload_pool(200 + N, N, T, H, E, "normal")
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    pool.tofile(src)
    rc = run_client(client, ["c_abi_client", str(N), str(T), str(H), str(L), str(persistent),
                             str(src), str(dst)])
    assert rc == 0
    got = np.fromfile(dst, dtype=np.uint16).reshape(2 * E + L, T, H)
    for e in range(E):                       # eager epochs 1..E
        assert np.array_equal(got[e], oracle.reduce(pool[e])), f"eager epoch {e + 1}"
    base = E + (E & 1)                       # a step starts at an even epoch base
    for i in range(L):
        g = base + i + 1
        assert np.array_equal(got[E + i], oracle.reduce(pool[(g - 1) % E])), f"step node {i}"
    for e in range(E):                       # sifar_allreduce_noalloc, entry by entry
        assert np.array_equal(got[E + L + e], oracle.reduce(pool[e])), f"allocation-free {e}"


def test_c_client_reports_bad_arguments(client, tmp_path):
    assert run_client(client, ["c_abi_client"]) == 2
    missing = str(tmp_path / "missing.bin")
    assert run_client(client, ["c_abi_client", "2", "1", "512", "2", "0", missing,
                               str(tmp_path / "o.bin")]) == 2
