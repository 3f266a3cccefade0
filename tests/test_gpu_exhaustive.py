"""GPU: every one of the 2^32 ordered pairs of bf16 bit patterns (a, b) reduced
at N=2 by the HIP path and by the C oracle (fixed-order fp32 sum, one bf16
rounding). 65,536 all-reduces of 65,536 elements: block k holds a = every
pattern along the row and b = 256 consecutive patterns down the tokens.

The oracle converts by definition and is slow (about a second per block on
one core), so the blocks are checked on up to 16 host threads while the GPU
runs ahead; measured about 8 s in all on an MI355X host. NaN outputs are
checked as NaN only (their payload bits are outside the contract).
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
import paper_2607_08973_amd as S
from oracle import ref_np

pytestmark = pytest.mark.gpu

from sifar_harness import DEV


def test_every_bf16_pair_on_gpu_against_oracle():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    S.load()
    H, T = 65536, 256
    blocks = 65536 // T
    a_host = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    a_dev = torch.from_numpy(a_host.view(np.int16).copy()).to(DEV)
    x_dev = torch.empty((2, T, H), dtype=torch.int16, device=DEV)
    out = torch.empty((T, H), dtype=torch.int16, device=DEV)

    def check(k: int, got: np.ndarray):
        x = np.empty((2, T, H), np.uint16)
        x[0] = a_host[None, :]
        x[1] = (np.arange(T, dtype=np.uint32) + k * T).astype(np.uint16)[:, None]
        exp = oracle.reduce(x)
        fin = ~np.isnan(ref_np.widen(exp))
        bad = int(np.count_nonzero(got[fin] != exp[fin]))
        bad += int(np.count_nonzero(~np.isnan(ref_np.widen(got[~fin]))))
        return k, bad, int(np.count_nonzero(~fin))

    workers = max(1, min(16, (os.cpu_count() or 1)))
    mismatches, nans, done = 0, 0, 0
    with S.Sifar(nranks=2, hidden=H, max_tokens=T, reduces_per_step=2, log_epochs=4) as s, \
            ThreadPoolExecutor(workers) as pool:
        pending = []
        for k in range(blocks):
            x_dev[0].copy_(a_dev.expand(T, H))
            b = (np.arange(T, dtype=np.uint32) + k * T).astype(np.uint16).view(np.int16)
            x_dev[1].copy_(torch.from_numpy(b.copy()).to(DEV)[:, None].expand(T, H))
            s.produce(x_dev, T)
            s.reduce(out, T)
            got = out.cpu().numpy().view(np.uint16)
            pending.append(pool.submit(check, k, got))
            while len(pending) > 2 * workers or (k == blocks - 1 and pending):
                kk, bad, nan = pending.pop(0).result()
                mismatches += bad
                nans += nan
                done += 1
                if done % 32 == 0:
                    print(f"blocks checked {done}/{blocks}, mismatches {mismatches}", flush=True)
        s.check()
    assert done == blocks
    print(f"pairs {blocks * T * H}, NaN outputs {nans}, mismatches {mismatches}", flush=True)
    assert mismatches == 0
