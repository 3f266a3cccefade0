"""Helpers shared by the GPU tests: seeded inputs on the device, chains run
through the C ABI, and the oracle's expected values for the same epochs.
(Not collected by pytest: no test_ prefix.)"""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2607_08973_amd as S
import synth
from oracle import ref_np, sim

DEV = "cuda:0"


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV)


def to_host(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


def ulp_distance(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """bf16 steps between two bit arrays, +0 == -0."""
    def key(x):
        x = x.astype(np.int32)
        return np.where(x & 0x8000, -(x & 0x7FFF), x)
    return np.abs(key(a) - key(b))


def inject_table(late: np.ndarray, withheld=None) -> list:
    late = np.asarray(late, dtype=np.uint16)
    w = np.zeros_like(late) if withheld is None else np.asarray(withheld, dtype=np.uint16)
    return [int(x) for x in (late | (w << 8))]


def expected_log_words(nranks, late_masks_by_epoch, order, forced=0):
    return sim.predict_log(nranks, late_masks_by_epoch, order, forced)


class StepRun:
    """A handle bound to a device-resident source pool and output ring."""

    def __init__(self, w: synth.Workload, tokens_max: int, validate=None, log_epochs=None,
                 waves_per_group=1, pool=None, **cfg):
        # persistent steps validate before they load (ORDERED); per-epoch
        # launches default to the paper's speculative reduction
        if validate is None:
            validate = "ordered" if cfg.get("persistent") else "spec"
        self.w = w
        self.N, self.H, self.L = w.nranks, w.hidden, w.reduces_per_step
        self.T_max = tokens_max
        self.pool = (pool if pool is not None else
                     synth.payload_pool(w.wid, w.nranks, tokens_max, w.hidden, w.pool_entries(), w.dist))
        self.pool_d = to_dev(self.pool)
        kw = dict(nranks=self.N, hidden=self.H, max_tokens=tokens_max, reduces_per_step=self.L,
                  validate=validate, epilogue=int(w.epilogue), rms_eps=w.rms_eps,
                  log_epochs=log_epochs or self.L, waves_per_group=waves_per_group)
        kw.update(cfg)
        self.s = S.Sifar(**kw)
        if w.epilogue:
            self.res0 = synth.residual_init(w.wid, tokens_max, self.H)
            self.weight = synth.rms_weight(w.wid, self.H)
            self.res_d = to_dev(self.res0)
            self.w_d = to_dev(self.weight)
            self.y_d = torch.zeros((self.L, tokens_max, self.H), dtype=torch.int16, device=DEV)
            self.s.bind_step(self.pool_d, residual=self.res_d, weight=self.w_d, y_ring=self.y_d)
        else:
            self.out_d = torch.zeros((self.L, tokens_max, self.H), dtype=torch.int16, device=DEV)
            self.s.bind_step(self.pool_d, out_ring=self.out_d)

    def step(self, tokens):
        g0, _ = self.s.epochs()
        self.s.step(tokens)
        g1, _ = self.s.epochs()
        return list(range(g1 - self.L, g1))


def read_stamp_log(s: "S.Sifar") -> np.ndarray:
    """The raw-stamp log as [log_epochs][w_max][2][N]: rank r's stamp at a
    chunk's first (index 0) and last (index 1) validation."""
    epochs, _, w_max = s.log_geometry()
    return s.read_stamp_log().reshape(epochs, w_max, 2, s.cfg.nranks)


def stale_mask(stamps: np.ndarray, g: int) -> np.ndarray:
    """Stale-rank masks recomputed from raw stamps [..., N] for epoch g."""
    N = stamps.shape[-1]
    bits = (stamps != (g & 0xFFFFFFFF)).astype(np.uint32) << np.arange(N, dtype=np.uint32)
    return bits.sum(axis=-1).astype(np.uint32)


def replay_logs(log: np.ndarray, stamp_log: np.ndarray, epochs, chunks: int):
    """Replay every logged decision from the stamps logged with it: the first
    and last stale-rank masks of each chunk's word must be the ones its
    first and last stamps imply, and a chunk is accepted (last mask 0) only
    when every stamp it validated against was fresh. Every stale stamp must be
    an earlier epoch of the same slot parity (g - 2k) or the initial 0.
    Returns (words checked, chunks that needed more than one validation)."""
    checked = retried = 0
    for g in epochs:
        row = (g - 1) % log.shape[0]
        words = log[row, :chunks]
        st = stamp_log[row, :chunks]
        first = stale_mask(st[:, 0], g)
        last = stale_mask(st[:, 1], g)
        assert np.array_equal((words >> 16) & 0xFF, first), f"epoch {g}: first masks"
        assert np.array_equal(words >> 24, last), f"epoch {g}: last masks"
        assert np.all(last == 0), f"epoch {g}: a chunk was accepted with a stale stamp"
        stale = st[st != g].astype(np.int64)
        assert np.all((stale == 0) | (((g - stale) % 2 == 0) & (stale < g))), \
            f"epoch {g}: a stale stamp that is not an earlier epoch of the slot"
        checked += chunks
        retried += int(np.count_nonzero((words & 0xFFFF) > 1))
    return checked, retried
