"""Seeded synthetic inputs for the one-shot all-reduce workloads.

This module is shared by the CPU oracle's tests and by the GPU path's tests and
benchmark. It holds no arithmetic of the method itself (no summation, no
rounding rule of the reduction, no normalisation): it only draws numbers and
turns them into bf16 bit patterns with PyTorch's own CPU conversion.

The paper's workloads are the all-reduces of tensor-parallel LLM decode
(two per layer, after attention and after the FFN, Sec. 2.4), on hidden
states of a dense 8B model and a large MoE model at batch size 1..4
(Sec. 5 and 6.2). Their activations are not public and not needed: every
payload here is drawn from a stated distribution with a stated seed.

All generators use ``numpy.random.default_rng([ROOT_SEED, *key])`` so that a
workload, rank count, shape and stream id fix the bytes exactly.
"""
from __future__ import annotations

import dataclasses
from typing import Sequence

import numpy as np

ROOT_SEED = 260708973


def rng(*key: int) -> np.random.Generator:
    """Generator for one named stream of a workload."""
    return np.random.default_rng([ROOT_SEED, *[int(k) for k in key]])


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) of float values, via PyTorch's CPU cast."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def draw(gen: np.random.Generator, shape: Sequence[int], dist: str) -> np.ndarray:
    """Float32 samples of one of the named distributions.

    ``normal``   N(0, 1)
    ``act``      decode activations: N(0, 1) * 0.5, each element independently
                 scaled by 50 with probability 0.001 (outlier channels)
    ``uniform``  U(-1, 1)
    ``weight``   N(1, 0.02)   (RMSNorm gain)
    ``ones``     all 1.0
    """
    shape = tuple(int(s) for s in shape)
    if dist == "normal":
        x = gen.standard_normal(shape)
    elif dist == "act":
        x = gen.standard_normal(shape) * 0.5
        outlier = gen.random(shape) < 0.001
        x = np.where(outlier, x * 50.0, x)
    elif dist == "uniform":
        x = gen.uniform(-1.0, 1.0, shape)
    elif dist == "weight":
        x = gen.normal(1.0, 0.02, shape)
    elif dist == "ones":
        x = np.ones(shape)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    return x.astype(np.float32)


def bf16(gen: np.random.Generator, shape: Sequence[int], dist: str) -> np.ndarray:
    return f32_to_bf16_bits(draw(gen, shape, dist))


def payload_pool(workload: int, nranks: int, tokens: int, hidden: int, entries: int,
                 dist: str, stream: int = 0) -> np.ndarray:
    """Pool of per-rank partial sums: uint16 ``[entries][nranks][tokens][hidden]``.

    Entry ``e`` holds the N ranks' partials for every epoch ``g`` with
    ``(g - 1) % entries == e``. With ``entries = 3L + 1`` for a chain of L
    reduces, stale data from two epochs earlier never equals fresh data and
    successive decode steps do not repeat a layer's inputs in lockstep.
    """
    g = rng(workload, nranks, tokens, hidden, stream)
    return bf16(g, (entries, nranks, tokens, hidden), dist)


def delay_table(workload: int, nranks: int, epochs: int, prob: float,
                stream: int = 7) -> np.ndarray:
    """Stale-stamp injection table: uint8 ``[epochs]``, bit r set when rank r's
    epoch stamp is written late at epoch ``g`` (entry ``(g - 1) % epochs``).

    Each (epoch, rank) is delayed independently with probability ``prob``.
    """
    if nranks > 8:
        raise ValueError("at most 8 ranks fit a uint8 mask")
    g = rng(workload, nranks, epochs, stream)
    bits = g.random((epochs, nranks)) < prob
    weights = (1 << np.arange(nranks)).astype(np.uint16)
    return (bits.astype(np.uint16) * weights).sum(axis=1).astype(np.uint8)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: shapes, chain length and value recipe."""

    wid: int
    name: str
    nranks: int
    tokens: tuple
    hidden: int
    reduces_per_step: int
    steps: int
    dist: str
    stale_prob: float = 0.0
    epilogue: bool = False
    rms_eps: float = 1e-6

    def pool_entries(self) -> int:
        return 3 * self.reduces_per_step + 1


# Workloads of the decode-time all-reduce, named by what they are.
SMOKE_N2 = Workload(1, "n2-t1-h4096-chain64", 2, (1,), 4096, 64, 1, "normal")
LLAMA8B_DECODE = Workload(2, "llama8b-decode-n8-h4096-chain64", 8, (1, 2, 4, 8), 4096,
                          64, 100, "act")
SPEC_STRESS = Workload(3, "spec-stress-n8-t4-h4096-stale0.1", 8, (4,), 4096, 64, 200,
                       "act", stale_prob=0.1)
PAYLOAD_SWEEP = tuple(
    Workload(4, f"sweep-n{n}-t{t}-h{h}", n, (t,), h, 100, 10, "uniform")
    for n in (2, 4, 8) for t in (1, 16, 64, 256) for h in (4096, 8192))
MOE_DECODE = Workload(5, "moe-decode-n8-h8192-chain120-rmsnorm", 8, (1, 8, 32), 8192,
                      120, 100, "act", stale_prob=0.05, epilogue=True)

ALL = (SMOKE_N2, LLAMA8B_DECODE, SPEC_STRESS, *PAYLOAD_SWEEP, MOE_DECODE)


def residual_init(workload: int, tokens: int, hidden: int) -> np.ndarray:
    """Initial residual stream, uint16 ``[tokens][hidden]``, N(0, 1)."""
    return bf16(rng(workload, tokens, hidden, 11), (tokens, hidden), "normal")


def rms_weight(workload: int, hidden: int) -> np.ndarray:
    """RMSNorm gain, uint16 ``[hidden]``, N(1, 0.02)."""
    return bf16(rng(workload, hidden, 13), (hidden,), "weight")
