"""GPU: the latency-floor probes run, finish their bounded waits, and land in
plausible ranges; the handoff probes run where they say (different XCDs, or
one XCD)."""
from __future__ import annotations

import math

import pytest
import torch

import paper_2607_08973_amd as S

pytestmark = pytest.mark.gpu

KINDS = [
    (S.SIFAR_FLOOR_GRAPH_NODE, 256),
    (S.SIFAR_FLOOR_EAGER_LAUNCH, 256),
    (S.SIFAR_FLOOR_ATOMIC, 4096),
    (S.SIFAR_FLOOR_ACQUIRE_LOAD, 4096),
    (S.SIFAR_FLOOR_COHERENT_LOAD, 4096),
    (S.SIFAR_FLOOR_WARM_LOAD, 4096),
    (S.SIFAR_FLOOR_COLD_LOAD, 1024),
    (S.SIFAR_FLOOR_RELEASE_FENCE, 4096),
    (S.SIFAR_FLOOR_PINGPONG_XCD, 2048),
    (S.SIFAR_FLOOR_PINGPONG_SAME_XCD, 2048),
]


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    S.load()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("kind,iterations", KINDS)
def test_floor_probe_completes(kind, iterations):
    print(f"floor kind {kind} x {iterations}", flush=True)
    ns, info = S.sifar_floor(kind, iterations)
    assert info[0] == 1
    # every floor is a single operation: more than a nanosecond, less than 100 us
    assert math.isfinite(ns) and 1.0 < ns < 1e5, ns
    assert 0 <= info[1] < 8 and 0 <= info[2] < 8
    if kind == S.SIFAR_FLOOR_PINGPONG_XCD:
        assert info[1] != info[2], info
    if kind == S.SIFAR_FLOOR_PINGPONG_SAME_XCD:
        assert info[1] == info[2], info


def test_floors_order():
    """A load that misses every cache costs more than one of recently read
    data."""
    warm, _ = S.sifar_floor(S.SIFAR_FLOOR_WARM_LOAD, 4096)
    cold, _ = S.sifar_floor(S.SIFAR_FLOOR_COLD_LOAD, 1024)
    assert cold > warm, (cold, warm)
