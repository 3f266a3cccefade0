"""GPU: the handoff litmus. The persistent step's reader (stamps, then acquire
from another XCD, then payload) must never accept a payload word of another
epoch, across XCDs or on one XCD, over millions of dual-buffered handoffs."""
from __future__ import annotations

import pytest
import torch

import paper_2607_08973_amd as S

pytestmark = pytest.mark.gpu

PAIRS, TRIALS = 256, 8192  # 2.1 million handoffs per placement


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    S.load()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("placement", [S.SIFAR_LITMUS_CROSS_XCD, S.SIFAR_LITMUS_SAME_XCD])
def test_ordered_handoff_never_stale(placement):
    print(f"litmus ordered placement {placement} pairs {PAIRS} trials {TRIALS}", flush=True)
    r = S.sifar_litmus(S.SIFAR_LITMUS_ORDERED, placement, PAIRS, TRIALS)
    print(r, flush=True)
    assert r["timeouts"] == 0
    assert r["trials"] == PAIRS * TRIALS
    assert r["violations"] == 0, r["first_bad"]
    assert r["pairs_placed"] == PAIRS


@pytest.mark.parametrize("placement", [S.SIFAR_LITMUS_CROSS_XCD, S.SIFAR_LITMUS_SAME_XCD])
def test_read_first_handoff(placement):
    """The paper's read-first order against a live producer. Across XCDs it
    accepts words of an earlier epoch (measured: about 0.2 % of the handoffs
    with 256 pairs), which shows that the litmus sees the hazard the ORDERED
    reader closes; on one XCD the rate is only reported."""
    print(f"litmus read-first placement {placement} pairs {PAIRS} trials {TRIALS}", flush=True)
    r = S.sifar_litmus(S.SIFAR_LITMUS_READ_FIRST, placement, PAIRS, TRIALS)
    print(r, flush=True)
    assert r["timeouts"] == 0
    assert r["trials"] == PAIRS * TRIALS
    if placement == S.SIFAR_LITMUS_CROSS_XCD:
        assert r["violations"] > 0
    if r["violations"]:
        g, found, want, _ = r["first_bad"]
        # a violation is a word of an earlier epoch of the same slot (or, in
        # the first two epochs, the slot's initial zeros)
        step = 0x9E3779B1
        earlier = {(k * step) % (1 << 32) for k in range(2, g + 1, 2)}
        assert (want - found) % (1 << 32) in earlier or (g <= 2 and found == 0)
