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
def test_prefetching_publication_never_stale(placement):
    """The persistent step's prefetching producer publishes a slot by waiting
    until only the next epoch's source loads are outstanding (vmcnt(8)) before
    it stores the flags on one XCD. With that exact sequence the ORDERED reader
    must accept no stale word in 2.1 million handoffs per placement."""
    print(f"litmus ordered-prefetch placement {placement} pairs {PAIRS} trials {TRIALS}",
          flush=True)
    r = S.sifar_litmus(S.SIFAR_LITMUS_ORDERED_PREFETCH, placement, PAIRS, TRIALS)
    print(r, flush=True)
    assert r["timeouts"] == 0
    assert r["trials"] == PAIRS * TRIALS
    assert r["violations"] == 0, r["first_bad"]
    assert r["pairs_placed"] == PAIRS


@pytest.mark.parametrize("placement", [S.SIFAR_LITMUS_CROSS_XCD, S.SIFAR_LITMUS_SAME_XCD])
def test_read_first_handoff(placement):
    """The paper's read-first order against a live producer. Whether it
    accepts a stale word depends on timing (the interleaving of the paper's
    monotonicity discussion: the payload load served before the producer's
    write arrives, the stamp load after its stamp), so the rate is reported,
    not asserted; every violation found must be a word of an earlier epoch of
    the same slot, or the slot's initial zeros."""
    print(f"litmus read-first placement {placement} pairs {PAIRS} trials {TRIALS}", flush=True)
    r = S.sifar_litmus(S.SIFAR_LITMUS_READ_FIRST, placement, PAIRS, TRIALS)
    print(r, flush=True)
    print(f"read-first violation rate {r['violations'] / r['trials']:.2e} "
          f"({r['violations']} of {r['trials']}, {r['violations_first_epochs']} in the first "
          f"two epochs)", flush=True)
    assert r["timeouts"] == 0
    assert r["trials"] == PAIRS * TRIALS
    if r["violations"]:
        g, found, want, _ = r["first_bad"]
        # a violation is a word of an earlier epoch of the same slot (or, in
        # the first two epochs, the slot's initial zeros)
        step = 0x9E3779B1
        earlier = {(k * step) % (1 << 32) for k in range(2, g + 1, 2)}
        assert (want - found) % (1 << 32) in earlier or (g <= 2 and found == 0)
