"""Pins of the protocol simulator (oracle/sim.py).

The protocol is the paper's: dual-buffered payloads and flags (Sec. 3.3, 4.1),
speculative reads validated by per-rank flags with a retry loop (Sec. 3.5,
4.2), a flag that grows by one per all-reduce (Sec. 4.2), and correctness that
rests on the monotonicity assumption (Sec. 8.1). Expected outcomes below are
fixed by that reasoning, by brute force over every interleaving of small
instances, and by the paper's own counter-example narrative.
"""
from __future__ import annotations

import os

import numpy as np
import pytest

import oracle
from oracle import sim

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_brute_force_matches_memoised_search():
    """N=2 ranks, 2 epochs: walk every interleaving one by one and compare the
    outcome counts with the memoised search."""
    for order in ("ordered", "spec_po"):
        m = sim.Model(nranks=2, epochs=2, attempts=1, order=order, rank_ordered_reads=True)
        assert sim.enumerate_paths(m) == sim.explore(m)
    m = sim.Model(nranks=2, epochs=1, attempts=2, order="spec")
    assert sim.enumerate_paths(m) == sim.explore(m)


def test_path_count_closed_form():
    """With attempts=1 and in-order reads, the number of complete+truncated
    interleavings of ORDERED at N=2, E=1 is the multinomial of three chains:
    two producers of 2 events and the consumer's 4 reads: 8!/(2!2!4!) = 420."""
    m = sim.Model(nranks=2, epochs=1, attempts=1, order="ordered", rank_ordered_reads=True)
    assert sum(sim.explore(m).values()) == 420


@pytest.mark.parametrize("m", [
    sim.Model(2, 2, 2, "ordered"),
    sim.Model(2, 3, 3, "ordered"),
    sim.Model(3, 2, 2, "ordered"),
    sim.Model(2, 3, 2, "ordered", buffers="single"),
])
def test_ordered_never_accepts_stale(m):
    res = sim.explore(m)
    assert not any(wrong for (_, wrong, _), n in res.items() if n)
    assert res.get(("complete", False, False), 0) > 0


@pytest.mark.parametrize("order", ["spec", "spec_po"])
def test_read_first_can_accept_stale_only_by_the_monotonicity_pattern(order):
    # explore() raises if a wrong accept is not the Sec. 8.1 pattern, or if the
    # flag-sum check and the per-rank check ever disagree.
    for m in (sim.Model(2, 2, 2, order), sim.Model(2, 3, 3, order), sim.Model(3, 2, 2, order)):
        res = sim.explore(m)
        assert sum(n for (_, wrong, _), n in res.items() if wrong) > 0


@pytest.mark.parametrize("order", ["ordered", "spec_po"])
def test_waw_guard_is_what_keeps_ordered_sound(order):
    """Dropping the dual-buffer rule (a slot rewritten before the reduction two
    epochs back has finished) makes even ORDERED accept stale data; a single
    buffer needs the bottom barrier (rewrite only after the previous
    reduction) to stay sound."""
    bad = sim.explore(sim.Model(2, 3, 2, order, buffers="dual_noguard"))
    assert sum(n for (_, wrong, _), n in bad.items() if wrong) > 0
    bad1 = sim.explore(sim.Model(2, 3, 2, order, buffers="single_noguard"))
    assert sum(n for (_, wrong, _), n in bad1.items() if wrong) > 0


def test_flag_sum_check_needs_the_guard():
    """The paper validates sum(flags) == N * flag (Sec. 4.2). With the WAW
    guard, stamps seen for epoch e are e or older and the sum check equals the
    per-rank check (explore raises otherwise). Without it a rank can be ahead
    and the sum of a stale and an early stamp can match."""
    res = sim.explore(sim.Model(2, 3, 2, "ordered", buffers="single_noguard"))
    assert sum(n for (_, _, sumdis), n in res.items() if sumdis) > 0


def _load_golden(name):
    model, events, expect = None, [], None
    for line in open(os.path.join(GOLDEN, name)):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        head, *rest = line.split()
        if head == "model":
            kv = dict(x.split("=") for x in rest)
            model = sim.Model(int(kv["nranks"]), int(kv["epochs"]), int(kv["attempts"]),
                              kv["order"], kv["buffers"])
        elif head == "expect":
            expect = {k: bool(int(v)) for k, v in (x.split("=") for x in rest)}
        else:
            events.append((head, int(rest[0])))
    return model, events, expect


def test_paper_counterexample_fixture():
    m, events, expect = _load_golden("monotonicity_counterexample.txt")
    s, log = sim.initial(m), []
    for e in events:
        assert e in sim.enabled(m, s), e
        s = sim.step(m, s, e, log)
    d = log[-1]
    assert d.accept == expect["accept"]
    assert d.wrong == expect["wrong"]
    assert d.pattern == expect["pattern"]
    # the same producer timing cannot fool ORDERED: stamps are read first
    mo = sim.Model(2, 1, 1, "ordered", "dual")
    s = sim.initial(mo)
    for e in [("P", 1), ("P", 1), ("R", 2), ("R", 3)]:
        s = sim.step(mo, s, e)
    # rank 0's stamp was read before it wrote: the attempt is rejected
    for e in [("R", 0), ("R", 1)]:
        s = sim.step(mo, s, e)
    assert s.ck == 0 and not s.wrong


def _versions_to_outputs(pool_by_epoch, decisions, nranks):
    """Numeric output of every accepted attempt: the reduction of the versions
    that were actually read (version v = the data of epoch v, 0 = zeros)."""
    outs = {}
    for d in decisions:
        if d.accept:
            x = np.stack([pool_by_epoch[v][r] for r, v in enumerate(d.versions)])
            outs[d.epoch] = oracle.reduce(x)
    return outs


@pytest.mark.parametrize("order", ["ordered", "spec"])
def test_permuted_schedules_give_the_plain_sum(order):
    """N=8, 64 epochs, seeded random interleavings. ORDERED outputs, and SPEC
    outputs on schedules free of the monotonicity pattern, equal the plain
    fixed-order sum of each epoch's data."""
    import synth
    N, E = 8, 64
    pool = synth.payload_pool(90, N, 1, 256, E, "act")
    by_epoch = {0: np.zeros((N, 1, 256), np.uint16)}
    by_epoch.update({e: pool[e - 1] for e in range(1, E + 1)})
    m = sim.Model(N, E, 10 ** 6, order)
    rng = np.random.default_rng(1234)
    checked = 0
    for trial in range(6):
        s, log = sim.run_schedule(m, sim.random_chooser(rng))
        assert s.ce == E + 1
        if order == "spec" and any(d.pattern for d in log if d.accept):
            assert any(d.wrong for d in log)
            continue
        outs = _versions_to_outputs(by_epoch, log, N)
        for e in range(1, E + 1):
            assert np.array_equal(outs[e], oracle.reduce(by_epoch[e]))
        checked += 1
    assert checked >= 1


def test_mode_d_log_prediction_closed_form():
    """Late flags land after the first failed validation: attempts are
    1 + [late], the first mask is the late mask, the last mask is empty. With
    k forced retries the first k validations fail regardless (Sec. 6.3's
    forced-retry measurement): attempts = 1 + max(k, [late])."""
    import synth
    for N in (2, 4, 8):
        late = synth.delay_table(3, N, 200, 0.1)
        for order in ("spec", "ordered"):
            for k in (0, 1, 3):
                got = sim.mode_d_decisions(N, late, order, forced_retries=k)
                for (att, first, last), m in zip(got, late):
                    assert att == 1 + max(k, int(m != 0))
                    assert first == m and last == 0


def test_log_word_packing():
    assert sim.pack_log(2, 0x81, 0) == 0x00810002
    assert sim.unpack_log(sim.pack_log(70000, 5, 3)) == (0xFFFF, 5, 3)
