"""Interleaving simulator of SiFAR's stamp / validate / retry protocol.
TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

What is modelled (one chunk; chunks are independent copies of the protocol):

* N ranks each run a producer: for epoch e = 1, 2, ... it writes its partial
  into its payload slot (event ``Pw(r, e)``) and then writes its flag, the epoch
  stamp ``e``, into the validation buffer (event ``Ps(r, e)``). This is the
  paper's "preceding operation writes its result, then each GPU writes a flag"
  (Sec. 4.1, speculative reduction design). Program order:
  Pw(r,e) < Ps(r,e) < Pw(r,e+1).
* Dual buffering (Sec. 3.3 and 4.1): epoch e uses slot and stamp of parity
  e mod 2, and a slot is rewritten only after the reduction that read it two
  epochs earlier has completed: Pw(r, e) is enabled only after Cdone(e - 2).
  Variants drop that guard (the WAW hazard the bottom barrier prevents) or use
  a single slot.
* One consumer reduces epochs 1..E in order. An attempt reads every rank's
  payload (``Rd``) and stamp (``Rs``), then accepts iff every stamp equals e
  (per-rank equality; the paper sums the flags and compares with N * flag,
  Sec. 4.2 -- both checks are evaluated and must agree). A rejected attempt is
  re-run (Sec. 4.2's retry loop), at most A attempts; a chunk that runs out of
  attempts is "truncated", not wrong.
* Orders of the reads inside an attempt:
    ``spec``     payload and stamp reads in any order (the paper's payload
                 warps and its concurrent validation warp, Sec. 4.2)
    ``spec_po``  all payload reads, then all stamp reads (read first, validate
                 after)
    ``ordered``  all stamp reads (acquire), then all payload reads

An accepted attempt is wrong when some payload version read differs from e.
The monotonicity failure of Sec. 8.1 is the pattern, for a rank r of the
accepted attempt, Rd(r) < Pw(r, e) < Ps(r, e) < Rs(r): the payload was read
before that rank wrote it and its flag after it caught up.

Every function here is deterministic; ``explore`` visits every interleaving of
the events (explicit-state search with memoisation on the full state, which
includes every bit of history a checked property depends on).
"""
from __future__ import annotations

import dataclasses
import functools
import itertools
from collections import Counter
from typing import Dict, Iterable, List, NamedTuple, Optional, Tuple

U32 = 1 << 32


@dataclasses.dataclass(frozen=True)
class Model:
    nranks: int = 2
    epochs: int = 2
    attempts: int = 2
    order: str = "spec"          # spec | spec_po | ordered
    buffers: str = "dual"        # dual | dual_noguard | single | single_noguard
    rank_ordered_reads: bool = False  # reads of one kind issued in rank order

    def parity(self, e: int) -> int:
        return 0 if self.buffers.startswith("single") else (e & 1)

    @property
    def guarded(self) -> bool:
        return not self.buffers.endswith("noguard")

    def write_enabled(self, e: int, cdone: int) -> bool:
        if self.buffers == "dual":
            return cdone >= e - 2
        if self.buffers == "single":
            return cdone >= e - 1
        return True


class State(NamedTuple):
    """Full protocol state (hashable)."""
    pp: tuple      # producer position per rank: 2(e-1) -> next is Pw(r,e), 2(e-1)+1 -> Ps(r,e)
    slot: tuple    # per rank (version in parity 0, version in parity 1); 0 = initial data
    stamp: tuple   # per rank (stamp in parity 0, stamp in parity 1); 0 = never written
    ce: int        # consumer's epoch (epochs + 1 when finished)
    ck: int        # consumer's attempt (0 = truncated)
    done: int      # reads done in this attempt: bit r = Rd(r), bit N+r = Rs(r)
    vread: tuple   # version read per rank in this attempt (-1 = not yet)
    sread: tuple   # stamp read per rank (-1 = not yet)
    early: int     # ranks whose Rd happened before Pw(r, ce)
    wrong: bool    # some accepted attempt so far returned a stale version
    sumdis: bool   # the flag-sum check and the per-rank check disagreed once


def initial(m: Model) -> State:
    n = m.nranks
    return State((0,) * n, ((0, 0),) * n, ((0, 0),) * n, 1, 1, 0,
                 (-1,) * n, (-1,) * n, 0, False, False)


def _set(t: tuple, i: int, v) -> tuple:
    return t[:i] + (v,) + t[i + 1:]


def _set2(t: tuple, i: int, j: int, v) -> tuple:
    inner = list(t[i])
    inner[j] = v
    return t[:i] + (tuple(inner),) + t[i + 1:]


class Violation(AssertionError):
    pass


@dataclasses.dataclass
class Decision:
    """One validation decision of the consumer."""
    epoch: int
    attempt: int
    stamps: Tuple[int, ...]
    versions: Tuple[int, ...]
    accept: bool
    sum_accept: bool
    wrong: bool
    pattern: bool


def enabled(m: Model, s: State) -> List[tuple]:
    """Events enabled in state s: ('P', r) producer step of rank r, ('R', i) read i."""
    pp, ce, ck, done = s.pp, s.ce, s.ck, s.done
    n, E = m.nranks, m.epochs
    ev = []
    cdone = ce - 1
    for r in range(n):
        pos = pp[r]
        if pos >= 2 * E:
            continue
        e = pos // 2 + 1
        if pos % 2 == 0 and not m.write_enabled(e, cdone):
            continue
        ev.append(("P", r))
    if ck >= 1 and ce <= E:
        rd_mask = (1 << n) - 1
        rs_mask = rd_mask << n
        if m.order == "spec":
            allowed = (1 << 2 * n) - 1
        elif m.order == "spec_po":
            allowed = rd_mask if (done & rd_mask) != rd_mask else rs_mask
        elif m.order == "ordered":
            allowed = rs_mask if (done & rs_mask) != rs_mask else rd_mask
        else:
            raise ValueError(m.order)
        cand = [i for i in range(2 * n) if (allowed >> i) & 1 and not (done >> i) & 1]
        if m.rank_ordered_reads:
            # keep only the lowest pending read of each kind
            firsts = []
            for lo, hi in ((0, n), (n, 2 * n)):
                ks = [i for i in cand if lo <= i < hi]
                if ks:
                    firsts.append(min(ks))
            cand = firsts
        ev.extend(("R", i) for i in cand)
    return ev


def step(m: Model, s: State, event: tuple, log: Optional[list] = None) -> State:
    pp, slot, stamp, ce, ck, done, vread, sread, early, wrong, sumdis = s
    n = m.nranks
    kind, i = event
    if kind == "P":
        r = i
        pos = pp[r]
        e = pos // 2 + 1
        p = m.parity(e)
        if pos % 2 == 0:
            slot = _set2(slot, r, p, e)
        else:
            stamp = _set2(stamp, r, p, e)
        pp = _set(pp, r, pos + 1)
        return State(pp, slot, stamp, ce, ck, done, vread, sread, early, wrong, sumdis)
    # consumer read
    p = m.parity(ce)
    if i < n:
        r = i
        vread = _set(vread, r, slot[r][p])
        if pp[r] <= 2 * (ce - 1):          # Pw(r, ce) has not happened yet
            early |= 1 << r
    else:
        r = i - n
        sread = _set(sread, r, stamp[r][p])
    done |= 1 << i
    if done != (1 << 2 * n) - 1:
        return State(pp, slot, stamp, ce, ck, done, vread, sread, early, wrong, sumdis)
    # validation of this attempt
    accept = all(x == ce for x in sread)
    sum_accept = (sum(sread) % U32) == (n * ce) % U32
    if accept != sum_accept:
        if m.guarded:
            raise Violation(f"sum check {sum_accept} != per-rank check {accept} at {s}")
        sumdis = True
    is_wrong = accept and any(v != ce for v in vread)
    pattern = any((early >> r) & 1 and sread[r] == ce for r in range(n))
    if log is not None:
        log.append(Decision(ce, ck, tuple(sread), tuple(vread), accept, sum_accept,
                            is_wrong, pattern))
    if m.buffers == "dual" and accept and is_wrong != pattern:
        raise Violation(f"monotonicity characterisation fails at {s}")
    wrong = wrong or is_wrong
    if accept:
        ce, ck = ce + 1, 1
    else:
        ck = ck + 1 if ck < m.attempts else 0
    return State(pp, slot, stamp, ce, ck, 0, (-1,) * n, (-1,) * n, 0, wrong, sumdis)


def _outcome(m: Model, s: State) -> Tuple[str, bool, bool]:
    status = "complete" if s.ce > m.epochs else ("truncated" if s.ck == 0 else "stuck")
    return (status, s.wrong, s.sumdis)


def explore(m: Model) -> Dict[Tuple[str, bool, bool], int]:
    """Count every interleaving of the model's events by outcome.

    Keys: (status, wrong, sumdis) with status 'complete' (all epochs
    accepted), 'truncated' (an epoch ran out of attempts) or 'stuck'
    (producers blocked forever); wrong = some accepted attempt returned a
    stale version; sumdis = the flag-sum check and the per-rank check
    disagreed at some validation (only possible without the WAW guard).
    Raises Violation if, with the WAW guard, the two checks ever disagree or,
    with dual buffers, a wrong accept is not exactly the Sec. 8.1 pattern.
    """

    @functools.lru_cache(maxsize=None)
    def go(s: State) -> Tuple[Tuple[Tuple[str, bool], int], ...]:
        ev = enabled(m, s)
        if not ev:
            return ((_outcome(m, s), 1),)
        acc: Counter = Counter()
        for e in ev:
            for k, v in go(step(m, s, e)):
                acc[k] += v
        return tuple(sorted(acc.items()))

    res = dict(go(initial(m)))
    go.cache_clear()
    return res


def enumerate_paths(m: Model) -> Dict[Tuple[str, bool, bool], int]:
    """Same counts as ``explore`` by walking every interleaving one by one (no
    memoisation). Only for tiny models: it is the brute-force cross-check."""
    counts: Counter = Counter()
    stack = [initial(m)]
    while stack:
        s = stack.pop()
        ev = enabled(m, s)
        if not ev:
            counts[_outcome(m, s)] += 1
            continue
        for e in ev:
            stack.append(step(m, s, e))
    return dict(counts)


def run_schedule(m: Model, choose, max_events: int = 10 ** 7) -> Tuple[State, List[Decision]]:
    """Run one interleaving picked by ``choose(state, enabled_events) -> event``."""
    s = initial(m)
    log: List[Decision] = []
    for _ in range(max_events):
        ev = enabled(m, s)
        if not ev:
            return s, log
        s = step(m, s, choose(s, ev), log)
    raise RuntimeError("schedule did not terminate")


def random_chooser(rng):
    def choose(s, ev):
        return ev[int(rng.integers(len(ev)))]
    return choose


# ---------------------------------------------------------------------------
# Deterministic stale injection ("mode D"): the log the GPU must reproduce.
#
# Per epoch g a mask of ranks whose flag is late. The producer writes every
# payload and the flags of the on-time ranks before the reduction of g starts;
# the late ranks' flags land right after the consumer's first failed
# validation. With forced retries k the consumer additionally treats its first
# k validations as failed (the forced-retry measurement of Sec. 6.3).

LOG_ATTEMPTS_MASK = 0xFFFF


def pack_log(attempts: int, mask_first: int, mask_last: int) -> int:
    """Log word: bits 0-15 attempts (saturating), 16-23 stale mask of the first
    attempt, 24-31 stale mask of the last attempt."""
    return (min(attempts, LOG_ATTEMPTS_MASK) | ((mask_first & 0xFF) << 16)
            | ((mask_last & 0xFF) << 24))


def unpack_log(word: int) -> Tuple[int, int, int]:
    return word & LOG_ATTEMPTS_MASK, (word >> 16) & 0xFF, (word >> 24) & 0xFF


def mode_d_decisions(nranks: int, late_masks: Iterable[int], order: str = "spec",
                     forced_retries: int = 0) -> List[Tuple[int, int, int]]:
    """Simulate the mode-D schedule epoch by epoch on the protocol model and
    return (attempts, first mask, last mask) per epoch."""
    late_masks = list(late_masks)
    E = len(late_masks)
    m = Model(nranks=nranks, epochs=E, attempts=2 + forced_retries + 1, order=order,
              rank_ordered_reads=True)
    s = initial(m)
    out = []
    for e in range(1, E + 1):
        late = late_masks[e - 1]
        # producer: every payload, then every on-time flag, of epoch e
        for r in range(nranks):
            s = step(m, s, ("P", r))                 # Pw(r, e)
            if not (late >> r) & 1:
                s = step(m, s, ("P", r))             # Ps(r, e)
        attempts, first, last = 0, None, 0
        while s.ce == e:
            log: List[Decision] = []
            for i in (range(2 * nranks) if order != "ordered"
                      else itertools.chain(range(nranks, 2 * nranks), range(nranks))):
                s = step(m, s, ("R", i), log)
            d = log[-1]
            attempts += 1
            mask = sum(1 << r for r in range(nranks) if d.stamps[r] != e)
            if first is None:
                first = mask
            last = mask
            forced = attempts <= forced_retries
            if d.accept and forced:
                # a forced retry: undo the acceptance, re-run the attempt
                s = s._replace(ce=e, ck=attempts + 1, done=0, vread=(-1,) * nranks,
                               sread=(-1,) * nranks, early=0)
            if attempts == 1 and late:
                for r in range(nranks):
                    if (late >> r) & 1:
                        s = step(m, s, ("P", r))     # the late flag lands
            if s.ck == 0:
                raise RuntimeError("mode-D schedule truncated")
        out.append((attempts, first, last))
    return out


def predict_log(nranks: int, late_masks: Iterable[int], order: str = "spec",
                forced_retries: int = 0) -> List[int]:
    return [pack_log(a, f, l) for a, f, l in
            mode_d_decisions(nranks, late_masks, order, forced_retries)]
