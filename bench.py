#!/usr/bin/env python3
"""Benchmark: microseconds per all-reduce of the emulated SiFAR one-shot
all-reduce on one MI355X, decode-shaped workload of a dense 8B model.

Workload ("llama8b-decode-n8-h4096-chain64"): N = 8 emulated tensor-parallel
ranks, hidden 4096 bf16, batch 1, 2, 4 and 8 tokens (8-64 KiB per rank), 64
chained all-reduces per decode step (32 layers x 2). Synthetic activations
N(0,1)*0.5 with 0.1 % outliers x50, seeded. Inputs are resident in HBM before
timing starts.

One benchmark step = one decode step of 64 all-reduces for each of the four
batch sizes: 256 all-reduces. By default (--persistent 1) a decode step is one
persistent kernel launch whose consumer waves poll the stamps before they load
the payload (ORDERED: no speculation) while producer waves play the peers
concurrently; --persistent 0 replays a captured graph with one launch per
all-reduce, whose reduction is the paper's speculative one (SPEC).

Printed JSON line (rank 0):
  value            microseconds per all-reduce over the timed steps (HIP events
                   around the step launches; includes the emulated peers'
                   writes and every dispatch gap)
  roofline         the dominant kernel: one consumer's algorithmic bytes per
                   launch (read N*K, write K, stamps; the emulated peers'
                   copies are reported apart) over its average launch period,
                   from HIP events on the launching stream; frac_cold the same
                   for steps run right after a 512 MiB scrub of the caches
  spec_graph       the speculative per-launch chain on the same workload, with
                   its own dominant kernel's fraction
  cpu_baseline     the CPU oracle on this host, on a bounded sample
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E


def reduce_bytes(N: int, T: int, H: int) -> int:
    """Algorithmic bytes of one all-reduce: read N payloads of T*H bf16, write
    one result, read N 4-byte stamps per 512-element chunk."""
    K = T * H * 2
    chunks = T * ((H + 511) // 512)
    return N * K + K + 4 * N * chunks


def epilogue_bytes(T: int, H: int) -> int:
    """Extra algorithmic bytes of the fused residual-add + RMSNorm: read and
    write the residual, write y (K each), read the weight (2H)."""
    return 3 * T * H * 2 + 2 * H


def produce_bytes(N: int, T: int, H: int) -> int:
    """Algorithmic bytes of the emulated peers' write of one epoch: read N
    partials, write them into the N slots, write N stamps per chunk."""
    K = T * H * 2
    chunks = T * ((H + 511) // 512)
    return 2 * N * K + 4 * N * chunks


def latency_floors() -> dict:
    """The library's latency probes (sifar_floor): launch and graph-node
    floors, one agent-scope atomic, acquire / coherent / warm / cache-missing
    load, a release fence after a store, a release -> acquire handoff across
    and within an XCD; and the dual-buffered slot loop of the handoff litmus
    (sifar_litmus), per epoch."""
    import paper_2607_08973_amd as S

    probes = (  # (name in the JSON line, kind, operations, scale from ns)
        ("graph_node_us", S.SIFAR_FLOOR_GRAPH_NODE, 256, 1e-3),
        ("eager_launch_us", S.SIFAR_FLOOR_EAGER_LAUNCH, 256, 1e-3),
        ("atomic_ns", S.SIFAR_FLOOR_ATOMIC, 4096, 1.0),
        ("acquire_load_ns", S.SIFAR_FLOOR_ACQUIRE_LOAD, 4096, 1.0),
        ("coherent_load_ns", S.SIFAR_FLOOR_COHERENT_LOAD, 4096, 1.0),
        ("warm_load_ns", S.SIFAR_FLOOR_WARM_LOAD, 4096, 1.0),
        ("cold_load_ns", S.SIFAR_FLOOR_COLD_LOAD, 2048, 1.0),
        ("release_fence_ns", S.SIFAR_FLOOR_RELEASE_FENCE, 4096, 1.0),
        ("handoff_cross_xcd_ns", S.SIFAR_FLOOR_PINGPONG_XCD, 4096, 1.0),
        ("handoff_same_xcd_ns", S.SIFAR_FLOOR_PINGPONG_SAME_XCD, 4096, 1.0),
    )
    out = {}
    for name, kind, ops, scale in probes:
        ns, info = S.sifar_floor(kind, ops)
        out[name] = round(ns * scale, 4 if scale != 1.0 else 1)
        if kind in (S.SIFAR_FLOOR_PINGPONG_XCD, S.SIFAR_FLOOR_PINGPONG_SAME_XCD):
            out[name.replace("_ns", "_xccs")] = info[1:3]
    # the persistent step's own per-chunk loop (dual-buffered slot, stamps,
    # release of the slot) with nothing else in it: 8 producer/consumer pairs,
    # as many as the chunks of one 4096-wide token
    for name, place in (("slot_loop_same_xcd_ns", S.SIFAR_LITMUS_SAME_XCD),
                        ("slot_loop_cross_xcd_ns", S.SIFAR_LITMUS_CROSS_XCD)):
        r = S.sifar_litmus(S.SIFAR_LITMUS_ORDERED, place, 8, 65536)
        out[name] = round(r["ns_per_trial"], 1)
    return out


def graph_floor_us(nodes: int) -> float:
    """Per-node time of a captured graph of minimal kernels (one-element
    in-place add): the dispatch floor every launch of a chain pays."""
    import torch

    x = torch.zeros(1, device="cuda:0")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for _ in range(3):
            x.add_(1.0)
    torch.cuda.current_stream().wait_stream(s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(nodes):
            x.add_(1.0)
    for _ in range(3):
        g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 20
    a.record()
    for _ in range(reps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1e3 / (reps * nodes)


TRAFFIC_PROFILES = {
    "persistent": os.path.join(ROOT, "profiles", "chain_llama8b_decode_n8_h4096.md"),
    "fused": os.path.join(ROOT, "profiles", "fused_reduce_llama8b_decode_n8_h4096.md"),
}


KERNEL_SOURCES = ("kernels.hip", "coherence.h", "sifar_kernels.h")


def kernel_code_digest() -> str:
    """sha256 of the kernel sources (kernels.hip and the headers it includes
    from csrc/) with comments, trailing blanks and empty lines removed: it
    changes when the kernel code does, not when a comment does."""
    import hashlib
    import re

    code = []
    for name in KERNEL_SOURCES:
        src = open(os.path.join(ROOT, "paper_2607_08973_amd", "csrc", name)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        lines = [re.sub(r"//.*$", "", ln).rstrip() for ln in src.splitlines()]
        code.append("\n".join(ln for ln in lines if ln))
    return hashlib.sha256("\n".join(code).encode()).hexdigest()


def measured_traffic(kind):
    """HBM bytes per launch of the dominant kernel from the committed FETCH_SIZE /
    WRITE_SIZE profile, or None when the kernel code changed since."""
    path = TRAFFIC_PROFILES[kind]
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and line.split(":")[0] in ("traffic_bytes_per_launch", "kernel_code_digest"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_code_digest") != kernel_code_digest() or "traffic_bytes_per_launch" not in kv:
        return None
    return float(kv["traffic_bytes_per_launch"])


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--mode", default=None, choices=["spec", "ordered", "none"],
                    help="validation; default: ordered for persistent steps (the only "
                         "mode they accept), spec for one launch per all-reduce")
    ap.add_argument("--fuse", type=int, default=1, choices=[0, 1],
                    help="1: the peers' next write shares the reduction's launch")
    ap.add_argument("--persistent", type=int, default=1, choices=[0, 1],
                    help="1: one persistent launch per decode step (peers and reduction "
                         "concurrent); 0: one launch per all-reduce")
    ap.add_argument("--buffers", type=int, default=2, choices=[1, 2],
                    help="2: dual buffering; 1: one slot per rank (bottom barrier)")
    ap.add_argument("--floor-nodes", type=int, default=64)
    ap.add_argument("--workload", default="llama8b-decode",
                    choices=["llama8b-decode", "smoke-n2", "spec-stress", "sweep", "moe-rmsnorm",
                             "ablation", "retry-curve", "reduce-cold", "litmus", "misspec-vs-tp"],
                    help="llama8b-decode is the headline line; the others print one "
                         "JSON line per configuration")
    ap.add_argument("--wpg", type=int, default=1, choices=[1, 2, 4, 8, 16],
                    help="reduce-cold: waves per workgroup of the reduction kernel")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="budget of the CPU-oracle baseline (0 disables it)")
    ap.add_argument("--spec-graph", type=int, default=1,
                    help="persistent runs: also time the speculative per-launch chain (1)")
    ap.add_argument("--wide-points", type=int, default=1,
                    help="also time the chain at 16 and 64 tokens (1) or not (0: profiling "
                         "runs, whose averages cover the headline launches only)")
    args = ap.parse_args()
    steps_persistent = args.persistent and args.workload not in ("ablation", "reduce-cold",
                                                                 "litmus")
    if args.mode is None:
        args.mode = "ordered" if steps_persistent else "spec"
    if steps_persistent and args.mode != "ordered":
        raise SystemExit("persistent steps validate before they load: use --mode ordered "
                         "(or --persistent 0 for spec / none)")
    return args


def cpu_baseline(pool, tokens, budget_s):
    """The C oracle, single-threaded, on the same pool entries the GPU reduces."""
    import numpy as np
    import oracle

    per_t = {}
    for T in tokens:
        xs = [np.ascontiguousarray(pool[e][:, :T]) for e in range(8)]
        n, t0 = 0, time.perf_counter()
        while True:
            oracle.reduce(xs[n % len(xs)])
            n += 1
            el = time.perf_counter() - t0
            if el > budget_s / len(tokens):
                break
        per_t[T] = el / n * 1e6
    mean_us = sum(per_t.values()) / len(per_t)
    return mean_us, per_t


def cpu_baseline_parallel(pool, tokens, budget_s, threads):
    """The same C oracle on `threads` native host threads (oracle's pthread
    driver: each thread runs the oracle's reduction on a contiguous slice of
    the T x H elements; bit-identical, checked once against the
    single-threaded call)."""
    import numpy as np
    import oracle

    per_t = {}
    for T in tokens:
        xs = [np.ascontiguousarray(pool[e][:, :T]) for e in range(8)]
        assert np.array_equal(oracle.reduce_threads(xs[0], threads), oracle.reduce(xs[0]))
        n, t0 = 0, time.perf_counter()
        while True:
            oracle.reduce_threads(xs[n % len(xs)], threads)
            n += 1
            el = time.perf_counter() - t0
            if el > budget_s / len(tokens):
                break
        per_t[T] = el / n * 1e6
    return sum(per_t.values()) / len(per_t), per_t


def host_cpu() -> str:
    """Model name of the host CPU and the cores this process may use."""
    model = "unknown CPU"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        avail = os.cpu_count() or 0
    return f"{model}, {avail} cores available"


def time_steps(s, T, steps, stream):
    """HIP-event time of `steps` replays of the step graph for T tokens (ms)."""
    import torch

    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record(stream)
    for _ in range(steps):
        s.step(T, stream)
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b)


def chain_point(w, T, args, *, T_max=None, pool_entries=None, inject=False, waves_per_group=1,
                check_nodes=(0, -1), forced=0):
    """Measure one captured chain configuration. Returns a JSON-ready dict."""
    import numpy as np
    import torch

    import oracle
    import paper_2607_08973_amd as S
    import synth
    from oracle import sim

    dev = "cuda:0"
    N, H, L = w.nranks, w.hidden, w.reduces_per_step
    T_max = T_max or T
    P = pool_entries or w.pool_entries()
    stream = torch.cuda.current_stream()
    try:
        s = S.Sifar(nranks=N, hidden=H, max_tokens=T_max, reduces_per_step=L,
                    validate=args.mode, log_epochs=L, fuse_peers=args.fuse,
                    epilogue=int(w.epilogue), rms_eps=w.rms_eps,
                    waves_per_group=waves_per_group, persistent=args.persistent,
                    buffers=args.buffers, forced_retries=forced)
    except S.SifarError as err:
        if args.persistent and err.code == S.SIFAR_EINVAL:
            return {"workload": w.name, "nranks": N, "tokens": T, "hidden": H, "chain": L,
                    "skipped": "persistent step needs more co-resident waves than the GPU holds"}
        raise
    pool = synth.payload_pool(w.wid, N, T_max, H, P, w.dist)
    pool_d = torch.from_numpy(pool.view(np.int16)).to(dev)
    if w.epilogue:
        res0 = synth.residual_init(w.wid, T_max, H)
        wgt = synth.rms_weight(w.wid, H)
        res_d = torch.from_numpy(res0.view(np.int16)).to(dev)
        w_d = torch.from_numpy(wgt.view(np.int16)).to(dev)
        ring = torch.zeros((L, T_max, H), dtype=torch.int16, device=dev)
        s.bind_step(pool_d, residual=res_d, weight=w_d, y_ring=ring)
    else:
        ring = torch.zeros((L, T_max, H), dtype=torch.int16, device=dev)
        s.bind_step(pool_d, out_ring=ring)
    late = None
    if inject and w.stale_prob > 0:
        E = L * (args.warmup + args.steps + 1)
        late = synth.delay_table(w.wid, N, E, w.stale_prob)
        s.set_injection([int(x) for x in late])
    for _ in range(args.warmup):
        s.step(T, stream)
    torch.cuda.synchronize()
    s.check()
    ms = time_steps(s, T, args.steps, stream)
    s.check()
    nxt, _ = s.epochs()
    epochs = list(range(nxt - L, nxt))
    out = {"workload": w.name, "nranks": N, "tokens": T, "hidden": H, "chain": L,
           "steps": args.steps, "us_per_reduce": ms * 1e3 / (args.steps * L)}
    fused_launch = args.fuse and args.buffers == 2
    launches = 1 if args.persistent else (L + 2 if fused_launch else 2 * L + 1)
    out["launch_period_us"] = ms * 1e3 / (args.steps * launches)
    red = reduce_bytes(N, T, H) + (epilogue_bytes(T, H) if w.epilogue else 0)
    out["reduce_bytes"] = red
    out["reduce_gbs"] = red / (out["us_per_reduce"] * 1e-6) / 1e9
    peers = produce_bytes(N, T, H) if (fused_launch or args.persistent) else 0
    per_launch = L if args.persistent else 1
    out["launch_bytes"] = red * per_launch
    out["launch_gbs"] = red * per_launch / (out["launch_period_us"] * 1e-6) / 1e9
    out["peer_copy_bytes_per_launch"] = peers * per_launch
    # parity check of the last replay (outside the timed region)
    got = ring.cpu().numpy().view(np.uint16)
    if not w.epilogue:
        for i in check_nodes:
            g = epochs[i]
            exp = oracle.reduce(pool[(g - 1) % P][:, :T])
            assert np.array_equal(got[i, :T], exp), f"{w.name} T={T} node {i}"
    else:
        # one more step, untimed, from a known residual: the residual after it
        # bit-exact, every node's y within 1 bf16 step
        res_before = res_d.cpu().numpy().view(np.uint16)[:T].copy()
        s.step(T, stream)
        torch.cuda.synchronize()
        s.check()
        nxt, _ = s.epochs()
        epochs = list(range(nxt - L, nxt))
        _, r_list, y_list = oracle.reduce_chain(pool, epochs, T,
                                                epilogue=(res_before, wgt, w.rms_eps))
        assert np.array_equal(res_d.cpu().numpy().view(np.uint16)[:T], r_list[-1]), \
            f"{w.name} T={T}: residual"
        y_got = ring[:, :T].cpu().numpy().view(np.uint16)
        key = lambda x: np.where(x.astype(np.int32) & 0x8000, -(x.astype(np.int32) & 0x7FFF),
                                 x.astype(np.int32))
        off = 0
        for i in range(L):
            d = np.abs(key(y_got[i]) - key(y_list[i]))
            assert d.max() <= 1, f"{w.name} T={T} node {i}: y off by {d.max()}"
            off += int(np.count_nonzero(d))
        out["y_elements_one_step_off"] = off
        out["y_elements_checked"] = L * T * H
    log = s.read_log()
    segs = (H + 511) // 512
    rows = np.array([log[(g - 1) % L, :T * segs] for g in epochs])
    att = rows & 0xFFFF
    out["chunks_retried_frac"] = float(np.mean(att > 1))
    out["mean_attempts"] = float(np.mean(att))
    assert np.all((rows >> 24) == 0), "a chunk was accepted with a stale stamp"
    if late is not None:
        masks = [int(late[(g - 1) % len(late)]) for g in epochs]
        out["epochs_with_late_stamp_frac"] = float(np.mean([m != 0 for m in masks]))
        if not args.persistent:
            # launches in stream order: every decision is predictable exactly
            pred = sim.predict_log(N, masks, args.mode, forced)
            assert all(np.all(rows[i] == pred[i]) for i in range(L)), "decision log != prediction"
            out["log_matches_prediction"] = True
    s.close()
    return out


def kernel_table(per_t, tokens, N, H, L, persistent, fused_launch):
    """Per batch size: the dominant kernel's launch period (from the HIP-event
    microseconds per all-reduce of a step), one consumer's algorithmic bytes
    per launch and the emulated peers' copy bytes per launch."""
    if persistent:
        launches, per_launch = 1, L
    else:
        launches, per_launch = (L + 2 if fused_launch else 2 * L + 1), 1
    kern = {}
    for T in tokens:
        period_us = per_t[T] * L / launches
        byts = per_launch * reduce_bytes(N, T, H)
        peers = per_launch * produce_bytes(N, T, H) if (fused_launch or persistent) else 0
        kern[T] = {"launch_period_us": period_us, "bytes_per_launch": byts,
                   "gbs": byts / (period_us * 1e-6) / 1e9,
                   "peer_copy_bytes_per_launch": peers}
    return kern


def spec_graph_point(w, pool, pool_d, args):
    """The paper's speculative reduction on the headline workload: one
    captured graph per decode step with one launch per all-reduce (the peers
    of epoch g + 1 written by a second plane of the launch that reduces g),
    payload and stamps loaded together, validated afterwards. Timed like the
    headline (HIP events around the graph replays); its dominant kernel is the
    fused reduction, L - 1 of a step's L + 2 launches. The last replay's
    outputs are checked against the oracle."""
    import numpy as np
    import torch

    import oracle
    import paper_2607_08973_amd as S

    N, H, L, tokens = w.nranks, w.hidden, w.reduces_per_step, w.tokens
    T_max = max(tokens)
    ring = torch.zeros((L, T_max, H), dtype=torch.int16, device="cuda:0")
    stream = torch.cuda.current_stream()
    s = S.Sifar(nranks=N, hidden=H, max_tokens=T_max, reduces_per_step=L, validate="spec",
                log_epochs=L, fuse_peers=1, persistent=0)
    s.bind_step(pool_d, out_ring=ring)
    per_t = {}
    for T in tokens:
        for _ in range(args.warmup):
            s.step(T, stream)
        per_t[T] = time_steps(s, T, args.steps, stream) * 1e3 / (args.steps * L)
        s.check()
        nxt, _ = s.epochs()
        got = ring.cpu().numpy().view(np.uint16)
        for i in (0, L // 2, L - 1):
            g = nxt - L + i
            assert np.array_equal(got[i, :T], oracle.reduce(pool[(g - 1) % pool.shape[0]][:, :T])), \
                f"spec graph T={T} node {i}"
    s.close()
    kern = kernel_table(per_t, tokens, N, H, L, False, True)
    period = sum(k["launch_period_us"] for k in kern.values()) / len(kern)
    byts = sum(k["bytes_per_launch"] for k in kern.values()) / len(kern)
    gbs = byts / (period * 1e-6) / 1e9
    return {"protocol": "SPEC: payload and stamps loaded together, validated after, retried "
                        "on a stale stamp; one graph launch per all-reduce",
            "us_per_reduce": round(sum(per_t.values()) / len(per_t), 4),
            "us_per_reduce_by_tokens": {str(k): round(v, 4) for k, v in per_t.items()},
            "dominant_kernel": "reduce_kernel<8, SPEC, no epilogue, fused peers>",
            "launch_period_us": round(period, 4), "bytes_per_launch": round(byts),
            "achieved_gbs": round(gbs, 3), "frac": round(gbs / HBM_PEAK_GBS, 6),
            "traffic": measured_traffic("fused")}


def reduce_point(w, args, scrub, reps=30):
    """One eager all-reduce (the plain reduction kernel, no peers in its
    launch), `reps` rounds warm (reduce right after its producer) and `reps`
    rounds cold (a 512 MiB write between producer and reduce pushes the slots
    out of L2 and the Infinity Cache). Event times here are per round (the
    producer and the scrub included); the reduction kernel's own duration in
    each condition comes from a kernel trace of this workload (in a trace, a
    cold reduce is the one dispatched right after the scrub's fill kernel)."""
    import numpy as np
    import torch

    import oracle
    import paper_2607_08973_amd as S
    import synth

    N, T, H = w.nranks, w.tokens[0], w.hidden
    P = 3
    pool = synth.payload_pool(w.wid, N, T, H, P, w.dist)
    src = torch.from_numpy(pool.view(np.int16)).to("cuda:0")
    out = torch.zeros((T, H), dtype=torch.int16, device="cuda:0")
    res = {"workload": "reduce-" + w.name, "nranks": N, "tokens": T, "hidden": H,
           "reduce_bytes": reduce_bytes(N, T, H), "reps": reps, "waves_per_group": args.wpg}
    with S.Sifar(nranks=N, hidden=H, max_tokens=T, reduces_per_step=2, validate=args.mode,
                 log_epochs=8, waves_per_group=args.wpg) as s:
        s.produce(src[0], T)
        s.reduce(out, T)
        for kind in ("warm", "cold"):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record()
            for k in range(reps):
                s.produce(src[k % P], T)
                if kind == "cold":
                    scrub.fill_(k & 0x7F)
                s.reduce(out, T)
            b.record()
            torch.cuda.synchronize()
            res[f"{kind}_round_us"] = a.elapsed_time(b) * 1e3 / reps
        s.check()
        assert np.array_equal(out.cpu().numpy().view(np.uint16),
                              oracle.reduce(pool[(reps - 1) % P])), f"{w.name}: output != oracle"
    return res


def torch_sum_reference(w, scrub, reps=30):
    """PyTorch's own reduction over the rank dimension (x.sum(0) on bf16 with
    fp32 accumulation: the same N reads and one write) at one sweep shape,
    warm and cold like reduce_point, for the kernel trace to compare with."""
    import numpy as np
    import torch

    import synth

    N, T, H = w.nranks, w.tokens[0], w.hidden
    pool = synth.payload_pool(w.wid, N, T, H, 3, w.dist)
    src = torch.from_numpy(pool.view(np.int16)).to("cuda:0").view(torch.bfloat16)
    x = torch.empty((N, T * H), dtype=torch.bfloat16, device="cuda:0")
    res = {"workload": "torch-sum-" + w.name, "nranks": N, "tokens": T, "hidden": H,
           "reduce_bytes": reduce_bytes(N, T, H), "reps": reps}
    x.copy_(src[0].reshape(N, T * H))
    y = x.sum(0)  # first call outside the timed rounds
    for kind in ("warm", "cold"):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for k in range(reps):
            x.copy_(src[k % 3].reshape(N, T * H))
            if kind == "cold":
                scrub.fill_(k & 0x7F)
            y = x.sum(0)
        b.record()
        torch.cuda.synchronize()
        res[f"{kind}_round_us"] = a.elapsed_time(b) * 1e3 / reps
    del y
    return res


def suite(args):
    """Secondary workloads: one JSON line each (not the headline metric)."""
    import synth

    if args.workload == "reduce-cold":
        import torch
        scrub = torch.empty(512 << 20, dtype=torch.uint8, device="cuda:0")
        pts = [reduce_point(w, args, scrub) for w in synth.PAYLOAD_SWEEP]
        pts.append(torch_sum_reference(synth.PAYLOAD_SWEEP[-1], scrub))
        for p in pts:
            print(json.dumps({k: (round(v, 4) if isinstance(v, float) else v)
                              for k, v in p.items()}), flush=True)
        return
    if args.workload == "litmus":
        # the handoff litmus (sifar_litmus): both reader orders, producer and
        # consumer on different XCDs or on one, 8 to 512 concurrent pairs
        import paper_2607_08973_amd as S
        trials = 65536
        for proto, pname in ((S.SIFAR_LITMUS_ORDERED, "ordered"),
                             (S.SIFAR_LITMUS_ORDERED_PREFETCH, "ordered-prefetching-producer"),
                             (S.SIFAR_LITMUS_READ_FIRST, "read-first")):
            for place, lname in ((S.SIFAR_LITMUS_CROSS_XCD, "cross-xcd"),
                                 (S.SIFAR_LITMUS_SAME_XCD, "same-xcd")):
                for pairs in (8, 64, 256, 512):
                    r = S.sifar_litmus(proto, place, pairs, trials)
                    print(json.dumps({
                        "workload": "litmus", "reader": pname, "placement": lname,
                        "pairs": pairs, "trials": r["trials"], "violations": r["violations"],
                        "violation_rate": r["violations"] / max(r["trials"], 1),
                        "violations_first_epochs": r["violations_first_epochs"],
                        "pairs_placed": r["pairs_placed"], "timeouts": r["timeouts"],
                        "ns_per_trial": round(r["ns_per_trial"], 1),
                        "first_violation": r["first_bad"]}), flush=True)
        return
    if args.workload == "smoke-n2":
        pts = [chain_point(synth.SMOKE_N2, 1, args)]
    elif args.workload == "spec-stress":
        pts = [chain_point(synth.SPEC_STRESS, 4, args, inject=True),
               chain_point(synth.SPEC_STRESS, 4, args, inject=False)]
    elif args.workload == "sweep":
        pts = [chain_point(w, w.tokens[0], args, pool_entries=5) for w in synth.PAYLOAD_SWEEP]
    elif args.workload == "ablation":
        # the paper's incremental optimisations (Sec. 6.3) as they exist here:
        # one buffer (bottom barrier) -> dual buffering; ORDERED (top barrier by
        # flag polling) -> SPEC (speculative); NONE = the "no barrier" ideal.
        # Persistent steps run ORDERED only (they validate before they load).
        import copy
        w = synth.LLAMA8B_DECODE
        pts = []
        combos = [(p_, b, m) for p_ in (0, 1) for b in (1, 2) for m in ("ordered", "spec", "none")
                  if not (p_ and m != "ordered")]
        for p_, b, m in combos:
            a2 = copy.copy(args)
            a2.persistent, a2.buffers, a2.mode = p_, b, m
            for T in w.tokens:
                pt = chain_point(w, T, a2, T_max=max(w.tokens))
                pt.update(persistent=p_, buffers=b, validate=m)
                pts.append(pt)
        for p in pts:
            print(json.dumps({k: (round(v, 4) if isinstance(v, float) else v)
                              for k, v in p.items()}), flush=True)
        return
    elif args.workload == "retry-curve":
        # forced retries (Sec. 6.3, "Retry Overhead") and late-stamp rates
        import copy
        w = synth.SPEC_STRESS
        pts = []
        for k in (0, 1, 2, 3, 4):
            a2 = copy.copy(args)
            a2.forced = k
            pt = chain_point(w, 4, a2, forced=k)
            pt.update(forced_retries=k)
            pts.append(pt)
        for prob in (0.0, 0.02, 0.05, 0.1, 0.2, 0.5):
            wp = dataclasses.replace(w, stale_prob=prob)
            pt = chain_point(wp, 4, args, inject=prob > 0)
            pt.update(stale_prob=prob)
            pts.append(pt)
    elif args.workload == "misspec-vs-tp":
        # how often a chunk's first stamp poll finds a rank not yet published,
        # by TP degree, with no injection (the paper's mis-speculation rate
        # grows with TP, Sec. 6.3): in a persistent step the emulated peers
        # run concurrently with the reduction, so this is their natural lag
        w0 = synth.LLAMA8B_DECODE
        pts = []
        for N in (2, 4, 8):
            w = dataclasses.replace(w0, nranks=N, name=f"llama8b-decode-n{N}-h4096-chain64")
            for T in w.tokens:
                pts.append(chain_point(w, T, args, T_max=max(w.tokens)))
    elif args.workload == "moe-rmsnorm":
        w = synth.MOE_DECODE
        pts = []
        for T in w.tokens:
            for G in (1, 4, 16):
                p = chain_point(w, T, args, T_max=max(w.tokens), inject=True, waves_per_group=G)
                p["waves_per_group"] = G
                pts.append(p)
    else:
        raise SystemExit(f"unknown workload {args.workload}")
    for p in pts:
        if "skipped" in p:
            print(json.dumps(p), flush=True)
            continue
        p["validate"] = args.mode
        p["fuse_peers"] = args.fuse
        p["persistent"] = args.persistent
        print(json.dumps({k: (round(v, 4) if isinstance(v, float) else v) for k, v in p.items()}),
              flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the library emulates the N ranks on a single "
              f"MI355X and has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)
    if args.workload != "llama8b-decode":
        import torch

        assert torch.cuda.is_available(), "bench.py needs a GPU"
        suite(args)
        return

    import numpy as np
    import torch

    import paper_2607_08973_amd as S
    import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = "cuda:0"
    torch.cuda.set_device(0)
    w = synth.LLAMA8B_DECODE
    N, H, L, tokens = w.nranks, w.hidden, w.reduces_per_step, w.tokens
    T_max = max(tokens)
    pool = synth.payload_pool(w.wid, N, T_max, H, w.pool_entries(), w.dist)
    pool_d = torch.from_numpy(pool.view(np.int16)).to(dev)
    ring = torch.zeros((L, T_max, H), dtype=torch.int16, device=dev)
    s = S.Sifar(nranks=N, hidden=H, max_tokens=T_max, reduces_per_step=L, validate=args.mode,
                log_epochs=L, fuse_peers=args.fuse, persistent=args.persistent,
                buffers=args.buffers)
    s.bind_step(pool_d, out_ring=ring)
    stream = torch.cuda.current_stream()

    def step():
        for T in tokens:
            s.step(T, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    s.check()

    # ---- timed region: K decode steps --------------------------------------
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_total = ev0.elapsed_time(ev1)
    s.check()
    reduces = args.steps * len(tokens) * L
    us_per_reduce = ms_total * 1e3 / reduces

    # per batch size, same method
    per_t = {}
    for T in tokens:
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(args.steps):
            s.step(T, stream)
        b.record(stream)
        torch.cuda.synchronize()
        per_t[T] = a.elapsed_time(b) * 1e3 / (args.steps * L)
    s.check()

    # ---- the metric's larger batch sizes, outside the timed region ---------
    # The metric spans 1-64 tokens; the workload's batch sizes stop at 8. The
    # same chain (64 all-reduces, N = 8, H = 4096, the same value recipe) at
    # 16 and 64 tokens, each on a handle of its own, parity spot-checked by
    # chain_point. Their pools hold 5 entries (coprime with the chain length),
    # as in the payload sweep: at 64 tokens the workload's 3L + 1 entries
    # would take 809 MB, and the peers' sources would come from HBM instead of
    # the Infinity Cache that holds the 8-token pool (101 MB).
    wide = {}
    for T in ((16, 64) if args.wide_points else ()):
        pt = chain_point(w, T, args, T_max=T, pool_entries=5, check_nodes=(0, L // 2, -1))
        wide[str(T)] = round(pt["us_per_reduce"], 4) if "us_per_reduce" in pt else pt["skipped"]

    # ---- dispatch floor: a captured graph of tiny kernels ------------------
    floor_us = graph_floor_us(args.floor_nodes)
    floors = latency_floors()

    # ---- roofline of the dominant kernel -----------------------------------
    # Persistent: one launch per step, L all-reduces in it. Per launch: with
    # fused peers a step is produce(g1), L-1 launches of the fused
    # reduce(g_i)+produce(g_i+1) kernel, reduce(g_L) and the epoch advance:
    # the fused kernel is L-1 of the L+2 launches; its average launch period
    # is the HIP-event step time over the launches of the step.
    # Algorithmic bytes are one consumer's share of each all-reduce (read
    # N*K, write K, read the stamps); the emulated peers' copies (read N*K,
    # write N*K, write the stamps) are reported apart.
    kern = kernel_table(per_t, tokens, N, H, L, args.persistent, args.fuse and args.buffers == 2)
    mean_period = sum(k["launch_period_us"] for k in kern.values()) / len(kern)
    mean_bytes = sum(k["bytes_per_launch"] for k in kern.values()) / len(kern)
    mean_peer = sum(k["peer_copy_bytes_per_launch"] for k in kern.values()) / len(kern)
    achieved = mean_bytes / (mean_period * 1e-6) / 1e9

    # ---- the same steps cold: a 512 MiB write before each step ------------
    # pushes the pool, the slots and the outputs out of the L2s and the
    # Infinity Cache; HIP events bracket the step alone.
    scrub = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    cold_t = {}
    for T in tokens:
        reps, tot = 10, 0.0
        for k in range(reps):
            scrub.fill_(k & 0x7F)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            s.step(T, stream)
            b.record(stream)
            torch.cuda.synchronize()
            tot += a.elapsed_time(b) * 1e3
        cold_t[T] = tot / (reps * L)
    s.check()
    kern_cold = kernel_table(cold_t, tokens, N, H, L, args.persistent,
                             args.fuse and args.buffers == 2)
    cold_period = sum(k["launch_period_us"] for k in kern_cold.values()) / len(kern_cold)
    achieved_cold = mean_bytes / (cold_period * 1e-6) / 1e9
    del scrub
    graph_next_epoch, _ = s.epochs()   # the ring now holds the last step at T = tokens[-1]
    graph_ring = ring.cpu().numpy().view(np.uint16).copy()

    # ---- the speculative per-launch chain (the paper's SPEC) --------------
    spec = None
    if args.persistent and args.spec_graph:
        spec = spec_graph_point(w, pool, pool_d, args)

    # ---- parity spot check of the timed graph (outside the timed region) --
    import oracle
    T = tokens[-1]
    for i in (0, L // 2, L - 1):
        g = graph_next_epoch - L + i
        exp = oracle.reduce(pool[(g - 1) % pool.shape[0]][:, :T])
        assert np.array_equal(graph_ring[i, :T], exp), f"graph parity node {i}"

    # ---- calibration copy for hardware byte counters ----------------------
    # A plain device-to-device copy of exactly 64 MiB: profilers' FETCH_SIZE and
    # WRITE_SIZE for it give the scale factor between counter units and bytes.
    calib = torch.empty(64 << 20, dtype=torch.uint8, device=dev)
    calib_dst = torch.empty_like(calib)
    calib_dst.copy_(calib)
    torch.cuda.synchronize()
    del calib, calib_dst

    traffic = None
    if args.mode == "ordered" and args.buffers == 2 and args.persistent:
        traffic = measured_traffic("persistent")
    elif args.mode == "spec" and args.buffers == 2 and args.fuse:
        traffic = measured_traffic("fused")

    cpu = None
    if args.cpu_seconds > 0:
        cpu_us, cpu_t = cpu_baseline(pool, tokens, args.cpu_seconds)
        cpu = {"value": round(cpu_us, 3), "unit": "us per all-reduce", "cores": 1,
               "kind": "oracle",
               "sample": f"C oracle, 1 thread ({host_cpu()}), the same N=8 x H=4096 pool "
                         f"entries at batch {list(tokens)} for {args.cpu_seconds:.0f} s total; mean "
                         f"over batch sizes of per-reduce time: " +
                         ", ".join(f"T={t}: {v:.1f} us" for t, v in cpu_t.items())}
        try:
            avail = len(os.sched_getaffinity(0))
        except (AttributeError, OSError):
            avail = os.cpu_count() or 1
        threads = max(1, avail)
        par_us, par_t = cpu_baseline_parallel(pool, tokens, args.cpu_seconds / 3, threads)
        cpu["parallel"] = {
            "value": round(par_us, 3), "unit": "us per all-reduce", "cores": threads,
            "sample": f"the same oracle reduction on {threads} native threads (every core this "
                      f"process may use), each a contiguous slice of the T x H elements, "
                      f"{args.cpu_seconds / 3:.0f} s total: " +
                      ", ".join(f"T={t}: {v:.1f} us" for t, v in par_t.items())}

    s.close()
    rec = {
        "metric": "us per all-reduce (N=8, 1-64 tokens x 4096 bf16) + achieved HBM GB/s fraction",
        "value": round(us_per_reduce, 4),
        "unit": "us/all-reduce",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_total / args.steps, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 (fp32 accumulate)",
        "data": "synthetic (seeded N(0,1)*0.5 activations, 0.1% outliers x50)",
        "config": {"workload": w.name, "nranks": N, "hidden": H, "tokens": list(tokens),
                   "reduces_per_step": L, "validate": args.mode, "fuse_peers": args.fuse,
                   "protocol": ("ORDERED: stamps polled before the payload is loaded (no "
                                "speculation), peers concurrent in one persistent launch"
                                if args.persistent else
                                f"{args.mode.upper()} in one launch per all-reduce"),
                   "persistent": args.persistent, "buffers": args.buffers,
                   "step": (f"{len(tokens)} decode steps of {L} all-reduces, one persistent "
                            f"launch each" if args.persistent else
                            f"{len(tokens)} captured decode-step graphs of {L} all-reduces")},
        "reduces_per_s": round(1e6 / us_per_reduce, 1),
        "us_per_reduce_by_tokens": {str(k): round(v, 4) for k, v in per_t.items()},
        "us_per_reduce_at_16_and_64_tokens": wide,
        "dominant_kernel": {str(k): {kk: (round(vv, 4) if isinstance(vv, float) else vv)
                                     for kk, vv in v.items()} for k, v in kern.items()},
        "graph_dispatch_floor_us": round(floor_us, 4),
        "floors": floors,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 3), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 6),
                     "traffic": traffic, "traffic_scope": "hardware byte counters of the whole "
                                                          "launch, the peers' copies included",
                     "bytes_per_launch": round(mean_bytes),
                     "bytes": "one consumer's share per all-reduce: read N*K, write K, "
                              "4*N bytes of stamps per 512-element chunk; times the "
                              "all-reduces per launch",
                     "residency": "warm: each epoch's slots were just written by the same "
                                  "step's producer waves",
                     "launch_period_us": round(mean_period, 4),
                     "frac_cold": round(achieved_cold / HBM_PEAK_GBS, 6),
                     "launch_period_cold_us": round(cold_period, 4),
                     "cold": "the same steps, each right after a 512 MiB write that pushes "
                             "the source pool, slots and outputs out of the L2s and the "
                             "Infinity Cache; HIP events around the step alone",
                     "peer_copy_bytes_per_launch": round(mean_peer),
                     "peer_copy_gbs": round(mean_peer / (mean_period * 1e-6) / 1e9, 3)},
        "spec_graph": spec,
        "cpu_baseline": cpu,
        "wall_s_timed": round(wall, 3),
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
