"""GPU parity: the HIP path, called through the C ABI, against the CPU oracle.

Bar: every all-reduce output and every residual-stream value bit-exact; the
RMSNorm output y within 1 bf16 step (the only value behind a reordered
reduction, the sum of squares over the hidden dimension); every decision-log
word bit-exact against the protocol simulator's prediction.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2607_08973_amd as S
import synth
from oracle import ref_np, sim

pytestmark = pytest.mark.gpu

from sifar_harness import (DEV, StepRun, expected_log_words, inject_table, read_stamp_log,
                           replay_logs, to_dev, to_host, ulp_distance)

ORDERS = {"spec": "spec", "ordered": "ordered"}


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    S.load()  # loud failure if the library is missing
    yield
    torch.cuda.synchronize()


def _eager_chain(N, T, H, epochs, mode, ahead=False, seed=0, dist="normal"):
    pool = synth.payload_pool(100 + seed, N, T, H, epochs, dist)
    src = to_dev(pool)
    outs = torch.zeros((epochs, T, H), dtype=torch.int16, device=DEV)
    with S.Sifar(nranks=N, hidden=H, max_tokens=T, reduces_per_step=2, validate=mode,
                 log_epochs=epochs) as s:
        if ahead:
            # the producer runs one epoch ahead: produce g+1 before reducing g
            s.produce(src[0], T)
            for g in range(1, epochs + 1):
                if g < epochs:
                    s.produce(src[g], T)
                s.reduce(outs[g - 1], T)
        else:
            for g in range(1, epochs + 1):
                s.produce(src[g - 1], T)
                s.reduce(outs[g - 1], T)
        s.check()
        log = s.read_log()
    got = to_host(outs)
    for g in range(epochs):
        exp = oracle.reduce(pool[g])
        assert np.array_equal(got[g], exp), f"epoch {g + 1}"
    return log


@pytest.mark.parametrize("mode", ["spec", "ordered", "none"])
@pytest.mark.parametrize("ahead", [False, True])
def test_eager_n2_chain64(mode, ahead):
    """Two ranks, one token of 4096, 64 sequential all-reduces on dual buffers."""
    log = _eager_chain(2, 1, 4096, 64, mode, ahead)
    assert np.all(log[:, :8] == sim.pack_log(1, 0, 0))


@pytest.mark.parametrize("N", [1, 2, 3, 5, 8])
@pytest.mark.parametrize("T,H", [(3, 4104), (1, 8), (2, 520), (5, 1000)])
def test_eager_ragged_shapes(N, T, H):
    """Several chunks and a ragged last chunk per row; hidden sizes that are not
    multiples of the 512-element chunk."""
    _eager_chain(N, T, H, 4, "spec", seed=N * 1000 + H)


def test_graph_step_n2_chain64():
    w = synth.SMOKE_N2
    run = StepRun(w, 1)
    epochs = run.step(1)
    run.s.check()
    got = to_host(run.out_d)
    exp = oracle.reduce_chain(run.pool, epochs, 1)
    for i in range(w.reduces_per_step):
        assert np.array_equal(got[i, :1], exp[i]), f"node {i}"
    run.s.close()


@pytest.mark.parametrize("fuse", [1, 0])
@pytest.mark.parametrize("mode", ["spec", "ordered", "none"])
def test_graph_llama_decode_steps(mode, fuse):
    """N=8, batch 1/2/4/8 x 4096, 64 chained all-reduces per decode step."""
    w = synth.LLAMA8B_DECODE
    run = StepRun(w, 8, validate=mode, fuse_peers=fuse)
    for T in w.tokens:
        for rep in range(2):
            epochs = run.step(T)
            run.s.check()
            got = to_host(run.out_d)
            exp = oracle.reduce_chain(run.pool, epochs, T)
            for i in range(w.reduces_per_step):
                assert np.array_equal(got[i, :T], exp[i]), f"T={T} rep={rep} node={i}"
            log = run.s.read_log()
            assert np.all(log[:, :T * 8] == sim.pack_log(1, 0, 0))
    run.s.close()


def test_graph_llama_full_run_sampled():
    """The benchmark's configuration: 100 decode steps per batch size, every
    step replayed from the captured graph; outputs sampled every 9th step."""
    w = synth.LLAMA8B_DECODE
    run = StepRun(w, 8)
    for T in w.tokens:
        for step in range(w.steps):
            epochs = run.step(T)
            if step % 9 == 0 or step == w.steps - 1:
                got = to_host(run.out_d)
                for i in range(0, w.reduces_per_step, 7):
                    g = epochs[i]
                    exp = oracle.reduce(run.pool[(g - 1) % run.pool.shape[0]][:, :T])
                    assert np.array_equal(got[i, :T], exp), f"T={T} step={step} node={i}"
        run.s.check()
    run.s.close()


@pytest.mark.parametrize("fuse", [1, 0])
@pytest.mark.parametrize("order", ["spec", "ordered"])
@pytest.mark.parametrize("forced", [0, 2])
def test_stale_injection_deterministic(order, forced, fuse):
    """Speculation stress: each rank's stamp is late with p = 0.1 per epoch;
    outputs equal the no-speculation oracle and every decision-log word equals
    the simulator's prediction."""
    w = synth.SPEC_STRESS
    steps = 12 if forced == 0 else 4
    late = synth.delay_table(w.wid, w.nranks, w.reduces_per_step * steps, w.stale_prob)
    run = StepRun(w, 4, validate=order, forced_retries=forced, fuse_peers=fuse)
    run.s.set_injection(inject_table(late))
    T = 4
    segs = 8
    for step in range(steps):
        epochs = run.step(T)
        got = to_host(run.out_d)
        exp = oracle.reduce_chain(run.pool, epochs, T)
        for i in range(w.reduces_per_step):
            assert np.array_equal(got[i, :T], exp[i]), f"step={step} node={i}"
        log = run.s.read_log()
        masks = [int(late[(g - 1) % len(late)]) for g in epochs]
        pred = expected_log_words(w.nranks, masks, order, forced)
        for i, g in enumerate(epochs):
            row = log[(g - 1) % log.shape[0], :T * segs]
            assert np.all(row == pred[i]), (step, i, hex(int(row[0])), hex(pred[i]))
    assert int(np.count_nonzero(late)) > 0
    run.s.check()
    run.s.close()


def test_spec_stress_full_length():
    """The speculation stress workload at its stated length: N = 8, 4 tokens,
    64 all-reduces per step, 200 steps, each rank's stamp late with p = 0.1.
    Per-epoch launches with the peers fused into the reduction's launch, the
    paper's speculative reduction. A late rank's payload waits in the stage
    and its slot still holds its previous epoch when the reduction first loads
    it, so only a retry that reloads the payload gets the sum right. Every
    output of every step equals the no-speculation oracle, every decision-log
    word equals the simulator's prediction, and every logged mask is the one
    the logged raw stamps imply (on-time ranks fresh at the first validation,
    late ranks holding the slot's previous epoch)."""
    w = synth.SPEC_STRESS
    steps, T, segs = w.steps, 4, 8
    late = synth.delay_table(w.wid, w.nranks, w.reduces_per_step * steps, w.stale_prob)
    run = StepRun(w, T, validate="spec", fuse_peers=1)
    run.s.set_injection(inject_table(late))
    retried = 0
    for step in range(steps):
        if step % 50 == 0:
            print(f"spec stress step {step} of {steps}", flush=True)
        epochs = run.step(T)
        got = to_host(run.out_d)
        exp = oracle.reduce_chain(run.pool, epochs, T)
        for i in range(w.reduces_per_step):
            assert np.array_equal(got[i, :T], exp[i]), f"step={step} node={i}"
        log = run.s.read_log()
        masks = [int(late[(g - 1) % len(late)]) for g in epochs]
        pred = expected_log_words(w.nranks, masks, "spec", 0)
        for i, g in enumerate(epochs):
            row = log[(g - 1) % log.shape[0], :T * segs]
            assert np.all(row == pred[i]), (step, i, hex(int(row[0])), hex(pred[i]))
        st = read_stamp_log(run.s)
        _, r = replay_logs(log, st, epochs, T * segs)
        retried += r
        for i, g in enumerate(epochs):
            first = st[(g - 1) % st.shape[0], :T * segs, 0]
            for rank in range(w.nranks):
                if (masks[i] >> rank) & 1:
                    assert np.all((first[:, rank] == g - 2) | (first[:, rank] == 0)), (g, rank)
                else:
                    assert np.all(first[:, rank] == g), (g, rank)
    run.s.check()
    run.s.close()
    frac = retried / (steps * w.reduces_per_step * T * segs)
    print(f"spec stress: {retried} chunk validations retried ({frac:.3f} of all)")
    assert retried > 0


def test_withheld_stamp_exhausts_budget():
    N, T, H = 4, 2, 1024
    pool = synth.payload_pool(7, N, T, H, 3, "normal")
    src = to_dev(pool)
    out = torch.zeros((T, H), dtype=torch.int16, device=DEV)
    s = S.Sifar(nranks=N, hidden=H, max_tokens=T, reduces_per_step=2, max_attempts=8)
    s.set_injection(inject_table([0, 0], withheld=[0, 0b0100]))
    s.produce(src[0], T)
    s.reduce(out, T)
    assert s.status() == S.SIFAR_OK
    s.produce(src[1], T)       # epoch 2: rank 2's stamp never lands
    s.reduce(out, T)
    assert s.status() == S.SIFAR_EDEVICE
    kind, epoch, chunk, attempts = s.error_info()
    assert (kind, epoch, attempts) == (S.SIFAR_DEV_RETRY_BUDGET, 2, 8)
    with pytest.raises(S.SifarError):
        s.produce(src[2], T)   # poisoned
    s.close()


@pytest.mark.parametrize("validate", ["spec", "ordered"])
def test_forced_slot_overrun_is_caught(validate):
    """The hazard dual buffering exists to prevent (Sec. 4.1), forced from the
    host: epoch 3 is produced into epoch 1's slot before epoch 1 is reduced.
    The producer's check latches the WAW error, and the reduction of epoch 1,
    which now finds epoch 3's stamps, never validates: its output is not
    epoch 1's sum."""
    N, T, H = 2, 1, 1024
    pool = synth.payload_pool(9, N, T, H, 3, "normal")
    src = to_dev(pool)
    out = torch.zeros((T, H), dtype=torch.int16, device=DEV)
    s = S.Sifar(nranks=N, hidden=H, max_tokens=T, reduces_per_step=2, max_attempts=4,
                validate=validate, log_epochs=4)
    s.set_injection(None, S.SIFAR_INJECT_SLOT_OVERRUN)
    s.produce(src[0], T)
    s.produce(src[1], T)
    s.produce(src[2], T)       # rewrites epoch 1's slot
    s.reduce(out, T)           # epoch 1
    log = s.read_log()
    assert s.status() == S.SIFAR_EDEVICE
    kind, epoch, chunk, prev = s.error_info()
    assert (kind, epoch, prev) == (S.SIFAR_DEV_WAW, 3, 1)
    segs = (H + 511) // 512
    assert np.all(log[0, :segs] & 0xFFFF == 4)               # budget spent
    assert np.all((log[0, :segs] >> 24) == 0b11)             # both ranks stale at the end
    assert not np.array_equal(to_host(out), oracle.reduce(pool[0]))
    s.close()


def test_slot_overrun_mode_off_restores_the_limit():
    N, T, H = 2, 1, 512
    pool = synth.payload_pool(10, N, T, H, 3, "normal")
    src = to_dev(pool)
    with S.Sifar(nranks=N, hidden=H, max_tokens=T, reduces_per_step=2) as s:
        s.set_injection(None, S.SIFAR_INJECT_SLOT_OVERRUN)
        s.set_injection(None, S.SIFAR_INJECT_OFF)
        s.produce(src[0], T)
        s.produce(src[1], T)
        with pytest.raises(S.SifarError) as e:
            s.produce(src[2], T)
        assert e.value.code == S.SIFAR_ESTATE
        s.check()


def test_protocol_order_errors():
    N, T, H = 2, 1, 512
    pool = synth.payload_pool(8, N, T, H, 4, "normal")
    src = to_dev(pool)
    out = torch.zeros((T, H), dtype=torch.int16, device=DEV)
    with S.Sifar(nranks=N, hidden=H, max_tokens=T, reduces_per_step=2) as s:
        with pytest.raises(S.SifarError) as e:
            s.reduce(out, T)                # nothing produced
        assert e.value.code == S.SIFAR_ESTATE
        s.produce(src[0], T)
        s.produce(src[1], T)                # one ahead: allowed
        with pytest.raises(S.SifarError) as e:
            s.produce(src[2], T)            # would overwrite epoch 1's slot
        assert e.value.code == S.SIFAR_ESTATE
        with pytest.raises(S.SifarError) as e:
            s.reduce(out, 0)
        assert e.value.code == S.SIFAR_EINVAL
        s.reduce(out, T)
        s.reduce(out, T)
        with pytest.raises(S.SifarError) as e:
            s.step(T)                       # nothing bound
        assert e.value.code == S.SIFAR_ESTATE
        s.check()
        assert np.array_equal(to_host(out), oracle.reduce(pool[1]))


def test_eager_then_graph_epochs_continue():
    """Eager epochs, then graph steps: epochs stay unique, parities stay right."""
    w = synth.Workload(60, "mix", 4, (2,), 2048, 6, 1, "normal")
    run = StepRun(w, 2)
    extra = to_dev(synth.payload_pool(61, 4, 2, 2048, 3, "normal"))
    out = torch.zeros((2, 2048), dtype=torch.int16, device=DEV)
    for k in range(3):
        run.s.produce(extra[k], 2)
        run.s.reduce(out, 2)
    for rep in range(3):
        epochs = run.step(2)
        got = to_host(run.out_d)
        exp = oracle.reduce_chain(run.pool, epochs, 2)
        for i in range(6):
            assert np.array_equal(got[i, :2], exp[i])
        run.s.produce(extra[rep], 2)
        run.s.reduce(out, 2)
        assert np.array_equal(to_host(out), oracle.reduce(synth.payload_pool(61, 4, 2, 2048, 3, "normal")[rep]))
    run.s.check()
    run.s.close()


def test_pairs_on_gpu_against_oracle():
    """N=2, H=65536 (the largest row): every bf16 pattern of rank 0 against 256
    values of rank 1 per reduce, 4 reduces (a sampled slice of all 2^32 pairs,
    including subnormals, infinities, signed zeros, overflow and ties)."""
    H, T = 65536, 256
    a = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    g = np.random.default_rng(23)
    special = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x007F, 0x0080, 0x3F80, 0xBF80,
                        0x7F7F, 0xFF7F, 0x7F80, 0xFF80, 0x3B80, 0xBB80, 0x7B00, 0x7A80], np.uint16)
    bvals = np.concatenate([special, g.integers(0, 65536, 4 * T - special.size,
                                                 dtype=np.uint32).astype(np.uint16)])
    with S.Sifar(nranks=2, hidden=H, max_tokens=T, reduces_per_step=2, log_epochs=4) as s:
        out = torch.zeros((T, H), dtype=torch.int16, device=DEV)
        for k in range(4):
            x = np.empty((2, T, H), np.uint16)
            x[0] = a[None, :]
            x[1] = bvals[k * T:(k + 1) * T, None]
            s.produce(to_dev(x), T)
            s.reduce(out, T)
            got = to_host(out)
            exp = ref_np.reduce(x)
            fin = ~np.isnan(ref_np.widen(exp))
            assert np.array_equal(got[fin], exp[fin])
            assert np.all(np.isnan(ref_np.widen(got[~fin])))
        s.check()


SWEEP_POINTS = [(w.nranks, w.tokens[0], w.hidden) for w in synth.PAYLOAD_SWEEP]


@pytest.mark.parametrize("persistent", [0, 1])
@pytest.mark.parametrize("N,T,H", SWEEP_POINTS)
def test_payload_sweep_points(N, T, H, persistent):
    """Every point of the latency-to-bandwidth sweep (8 KiB to 4 MiB per rank),
    U(-1, 1) values, full outputs of a 4-reduce step, per-launch and
    persistent (where the persistent step fits the GPU)."""
    w = synth.Workload(4, f"sweep-n{N}-t{T}-h{H}", N, (T,), H, 4, 1, "uniform")
    print(f"sweep N={N} T={T} H={H} persistent={persistent}", flush=True)
    try:
        run = StepRun(w, T, pool=synth.payload_pool(4, N, T, H, 5, "uniform"),
                      persistent=persistent)
    except S.SifarError as e:
        if persistent and e.code == S.SIFAR_EINVAL:
            pytest.skip("the persistent step needs more co-resident waves than the GPU holds")
        raise
    epochs = run.step(T)
    got = to_host(run.out_d)
    for i in range(0, 4):
        g = epochs[i]
        assert np.array_equal(got[i], oracle.reduce(run.pool[(g - 1) % 5])), f"node {i}"
    run.s.check()
    run.s.close()


def test_persistent_largest_sweep_point_fits():
    """The sweep's largest persistent step (N=8, T=256, H=8192: 4096 chunks,
    8192 co-resident waves) must be accepted on an MI355X: the step kernel
    then runs in its lower-register form, the prefetching producer needing
    more registers than 8 waves per SIMD allow. Checks one step in full."""
    N, T, H = 8, 256, 8192
    props = torch.cuda.get_device_properties(0)
    if props.multi_processor_count < 256:
        pytest.skip("fewer compute units than an MI355X")
    w = synth.Workload(4, f"sweep-n{N}-t{T}-h{H}", N, (T,), H, 4, 1, "uniform")
    print(f"largest persistent sweep step N={N} T={T} H={H}", flush=True)
    run = StepRun(w, T, pool=synth.payload_pool(4, N, T, H, 5, "uniform"), persistent=1)
    epochs = run.step(T)
    got = to_host(run.out_d)
    for i in range(4):
        g = epochs[i]
        assert np.array_equal(got[i], oracle.reduce(run.pool[(g - 1) % 5])), f"node {i}"
    run.s.check()
    run.s.close()


def test_persistent_small_steps_on_a_full_size_handle():
    """A handle sized for the sweep's largest step (N=8, T_max=256, H=8192)
    cannot hold the prefetching one-wave kernel's waves at T_max, so its
    one-wave steps run the non-prefetching form. Steps of 1 and 8 tokens
    (16 and 128 chunks, one wave per chunk) on it, every output checked."""
    N, T_max, H = 8, 256, 8192
    props = torch.cuda.get_device_properties(0)
    if props.multi_processor_count < 256:
        pytest.skip("fewer compute units than an MI355X")
    w = synth.Workload(4, f"sweep-n{N}-t{T_max}-h{H}", N, (T_max,), H, 4, 1, "uniform")
    print(f"small persistent steps on a handle for N={N} T_max={T_max} H={H}", flush=True)
    run = StepRun(w, T_max, pool=synth.payload_pool(4, N, T_max, H, 5, "uniform"), persistent=1)
    for T in (1, 8):
        epochs = run.step(T)
        got = to_host(run.out_d)
        for i in range(4):
            g = epochs[i]
            assert np.array_equal(got[i, :T], oracle.reduce(run.pool[(g - 1) % 5][:, :T])), \
                f"T={T} node {i}"
        run.s.check()
    run.s.close()


@pytest.mark.parametrize("fuse", [1, 0])
@pytest.mark.parametrize("waves_per_group", [1, 4, 16])
@pytest.mark.parametrize("T", [1, 8, 32])
def test_epilogue_moe_chain(T, waves_per_group, fuse):
    """N=8, hidden 8192, 120 chained all-reduces, each followed by residual-add
    + RMSNorm, with 5 % late stamps: residual bit-exact at every node, y within
    1 bf16 step, decision log as predicted."""
    w = synth.MOE_DECODE
    steps = 2
    late = synth.delay_table(w.wid, w.nranks, w.reduces_per_step * steps, w.stale_prob)
    run = StepRun(w, 32, waves_per_group=waves_per_group, fuse_peers=fuse)
    run.s.set_injection(inject_table(late))
    res = run.res0[:T].copy()
    segs = 16
    worst = 0
    for step in range(steps):
        res_before = to_host(run.res_d)[:T].copy()
        assert np.array_equal(res_before, res)
        epochs = run.step(T)
        y_got = to_host(run.y_d)
        a_list, r_list, y_list = oracle.reduce_chain(run.pool, epochs, T,
                                                     epilogue=(res, run.weight, w.rms_eps))
        # the residual stream after the last node is on the device
        assert np.array_equal(to_host(run.res_d)[:T], r_list[-1])
        for i in range(w.reduces_per_step):
            d = ulp_distance(y_got[i, :T], y_list[i])
            worst = max(worst, int(d.max()))
            assert d.max() <= 1, f"step {step} node {i}: y off by {d.max()} steps"
        res = r_list[-1]
        log = run.s.read_log()
        masks = [int(late[(g - 1) % len(late)]) for g in epochs]
        pred = expected_log_words(w.nranks, masks, "spec")
        for i, g in enumerate(epochs):
            row = log[(g - 1) % log.shape[0], :T * segs]
            assert np.all(row == pred[i]), (step, i)
    run.s.check()
    run.s.close()
    print(f"epilogue T={T} G={waves_per_group}: max y distance {worst} step(s)")


@pytest.mark.parametrize("N,T,H,persistent,G", [
    (8, 3, 65536, 0, 2), (3, 2, 65528, 0, 2),    # per launch: 64 groups of 2 waves per token
    (8, 3, 32768, 1, 1), (3, 2, 32760, 1, 1),    # persistent: 64 one-wave groups per token
])
def test_epilogue_widest_rows(N, T, H, persistent, G):
    """Residual-add + RMSNorm at the widest rows each kind of step takes: the
    per-token sum of squares is exchanged between 64 workgroups, one word per
    lane of the polling wave, the most it holds; full and ragged last chunks;
    8 chained nodes, two steps."""
    w = synth.Workload(90 + N, f"epilogue-n{N}-h{H}", N, (T,), H, 8, 2, "act",
                       epilogue=True)
    # a 5-entry source pool: epochs reuse entries cyclically
    run = StepRun(w, T, persistent=persistent, waves_per_group=G,
                  pool=synth.payload_pool(w.wid, N, T, H, 5, w.dist))
    res = run.res0[:T].copy()
    for step in range(2):
        epochs = run.step(T)
        y_got = to_host(run.y_d)
        _, r_list, y_list = oracle.reduce_chain(run.pool, epochs, T,
                                                epilogue=(res, run.weight, w.rms_eps))
        assert np.array_equal(to_host(run.res_d)[:T], r_list[-1])
        for i in range(w.reduces_per_step):
            assert ulp_distance(y_got[i, :T], y_list[i]).max() <= 1, f"step {step} node {i}"
        res = r_list[-1]
    run.s.check()
    run.s.close()


@pytest.mark.parametrize("N,T,H", [(5, 64, 3896), (3, 130, 2040)])
def test_persistent_epilogue_grouped_ragged(N, T, H):
    """Persistent residual-add + RMSNorm steps from 512 chunks run in 4-wave
    workgroups: 3896 leaves a partial last chunk inside each token's last
    group; 130 tokens pad the grid to 136 (one XCD per token), so the padding
    tokens' workgroups only arrive on the counter. Two steps of 8 chained
    nodes: residual bit-exact, y within 1 bf16 step."""
    w = synth.Workload(97 + N, f"epilogue-grouped-n{N}-t{T}-h{H}", N, (T,), H, 8, 2, "act",
                       epilogue=True)
    run = StepRun(w, T, persistent=1, pool=synth.payload_pool(w.wid, N, T, H, 5, w.dist))
    res = run.res0[:T].copy()
    for step in range(2):
        print(f"epilogue grouped N={N} T={T} H={H} step {step}", flush=True)
        epochs = run.step(T)
        y_got = to_host(run.y_d)
        _, r_list, y_list = oracle.reduce_chain(run.pool, epochs, T,
                                                epilogue=(res, run.weight, w.rms_eps))
        assert np.array_equal(to_host(run.res_d)[:T], r_list[-1])
        for i in range(w.reduces_per_step):
            assert ulp_distance(y_got[i, :T], y_list[i]).max() <= 1, f"step {step} node {i}"
        res = r_list[-1]
    run.s.check()
    run.s.close()


@pytest.mark.parametrize("H,persistent,G", [(65536, 0, 1), (32776, 1, 1), (65536, 1, 4)])
def test_epilogue_rows_beyond_the_exchange_are_refused(H, persistent, G):
    """More than 64 groups per token (or, persistent, more than 64 chunks) would
    not fit the one-word-per-lane exchange: refused at init."""
    with pytest.raises(S.SifarError) as e:
        S.Sifar(nranks=8, hidden=H, max_tokens=2, reduces_per_step=2, epilogue=1,
                waves_per_group=G, persistent=persistent,
                validate="ordered" if persistent else "spec")
    assert e.value.code == S.SIFAR_EINVAL


def test_epilogue_residual_chain_every_node_eager():
    """Eager fused calls: the residual after every node, bit-exact."""
    N, T, H = 8, 3, 8192
    pool = synth.payload_pool(55, N, T, H, 5, "act")
    res0 = synth.residual_init(55, T, H)
    wgt = synth.rms_weight(55, H)
    res_d, w_d = to_dev(res0), to_dev(wgt)
    y = torch.zeros((T, H), dtype=torch.int16, device=DEV)
    res = res0.copy()
    with S.Sifar(nranks=N, hidden=H, max_tokens=T, reduces_per_step=2, epilogue=1,
                 waves_per_group=2) as s:
        src = to_dev(pool)
        for g in range(5):
            s.produce(src[g], T)
            s.reduce_rmsnorm(res_d, w_d, y, T)
            a = oracle.reduce(pool[g])
            res, yy = oracle.residual_rmsnorm(a, res, wgt, float(np.float32(1e-6)))
            assert np.array_equal(to_host(res_d), res)
            assert ulp_distance(to_host(y), yy).max() <= 1
        s.check()


# ---- persistent decode step: producers and reduction in one launch ----------

def test_persistent_llama_decode_steps():
    """One launch per decode step, the peers writing while the reduction runs:
    every output bit-exact; every chunk's last validation clean."""
    w = synth.LLAMA8B_DECODE
    run = StepRun(w, 8, persistent=1)
    for T in w.tokens:
        for rep in range(3):
            epochs = run.step(T)
            run.s.check()
            got = to_host(run.out_d)
            exp = oracle.reduce_chain(run.pool, epochs, T)
            for i in range(w.reduces_per_step):
                assert np.array_equal(got[i, :T], exp[i]), f"T={T} rep={rep} node={i}"
            log = run.s.read_log()[:, :T * 8]
            assert np.all((log >> 24) == 0), "a chunk was accepted with a stale stamp"
            assert np.all((log & 0xFFFF) >= 1)
    run.s.close()


def test_persistent_many_steps_sampled():
    """100 persistent steps per batch size (the benchmark's shape), sampled."""
    w = synth.LLAMA8B_DECODE
    run = StepRun(w, 8, persistent=1)
    for T in w.tokens:
        for step in range(w.steps):
            epochs = run.step(T)
            if step % 11 == 0:
                got = to_host(run.out_d)
                for i in range(0, w.reduces_per_step, 5):
                    g = epochs[i]
                    exp = oracle.reduce(run.pool[(g - 1) % run.pool.shape[0]][:, :T])
                    assert np.array_equal(got[i, :T], exp), f"T={T} step={step} node={i}"
        run.s.check()
    run.s.close()


@pytest.mark.parametrize("persistent", [0, 1])
def test_steps_with_a_changing_batch_size(persistent):
    """Decode steps whose token count changes from step to step (seeded draws
    from 1..8), so chunks sit idle for some steps and are picked up again with
    older stamps and slot words; every output of every step is checked."""
    w = synth.LLAMA8B_DECODE
    run = StepRun(w, 8, persistent=persistent)
    rng = np.random.default_rng(4242)
    for step in range(24):
        T = int(rng.integers(1, 9))
        epochs = run.step(T)
        got = to_host(run.out_d)
        for i, g in enumerate(epochs):
            exp = oracle.reduce(run.pool[(g - 1) % run.pool.shape[0]][:, :T])
            assert np.array_equal(got[i, :T], exp), f"step {step} T={T} node {i}"
    run.s.check()
    run.s.close()


@pytest.mark.parametrize("T", [4, 8])
def test_persistent_late_stamps(T):
    """Late ranks' stamps land after a delay while the reduction waits on them:
    outputs equal the oracle; the decision log shows retries and ends clean.
    (The grouped producer meets late stamps in the epilogue tests below.)"""
    w = synth.SPEC_STRESS
    steps = 6
    late = synth.delay_table(w.wid, w.nranks, w.reduces_per_step * steps, w.stale_prob)
    run = StepRun(w, T, persistent=1, late_delay=4)
    run.s.set_injection(inject_table(late))
    retried = 0
    for step in range(steps):
        print(f"late stamps T={T} step {step}", flush=True)
        epochs = run.step(T)
        got = to_host(run.out_d)
        exp = oracle.reduce_chain(run.pool, epochs, T)
        for i in range(w.reduces_per_step):
            assert np.array_equal(got[i, :T], exp[i]), f"step={step} node={i}"
        log = run.s.read_log()[:, :T * 8]
        assert np.all((log >> 24) == 0)
        retried += int(np.count_nonzero((log & 0xFFFF) > 1))
    run.s.check()
    run.s.close()
    assert retried > 0


@pytest.mark.parametrize("T,H,epilogue", [(2, 1024, False), (8, 4096, False), (64, 4096, True)])
def test_persistent_withheld_stamp_latches(T, H, epilogue):
    """A stamp that never lands ends the step with a latched error instead of
    a hang. With the epilogue, 64 tokens x 8 chunks run in 4-wave workgroups:
    the grouped producer, and groups that wait for each other's sums of
    squares while their own wait fails."""
    w = synth.Workload(70, "withheld", 4, (T,), H, 8, 1, "normal", epilogue=epilogue)
    run = StepRun(w, T, persistent=1, max_attempts=64, spin_limit=1 << 14)
    table = [0] * 16
    table[4] = 0b0010 << 8      # epoch 5: rank 1's stamp never lands
    run.s.set_injection(table)
    print(f"withheld T={T} H={H} epilogue={epilogue}", flush=True)
    run.step(T)
    assert run.s.status() == S.SIFAR_EDEVICE
    kind, epoch, chunk, attempts = run.s.error_info()
    assert kind in (S.SIFAR_DEV_RETRY_BUDGET, S.SIFAR_DEV_WAW)
    assert epoch >= 5
    run.s.close()


@pytest.mark.parametrize("T", [1, 8, 32])
def test_persistent_epilogue_moe_chain(T):
    """120 chained all-reduces + residual-add + RMSNorm in one launch per step."""
    w = synth.MOE_DECODE
    run = StepRun(w, 32, persistent=1)
    res = run.res0[:T].copy()
    for step in range(2):
        epochs = run.step(T)
        y_got = to_host(run.y_d)
        _, r_list, y_list = oracle.reduce_chain(run.pool, epochs, T,
                                                epilogue=(res, run.weight, w.rms_eps))
        assert np.array_equal(to_host(run.res_d)[:T], r_list[-1])
        for i in range(w.reduces_per_step):
            assert ulp_distance(y_got[i, :T], y_list[i]).max() <= 1, f"step {step} node {i}"
        res = r_list[-1]
    run.s.check()
    run.s.close()


@pytest.mark.parametrize("T,steps", [(1, 100), (8, 10), (32, 3)])
def test_persistent_epilogue_moe_chain_late_stamps(T, steps):
    """The large-MoE workload as the persistent step runs it: N = 8, hidden
    8192, 120 all-reduces per step, each followed by residual-add + RMSNorm,
    each rank's stamp late (it lands late_delay sleeps after its payload) with
    p = 0.05. After every step the residual stream is bit-exact and every y
    within 1 bf16 step of the oracle; every chunk's decision word ends with a
    clean validation, and every logged mask is the one the logged raw stamps
    imply. Reports how many y elements sit 1 step away."""
    w = synth.MOE_DECODE
    late = synth.delay_table(w.wid, w.nranks, w.reduces_per_step * steps, w.stale_prob)
    run = StepRun(w, 32, persistent=1, late_delay=8)
    run.s.set_injection(inject_table(late))
    res = run.res0[:T].copy()
    segs = 16
    off_by_one = total = retried = 0
    for step in range(steps):
        if step % 10 == 0:
            print(f"persistent moe late stamps T={T} step {step} of {steps}", flush=True)
        epochs = run.step(T)
        y_got = to_host(run.y_d[:, :T])
        _, r_list, y_list = oracle.reduce_chain(run.pool, epochs, T,
                                                epilogue=(res, run.weight, w.rms_eps))
        assert np.array_equal(to_host(run.res_d)[:T], r_list[-1]), f"step {step}: residual"
        for i in range(w.reduces_per_step):
            d = ulp_distance(y_got[i, :T], y_list[i])
            assert d.max() <= 1, f"step {step} node {i}: y off by {d.max()} steps"
            off_by_one += int(np.count_nonzero(d))
            total += d.size
        res = r_list[-1]
        log = run.s.read_log()
        _, r = replay_logs(log, read_stamp_log(run.s), epochs, T * segs)
        retried += r
    run.s.check()
    run.s.close()
    print(f"persistent moe T={T}: {off_by_one} of {total} y elements 1 bf16 step from the "
          f"oracle ({off_by_one / total:.2e}); {retried} chunk validations polled again")
    assert retried > 0


@pytest.mark.parametrize("T", [4, 8])
def test_persistent_late_stamps_log_replay(T):
    """Free-running persistent steps with late stamps: each decision word is
    replayed from the raw stamps logged with it."""
    w = synth.SPEC_STRESS
    steps = 20
    late = synth.delay_table(w.wid, w.nranks, w.reduces_per_step * steps, w.stale_prob)
    run = StepRun(w, T, persistent=1, late_delay=4)
    run.s.set_injection(inject_table(late))
    checked = retried = 0
    for step in range(steps):
        epochs = run.step(T)
        got = to_host(run.out_d)
        for i in range(0, w.reduces_per_step, 9):
            g = epochs[i]
            assert np.array_equal(got[i, :T], oracle.reduce(run.pool[(g - 1) % run.pool.shape[0]][:, :T]))
        c, r = replay_logs(run.s.read_log(), read_stamp_log(run.s), epochs, T * 8)
        checked += c
        retried += r
    run.s.check()
    run.s.close()
    print(f"log replay T={T}: {checked} words, {retried} polled more than once")
    assert retried > 0


@pytest.mark.parametrize("N,T,H", [(5, 16, 3896), (8, 8, 4608), (3, 32, 2048),
                                   (8, 1, 1024), (4, 3, 1536), (2, 1, 512), (8, 5, 4608),
                                   (1, 4, 2048), (7, 2, 4096), (6, 128, 4096)])
def test_persistent_ragged_shapes(N, T, H):
    """Persistent steps on shapes off the benchmark grid: 3896 leaves a partial
    last chunk in each row (8 chunks per token, 128 chunks); 4608 has 9 chunks
    per token; N = 3 with 64 chunks. The next four have a number of workgroups
    per plane that is not a multiple of the 8 XCDs (2, 9, 1 and 45 chunks), so
    a chunk's producer and consumer run on different XCDs and meet only through
    agent-scope memory. Then one rank, an odd rank count, and 1024 chunks at
    N = 6."""
    w = synth.Workload(73, f"ragged-{N}-{T}-{H}", N, (T,), H, 12, 1, "normal")
    run = StepRun(w, T, persistent=1)
    for rep in range(3):
        print(f"ragged persistent N={N} T={T} H={H} rep {rep}", flush=True)
        epochs = run.step(T)
        got = to_host(run.out_d)
        exp = oracle.reduce_chain(run.pool, epochs, T)
        for i in range(w.reduces_per_step):
            assert np.array_equal(got[i, :T], exp[i]), f"rep={rep} node={i}"
    run.s.check()
    run.s.close()


def test_persistent_cross_xcd_many_steps():
    """64-all-reduce persistent steps, 2 chunks per plane (producer and
    consumer of a chunk on different XCDs), 40 steps, sampled."""
    w = synth.Workload(74, "cross-xcd", 8, (1,), 1024, 64, 40, "act")
    run = StepRun(w, 1, persistent=1)
    for step in range(w.steps):
        epochs = run.step(1)
        if step % 7 == 0:
            print(f"cross-xcd step {step}", flush=True)
            got = to_host(run.out_d)
            for i in range(0, w.reduces_per_step, 3):
                g = epochs[i]
                exp = oracle.reduce(run.pool[(g - 1) % run.pool.shape[0]][:, :1])
                assert np.array_equal(got[i, :1], exp), f"step={step} node={i}"
    run.s.check()
    log = run.s.read_log()[:, :2]
    assert np.all((log >> 24) == 0)
    run.s.close()


@pytest.mark.parametrize("N,T,H", [(8, 5, 4608), (8, 1, 1024)])
def test_persistent_cross_xcd_every_output(N, T, H):
    """150 persistent steps of 12 all-reduces with each chunk's producer and
    consumer on different XCDs, every output checked. A reduction that loaded
    the payload together with the stamps (the paper's speculation) accepted a
    rank's previous epoch under a fresh stamp in ~2 % of these all-reduces;
    the persistent step must validate before it loads."""
    w = synth.Workload(75, f"cross-xcd-{N}-{T}-{H}", N, (T,), H, 12, 150, "normal")
    run = StepRun(w, T, persistent=1)
    P = run.pool.shape[0]
    bad = []
    for step in range(w.steps):
        if step % 50 == 0:
            print(f"cross-xcd every output N={N} T={T} H={H} step {step}", flush=True)
        epochs = run.step(T)
        got = to_host(run.out_d)
        for i, g in enumerate(epochs):
            if not np.array_equal(got[i, :T], oracle.reduce(run.pool[(g - 1) % P][:, :T])):
                bad.append((step, i))
    run.s.check()
    run.s.close()
    assert not bad, f"{len(bad)} of {w.steps * w.reduces_per_step} all-reduces differ: {bad[:5]}"


def test_persistent_after_eager_and_graph_steps():
    """Eager epochs, fused graph steps and persistent steps on one handle."""
    w = synth.Workload(71, "mixed-modes", 8, (2,), 4096, 6, 1, "act")
    pool = synth.payload_pool(71, 8, 2, 4096, 19, "act")
    run_p = StepRun(w, 2, persistent=1, pool=pool)
    out = torch.zeros((2, 4096), dtype=torch.int16, device=DEV)
    extra = to_dev(synth.payload_pool(72, 8, 2, 4096, 3, "act"))
    extra_h = synth.payload_pool(72, 8, 2, 4096, 3, "act")
    for k in range(3):
        run_p.s.produce(extra[k], 2)
        run_p.s.reduce(out, 2)
        assert np.array_equal(to_host(out), oracle.reduce(extra_h[k]))
        epochs = run_p.step(2)
        got = to_host(run_p.out_d)
        exp = oracle.reduce_chain(run_p.pool, epochs, 2)
        for i in range(6):
            assert np.array_equal(got[i, :2], exp[i]), (k, i)
    run_p.s.check()
    run_p.s.close()


# ---- one buffer per rank: the bottom-barrier baseline ----------------------

@pytest.mark.parametrize("mode,persistent", [("spec", 0), ("ordered", 0), ("ordered", 1)])
def test_single_buffer_steps(mode, persistent):
    """buffers = 1: each rank has one slot, rewritten only after the previous
    all-reduce finished reading it. Same outputs, bit-exact."""
    w = synth.LLAMA8B_DECODE
    run = StepRun(w, 8, validate=mode, persistent=persistent, buffers=1)
    for T in (1, 8):
        for rep in range(2):
            epochs = run.step(T)
            got = to_host(run.out_d)
            exp = oracle.reduce_chain(run.pool, epochs, T)
            for i in range(w.reduces_per_step):
                assert np.array_equal(got[i, :T], exp[i]), f"T={T} rep={rep} node={i}"
    run.s.check()
    run.s.close()


def test_single_buffer_eager_order():
    N, T, H = 4, 1, 1024
    pool = synth.payload_pool(9, N, T, H, 3, "normal")
    src = to_dev(pool)
    out = torch.zeros((T, H), dtype=torch.int16, device=DEV)
    with S.Sifar(nranks=N, hidden=H, max_tokens=T, reduces_per_step=2, buffers=1) as s:
        s.produce(src[0], T)
        with pytest.raises(S.SifarError) as e:
            s.produce(src[1], T)   # the only slot still holds epoch 1
        assert e.value.code == S.SIFAR_ESTATE
        s.reduce(out, T)
        assert np.array_equal(to_host(out), oracle.reduce(pool[0]))
        s.produce(src[1], T)
        s.reduce(out, T)
        assert np.array_equal(to_host(out), oracle.reduce(pool[1]))
        s.check()


def test_single_buffer_epilogue_persistent():
    w = synth.MOE_DECODE
    run = StepRun(w, 8, persistent=1, buffers=1)
    T = 8
    res = run.res0[:T].copy()
    epochs = run.step(T)
    y_got = to_host(run.y_d)
    _, r_list, y_list = oracle.reduce_chain(run.pool, epochs, T, epilogue=(res, run.weight, w.rms_eps))
    assert np.array_equal(to_host(run.res_d)[:T], r_list[-1])
    for i in range(w.reduces_per_step):
        assert ulp_distance(y_got[i, :T], y_list[i]).max() <= 1
    run.s.check()
    run.s.close()


def test_two_persistent_handles_step_concurrently():
    """Two handles whose persistent steps are enqueued on two streams at once
    (default priority), small enough that both steps' waves are resident
    together: each handle's chain is its own (own slots, stamps and epoch
    counter), so both sequences of outputs equal the oracle's."""
    wa = synth.Workload(80, "concurrent-a", 8, (1,), 4096, 64, 1, "act")
    wb = synth.Workload(81, "concurrent-b", 4, (2,), 2048, 32, 1, "normal")
    ra = StepRun(wa, 1, persistent=1)
    rb = StepRun(wb, 2, persistent=1)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for step in range(10):
        with torch.cuda.stream(sa):
            ea = ra.step(1)
        with torch.cuda.stream(sb):
            eb = rb.step(2)
    torch.cuda.synchronize()
    print("two handles: 10 concurrent steps each", flush=True)
    for run, epochs, T in ((ra, ea, 1), (rb, eb, 2)):
        run.s.check()
        got = to_host(run.out_d)
        exp = oracle.reduce_chain(run.pool, epochs, T)
        for i in range(run.L):
            assert np.array_equal(got[i, :T], exp[i]), (run.w.name, i)
        run.s.close()


@pytest.mark.parametrize("G", [2, 8, 16])
@pytest.mark.parametrize("mode", ["spec", "ordered"])
def test_graph_steps_multiwave_groups(G, mode):
    """Per-launch steps with several waves per workgroup: the shape word the
    kernel receives as a preloaded argument carries log2 of the waves per
    group, and rows of 9 and 3 chunks leave idle waves in the last group of
    each token (they must load in bounds and store nothing). Every output of
    two steps per batch size."""
    w = synth.Workload(82, f"multiwave-g{G}", 8, (1, 5), 4608, 8, 1, "act")
    run = StepRun(w, 5, validate=mode, waves_per_group=G, pool=synth.payload_pool(82, 8, 5, 4608, 7, "act"))
    for T in (1, 5):
        for rep in range(2):
            epochs = run.step(T)
            got = to_host(run.out_d)
            exp = oracle.reduce_chain(run.pool, epochs, T)
            for i in range(w.reduces_per_step):
                assert np.array_equal(got[i, :T], exp[i]), (G, mode, T, rep, i)
    run.s.check()
    run.s.close()
    w2 = synth.Workload(83, f"multiwave-small-g{G}", 3, (2,), 1032, 6, 1, "normal")
    run2 = StepRun(w2, 2, validate=mode, waves_per_group=G, pool=synth.payload_pool(83, 3, 2, 1032, 5, "normal"))
    epochs = run2.step(2)
    got = to_host(run2.out_d)
    exp = oracle.reduce_chain(run2.pool, epochs, 2)
    for i in range(w2.reduces_per_step):
        assert np.array_equal(got[i, :2], exp[i]), (G, mode, "small", i)
    run2.s.check()
    run2.s.close()


def _random_shapes(n=12, seed=2607):
    """Seeded shapes off every grid: N = 1..8 ranks, rows of 8..9000 elements
    (ragged last chunks), 1..48 tokens (at most 1024 chunks), with or without
    the epilogue, 3..8 all-reduces per step."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        N = int(rng.integers(1, 9))
        H = 8 * int(rng.integers(1, 1126))
        T = int(rng.integers(1, 49))
        if T * -(-H // 512) > 1024:
            continue
        cases.append((N, T, H, bool(rng.integers(0, 2)), int(rng.integers(3, 9))))
    return cases


@pytest.mark.parametrize("case", range(12))
def test_random_shapes_both_step_forms(case):
    """The same seeded shape as a captured per-launch step (SPEC) and as a
    persistent step (ORDERED), two steps each: every all-reduce output
    bit-exact, or with the epilogue the residual bit-exact and every y within
    1 bf16 step."""
    N, T, H, epi, L = _random_shapes()[case]
    for persistent in (0, 1):
        w = synth.Workload(120 + case, f"random-{case}", N, (T,), H, L, 2, "act", epilogue=epi)
        run = StepRun(w, T, persistent=persistent,
                      pool=synth.payload_pool(w.wid, N, T, H, 5, w.dist))
        res = run.res0[:T].copy() if epi else None
        for step in range(2):
            print(f"random case {case}: N={N} T={T} H={H} epilogue={epi} L={L} "
                  f"persistent={persistent} step {step}", flush=True)
            epochs = run.step(T)
            if epi:
                y_got = to_host(run.y_d)
                _, r_list, y_list = oracle.reduce_chain(run.pool, epochs, T,
                                                        epilogue=(res, run.weight, w.rms_eps))
                assert np.array_equal(to_host(run.res_d)[:T], r_list[-1]), (case, persistent, step)
                for i in range(L):
                    assert ulp_distance(y_got[i, :T], y_list[i]).max() <= 1, (case, persistent, step, i)
                res = r_list[-1]
            else:
                got = to_host(run.out_d)
                exp = oracle.reduce_chain(run.pool, epochs, T)
                for i in range(L):
                    assert np.array_equal(got[i, :T], exp[i]), (case, persistent, step, i)
        run.s.check()
        run.s.close()
