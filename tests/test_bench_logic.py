"""The benchmark's byte accounting on the CPU: one consumer's algorithmic bytes
per all-reduce, the emulated peers' copies apart, and the per-launch table the
roofline fields are computed from. No GPU."""
from __future__ import annotations

import bench


def test_consumer_bytes_per_all_reduce():
    # read N payloads of T x H bf16, write one result, read N 4-byte stamps
    # per 512-element chunk
    assert bench.reduce_bytes(8, 1, 4096) == 8 * 8192 + 8192 + 4 * 8 * 8
    assert bench.reduce_bytes(2, 3, 1000) == 2 * 6000 + 6000 + 4 * 2 * 3 * 2
    # the epilogue adds res read + write, y write, and the weight
    assert bench.epilogue_bytes(4, 8192) == 3 * 4 * 8192 * 2 + 2 * 8192


def test_peer_copies_are_not_counted_as_all_reduce_bytes():
    N, T, H = 8, 4, 4096
    K = T * H * 2
    assert bench.produce_bytes(N, T, H) == 2 * N * K + 4 * N * T * 8
    per_t = {1: 0.8, 8: 0.85}
    # persistent: one launch of L all-reduces; its bytes are L consumer shares
    kp = bench.kernel_table(per_t, (1, 8), N, H, 64, True, True)
    assert kp[1]["bytes_per_launch"] == 64 * bench.reduce_bytes(N, 1, H)
    assert kp[1]["peer_copy_bytes_per_launch"] == 64 * bench.produce_bytes(N, 1, H)
    assert abs(kp[8]["launch_period_us"] - 0.85 * 64) < 1e-9
    # per launch with fused peers: L + 2 launches per step, one all-reduce each
    kl = bench.kernel_table(per_t, (1, 8), N, H, 64, False, True)
    assert kl[1]["bytes_per_launch"] == bench.reduce_bytes(N, 1, H)
    assert abs(kl[1]["launch_period_us"] - 0.8 * 64 / 66) < 1e-9
    assert abs(kl[1]["gbs"] - kl[1]["bytes_per_launch"] / (kl[1]["launch_period_us"] * 1e-6) / 1e9) < 1e-6
    # per launch without fused peers: the producer has launches of its own
    kn = bench.kernel_table(per_t, (1,), N, H, 64, False, False)
    assert kn[1]["peer_copy_bytes_per_launch"] == 0
    assert abs(kn[1]["launch_period_us"] - 0.8 * 64 / 129) < 1e-9


def test_kernel_digest_ignores_comments():
    d = bench.kernel_code_digest()
    assert len(d) == 64 and int(d, 16) >= 0
