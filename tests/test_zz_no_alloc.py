"""GPU: the allocation-free all-reduce (sifar_allreduce_noalloc), called
through the C ABI, against the handle-based entry points it is a variant of
(sifar_produce + sifar_reduce on a SIFAR_VALIDATE_SPEC handle) and against the
CPU oracle: bit-exact, on calls in a row whose sizes shrink, so that each call
runs over what the previous one left in the static array."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2607_08973_amd as S
import synth

from sifar_harness import DEV, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    S.load()
    yield
    torch.cuda.synchronize()


def _handle_result(x: np.ndarray) -> np.ndarray:
    """The same all-reduce through a handle: sifar_produce, then sifar_reduce."""
    N, T, H = x.shape
    out = torch.zeros((T, H), dtype=torch.int16, device=DEV)
    with S.Sifar(nranks=N, hidden=H, max_tokens=T, reduces_per_step=2, validate="spec",
                 log_epochs=2) as s:
        s.produce(to_dev(x), T)
        s.reduce(out, T)
        s.check()
    return to_host(out)


def _noalloc(x_d: torch.Tensor, N: int, T: int, H: int, rank_stride: int) -> torch.Tensor:
    out = torch.zeros((T, H), dtype=torch.int16, device=DEV)
    torch.cuda.synchronize()  # the output exists before the call; the call allocates nothing
    S.sifar_allreduce_noalloc(x_d, rank_stride, N, T, H, out)
    return out


# (N, T, H): the first call of each sequence is the larger one
SEQUENCES = [
    [(8, 8, 4096), (4, 3, 1000)],        # the decode workload's widest batch, then a ragged row
    [(8, 64, 4096), (2, 1, 4096)],       # the largest accepted size, then the smallest decode shape
    [(5, 16, 8192), (8, 1, 520)],        # odd rank count; then a 2-chunk row with a short tail
]


@pytest.mark.parametrize("seq", SEQUENCES, ids=lambda q: "-".join(f"n{n}t{t}h{h}" for n, t, h in q))
def test_noalloc_matches_the_handle_path(seq):
    for k, (N, T, H) in enumerate(seq):
        print(f"noalloc call {k}: N={N} T={T} H={H}", flush=True)
        x = synth.payload_pool(300 + k, N, T, H, 1, "act")[0]
        got = to_host(_noalloc(to_dev(x), N, T, H, T * H))
        torch.cuda.synchronize()
        want = _handle_result(x)
        assert np.array_equal(got, want), f"call {k}: differs from sifar_produce + sifar_reduce"
        assert np.array_equal(got, oracle.reduce(x)), f"call {k}: differs from the oracle"


def test_noalloc_calls_queued_back_to_back():
    """Eight calls enqueued on one stream without a synchronisation between
    them, sizes shrinking and growing, a padded rank stride; every output
    checked afterwards."""
    shapes = [(8, 8, 4096), (8, 2, 4096), (3, 5, 1536), (8, 1, 4096), (1, 4, 2048),
              (8, 4, 4096), (6, 2, 8192), (2, 1, 8)]
    xs, outs = [], []
    for k, (N, T, H) in enumerate(shapes):
        x = synth.payload_pool(400 + k, N, T, H, 1, "normal")[0]
        stride = T * H + 8 * k  # a rank stride longer than the row block
        xpad = np.zeros((N, stride), np.uint16)
        xpad[:, :T * H] = x.reshape(N, T * H)
        xs.append(x)
        outs.append((to_dev(xpad), torch.zeros((T, H), dtype=torch.int16, device=DEV)))
    torch.cuda.synchronize()
    print("noalloc: 8 calls queued", flush=True)
    for (N, T, H), (x_d, out) in zip(shapes, outs):
        S.sifar_allreduce_noalloc(x_d, x_d.shape[1], N, T, H, out)
    torch.cuda.synchronize()
    for k, (x, (_, out)) in enumerate(zip(xs, outs)):
        assert np.array_equal(to_host(out), oracle.reduce(x)), f"call {k}"


def test_noalloc_refuses_a_size_beyond_its_array():
    x_d = torch.zeros((2, 64 * 8192), dtype=torch.int16, device=DEV)
    out = torch.zeros((64, 8192), dtype=torch.int16, device=DEV)
    with pytest.raises(S.SifarError) as e:
        S.sifar_allreduce_noalloc(x_d, 64 * 8192, 2, 64, 8192, out)
    assert e.value.code == S.SIFAR_EINVAL
