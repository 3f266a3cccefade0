"""Python binding of libsifar, the MI355X one-shot all-reduce of SiFAR.

Argument marshalling only: every step of the all-reduce runs in the HIP
kernels behind ``include/sifar.h``. PyTorch supplies device memory and streams;
tensors are passed as raw device pointers (``torch.bfloat16`` tensors, or
``int16``/``uint16`` views of bf16 bits) and streams as ``hipStream_t``.

The functions keep the C names (``sifar_init``, ``sifar_produce``,
``sifar_reduce``, ``sifar_reduce_rmsnorm``, ``sifar_bind_step``, ``sifar_step``
...) and raise ``SifarError`` on a negative return code. ``Sifar`` is a small
owning wrapper around a handle.

The shared library is built in-tree by ``paper_2607_08973_amd.build``; this
module refuses to load without it (there is no fallback path).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libsifar.so")

SIFAR_OK = 0
SIFAR_EINVAL = -1
SIFAR_ENOMEM = -2
SIFAR_EHIP = -3
SIFAR_ESTATE = -4
SIFAR_EDEVICE = -5

SIFAR_DEV_RETRY_BUDGET = 1
SIFAR_DEV_WAW = 2
SIFAR_DEV_EXCHANGE = 3

SIFAR_VALIDATE_SPEC = 0
SIFAR_VALIDATE_ORDERED = 1
SIFAR_VALIDATE_NONE = 2
VALIDATE = {"spec": 0, "ordered": 1, "none": 2}

SIFAR_INJECT_OFF = 0
SIFAR_INJECT_DETERMINISTIC = 1
SIFAR_INJECT_SLOT_OVERRUN = 2

# latency floors (sifar_floor kinds)
SIFAR_FLOOR_GRAPH_NODE = 0
SIFAR_FLOOR_EAGER_LAUNCH = 1
SIFAR_FLOOR_ATOMIC = 2
SIFAR_FLOOR_ACQUIRE_LOAD = 3
SIFAR_FLOOR_COHERENT_LOAD = 4
SIFAR_FLOOR_WARM_LOAD = 5
SIFAR_FLOOR_COLD_LOAD = 6
SIFAR_FLOOR_RELEASE_FENCE = 7
SIFAR_FLOOR_PINGPONG_XCD = 8
SIFAR_FLOOR_PINGPONG_SAME_XCD = 9

SIFAR_LITMUS_ORDERED = 0
SIFAR_LITMUS_READ_FIRST = 1
SIFAR_LITMUS_ORDERED_PREFETCH = 2
SIFAR_LITMUS_CROSS_XCD = 0
SIFAR_LITMUS_SAME_XCD = 1

# the allocation-free entry point's limits and its static array
SIFAR_NOALLOC_MAX_TOKENS = 64
SIFAR_NOALLOC_MAX_ELEMS = 262144
SIFAR_NOALLOC_SCRATCH_BYTES = 8437248

CHUNK = 512  # elements per chunk (one 64-lane wave, 16 bytes per lane)

# every symbol include/sifar.h declares
EXPORTS = (
    "sifar_config_default", "sifar_version", "sifar_init", "sifar_destroy",
    "sifar_produce", "sifar_reduce", "sifar_reduce_rmsnorm", "sifar_bind_step",
    "sifar_step", "sifar_set_injection", "sifar_log_geometry", "sifar_read_log",
    "sifar_read_stamp_log",
    "sifar_epochs", "sifar_status", "sifar_error_info", "sifar_strerror", "sifar_floor",
    "sifar_litmus", "sifar_allreduce_noalloc",
)


class sifar_litmus_result(ctypes.Structure):
    _fields_ = [
        ("trials", ctypes.c_uint64),
        ("violations", ctypes.c_uint64),
        ("violations_first_epochs", ctypes.c_uint64),
        ("timeouts", ctypes.c_uint64),
        ("pairs_placed", ctypes.c_uint32),
        ("pairs", ctypes.c_uint32),
        ("ns_per_trial", ctypes.c_double),
        ("first_bad", ctypes.c_uint32 * 4),
    ]


class sifar_config(ctypes.Structure):
    _fields_ = [
        ("nranks", ctypes.c_int32),
        ("hidden", ctypes.c_int32),
        ("max_tokens", ctypes.c_int32),
        ("reduces_per_step", ctypes.c_int32),
        ("validate", ctypes.c_int32),
        ("epilogue", ctypes.c_int32),
        ("rms_eps", ctypes.c_float),
        ("max_attempts", ctypes.c_uint32),
        ("forced_retries", ctypes.c_uint32),
        ("spin_limit", ctypes.c_uint32),
        ("log_epochs", ctypes.c_int32),
        ("waves_per_group", ctypes.c_int32),
        ("fuse_peers", ctypes.c_int32),
        ("persistent", ctypes.c_int32),
        ("late_delay", ctypes.c_uint32),
        ("buffers", ctypes.c_int32),
    ]


class sifar_step_buffers(ctypes.Structure):
    _fields_ = [
        ("src_pool", ctypes.c_void_p),
        ("pool_entries", ctypes.c_int32),
        ("pool_entry_stride", ctypes.c_int64),
        ("pool_rank_stride", ctypes.c_int64),
        ("out_ring", ctypes.c_void_p),
        ("residual", ctypes.c_void_p),
        ("weight", ctypes.c_void_p),
        ("y_ring", ctypes.c_void_p),
    ]


class SifarError(RuntimeError):
    def __init__(self, fn: str, code: int, info=None):
        msg = f"{fn} failed: {code} ({strerror(code)})"
        if info is not None:
            msg += f"; device info {list(info)}"
        super().__init__(msg)
        self.code = code
        self.info = info


_lib = None


def load(path: str = LIB_PATH):
    """Load libsifar.so (once). PyTorch is imported first so that the library
    binds to the same HIP runtime as the tensors and streams it receives."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (shares its HIP runtime with the library)

    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: run `python -m paper_2607_08973_amd.build` "
                          "(or __graft_entry__.build()) first; there is no fallback path")
    L = ctypes.CDLL(path)
    P, I32, I64, U32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_size_t
    sig = {
        "sifar_config_default": (None, [ctypes.POINTER(sifar_config)]),
        "sifar_version": (ctypes.c_int, []),
        "sifar_init": (ctypes.c_int, [ctypes.POINTER(sifar_config), ctypes.POINTER(P)]),
        "sifar_destroy": (None, [P]),
        "sifar_produce": (ctypes.c_int, [P, P, I64, I32, P]),
        "sifar_reduce": (ctypes.c_int, [P, P, I32, P]),
        "sifar_reduce_rmsnorm": (ctypes.c_int, [P, P, P, P, I32, P]),
        "sifar_bind_step": (ctypes.c_int, [P, ctypes.POINTER(sifar_step_buffers)]),
        "sifar_step": (ctypes.c_int, [P, I32, P]),
        "sifar_set_injection": (ctypes.c_int, [P, P, I32, I32]),
        "sifar_log_geometry": (ctypes.c_int, [P, ctypes.POINTER(I32), ctypes.POINTER(I32),
                                              ctypes.POINTER(I32)]),
        "sifar_read_log": (ctypes.c_int, [P, P, SZ]),
        "sifar_read_stamp_log": (ctypes.c_int, [P, P, SZ]),
        "sifar_epochs": (ctypes.c_int, [P, ctypes.POINTER(U32), ctypes.POINTER(U32)]),
        "sifar_status": (ctypes.c_int, [P]),
        "sifar_error_info": (ctypes.c_int, [P, ctypes.POINTER(U32)]),
        "sifar_strerror": (ctypes.c_char_p, [ctypes.c_int]),
        "sifar_floor": (ctypes.c_int, [I32, I32, P, ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(U32)]),
        "sifar_litmus": (ctypes.c_int, [I32, I32, I32, I32, P,
                                        ctypes.POINTER(sifar_litmus_result)]),
        "sifar_allreduce_noalloc": (ctypes.c_int, [P, I64, I32, I32, I32, P, P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def strerror(code: int) -> str:
    return load().sifar_strerror(int(code)).decode()


def _check(fn: str, code: int):
    if code != SIFAR_OK:
        raise SifarError(fn, code)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ---- C-named thin wrappers -------------------------------------------------

def sifar_config_default() -> sifar_config:
    c = sifar_config()
    load().sifar_config_default(ctypes.byref(c))
    return c


def sifar_version() -> int:
    return load().sifar_version()


def sifar_init(cfg: sifar_config) -> int:
    h = ctypes.c_void_p()
    _check("sifar_init", load().sifar_init(ctypes.byref(cfg), ctypes.byref(h)))
    return h.value


def sifar_destroy(h: int) -> None:
    load().sifar_destroy(h)


def sifar_produce(h: int, src, src_rank_stride: int, tokens: int, stream=None) -> None:
    _check("sifar_produce", load().sifar_produce(h, _ptr(src), src_rank_stride, tokens,
                                                 _stream(stream)))


def sifar_reduce(h: int, out, tokens: int, stream=None) -> None:
    _check("sifar_reduce", load().sifar_reduce(h, _ptr(out), tokens, _stream(stream)))


def sifar_reduce_rmsnorm(h: int, residual, weight, y, tokens: int, stream=None) -> None:
    _check("sifar_reduce_rmsnorm", load().sifar_reduce_rmsnorm(
        h, _ptr(residual), _ptr(weight), _ptr(y), tokens, _stream(stream)))


def sifar_bind_step(h: int, src_pool, pool_entries: int, pool_entry_stride: int,
                    pool_rank_stride: int, out_ring=None, residual=None, weight=None,
                    y_ring=None) -> None:
    b = sifar_step_buffers(_ptr(src_pool), pool_entries, pool_entry_stride, pool_rank_stride,
                           _ptr(out_ring), _ptr(residual), _ptr(weight), _ptr(y_ring))
    _check("sifar_bind_step", load().sifar_bind_step(h, ctypes.byref(b)))


def sifar_step(h: int, tokens: int, stream=None) -> None:
    _check("sifar_step", load().sifar_step(h, tokens, _stream(stream)))


def sifar_set_injection(h: int, table: Optional[Sequence[int]], mode: int) -> None:
    if mode == SIFAR_INJECT_SLOT_OVERRUN:
        _check("sifar_set_injection", load().sifar_set_injection(h, None, 0, mode))
        return
    if table is None or mode == SIFAR_INJECT_OFF:
        _check("sifar_set_injection", load().sifar_set_injection(h, None, 0, SIFAR_INJECT_OFF))
        return
    arr = (ctypes.c_uint16 * len(table))(*[int(x) for x in table])
    _check("sifar_set_injection", load().sifar_set_injection(h, arr, len(table), mode))


def sifar_log_geometry(h: int):
    a, b, c = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    _check("sifar_log_geometry", load().sifar_log_geometry(h, ctypes.byref(a), ctypes.byref(b),
                                                           ctypes.byref(c)))
    return a.value, b.value, c.value


def sifar_read_log(h: int):
    import numpy as np
    epochs, _, w_max = sifar_log_geometry(h)
    out = np.zeros((epochs, w_max), dtype=np.uint32)
    _check("sifar_read_log", load().sifar_read_log(h, out.ctypes.data, out.size))
    return out


def sifar_read_stamp_log(h: int, nranks: int):
    """Raw stamps of each chunk's first and last validation, flat
    ([log_epochs][w_max][2][N] in the header's order)."""
    import numpy as np
    epochs, _, w_max = sifar_log_geometry(h)
    out = np.zeros(epochs * w_max * 2 * nranks, dtype=np.uint32)
    _check("sifar_read_stamp_log", load().sifar_read_stamp_log(h, out.ctypes.data, out.size))
    return out


def sifar_epochs(h: int):
    a, b = ctypes.c_uint32(), ctypes.c_uint32()
    _check("sifar_epochs", load().sifar_epochs(h, ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def sifar_error_info(h: int):
    info = (ctypes.c_uint32 * 4)()
    _check("sifar_error_info", load().sifar_error_info(h, info))
    return list(info)


def sifar_floor(kind: int, iterations: int, stream=None):
    """One latency floor: returns (ns per operation, [completed, xcc_a, xcc_b, 0])."""
    ns = ctypes.c_double()
    info = (ctypes.c_uint32 * 4)()
    _check("sifar_floor", load().sifar_floor(kind, iterations, _stream(stream),
                                             ctypes.byref(ns), info))
    return ns.value, list(info)


def sifar_litmus(protocol: int, placement: int, pairs: int, trials: int, stream=None) -> dict:
    """Handoff litmus: returns the result fields as a dict. A bounded wait that
    gave up raises (after the result was read back)."""
    r = sifar_litmus_result()
    rc = load().sifar_litmus(protocol, placement, pairs, trials, _stream(stream), ctypes.byref(r))
    out = {name: getattr(r, name) for name, _ in sifar_litmus_result._fields_}
    out["first_bad"] = list(r.first_bad)
    if rc != SIFAR_OK:
        err = SifarError("sifar_litmus", rc)
        err.result = out
        raise err
    return out


def sifar_allreduce_noalloc(src, src_rank_stride: int, nranks: int, tokens: int, hidden: int,
                            out, stream=None) -> None:
    """One all-reduce on the library's static scratch (no allocation)."""
    _check("sifar_allreduce_noalloc", load().sifar_allreduce_noalloc(
        _ptr(src), src_rank_stride, nranks, tokens, hidden, _ptr(out), _stream(stream)))


def sifar_status(h: int) -> int:
    """Returns the status code (does not raise)."""
    return load().sifar_status(h)


# ---- owning wrapper --------------------------------------------------------

class Sifar:
    """One handle: ``Sifar(nranks=8, hidden=4096, max_tokens=8, ...)``."""

    def __init__(self, **kw):
        cfg = sifar_config_default()
        for k, v in kw.items():
            if k == "validate" and isinstance(v, str):
                v = VALIDATE[v]
            if not hasattr(cfg, k):
                raise TypeError(f"unknown config field {k!r}")
            setattr(cfg, k, v)
        self.cfg = cfg
        self.h = sifar_init(cfg)

    def close(self):
        if self.h:
            sifar_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def produce(self, src, tokens, src_rank_stride=None, stream=None):
        if src_rank_stride is None:
            src_rank_stride = src[0].numel()
        sifar_produce(self.h, src, src_rank_stride, tokens, stream)

    def reduce(self, out, tokens, stream=None):
        sifar_reduce(self.h, out, tokens, stream)

    def reduce_rmsnorm(self, residual, weight, y, tokens, stream=None):
        sifar_reduce_rmsnorm(self.h, residual, weight, y, tokens, stream)

    def bind_step(self, src_pool, out_ring=None, residual=None, weight=None, y_ring=None):
        """src_pool: [P][N][T_max][H] tensor."""
        P = src_pool.shape[0]
        sifar_bind_step(self.h, src_pool, P, src_pool.stride(0), src_pool.stride(1),
                        out_ring, residual, weight, y_ring)

    def step(self, tokens, stream=None):
        sifar_step(self.h, tokens, stream)

    def set_injection(self, table, mode=SIFAR_INJECT_DETERMINISTIC):
        sifar_set_injection(self.h, table, mode)

    def read_log(self):
        return sifar_read_log(self.h)

    def read_stamp_log(self):
        return sifar_read_stamp_log(self.h, self.cfg.nranks)

    def log_geometry(self):
        return sifar_log_geometry(self.h)

    def epochs(self):
        return sifar_epochs(self.h)

    def status(self) -> int:
        return sifar_status(self.h)

    def check(self):
        rc = sifar_status(self.h)
        if rc != SIFAR_OK:
            info = sifar_error_info(self.h) if rc == SIFAR_EDEVICE else None
            raise SifarError("sifar_status", rc, info)

    def error_info(self):
        return sifar_error_info(self.h)
