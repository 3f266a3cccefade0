"""CPU oracle for SiFAR's one-shot all-reduce -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import, call, link or execute anything under ``oracle/``. The
GPU library never does, and it shares no code with this package: the two meet
only on the seeded inputs drawn by ``synth``.

Contents
  ref.c      plain C: the fixed-order fp32 sum rounded to bf16 (Sec. 3.1 and
             the pull-and-reduce listing of Sec. 4.2) and the residual-add +
             RMSNorm epilogue (paper silent; fp64 reading)
  ref_np.py  a second, bit-level numpy implementation of the same definitions,
             cross-checked against ref.c
  sim.py     a deterministic interleaving simulator of the stamp / validate /
             retry protocol (Sec. 4.1-4.2, correctness argument of Sec. 8.1)
  par.c      a host-thread driver of ref.c's reduction over slices of the
             elements (no arithmetic of its own), for the benchmark's
             multi-core CPU baseline

This module wraps ref.c through ctypes. ``build()`` compiles it with gcc.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "ref.c")
PAR = os.path.join(HERE, "par.c")
LIB = os.path.join(HERE, "libsifar_oracle.so")
CFLAGS = ["-O2", "-fno-fast-math", "-ffp-contract=off", "-fPIC", "-shared", "-std=c11"]

_lib = None


def build(force: bool = True) -> str:
    """Compile ref.c into libsifar_oracle.so (always, unless force=False and it exists)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.run(["gcc", *CFLAGS, SRC, PAR, "-o", tmp, "-lm", "-lpthread"], check=True)
        os.replace(tmp, LIB)
    return LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build(force=False)
        L = ctypes.CDLL(LIB)
        L.oracle_bf16_value.argtypes = [ctypes.c_uint16]
        L.oracle_bf16_value.restype = ctypes.c_double
        L.oracle_bf16_round.argtypes = [ctypes.c_double]
        L.oracle_bf16_round.restype = ctypes.c_uint16
        L.oracle_reduce.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t,
                                    ctypes.c_size_t, ctypes.c_void_p]
        L.oracle_reduce.restype = None
        L.oracle_residual_rmsnorm.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                              ctypes.c_double, ctypes.c_void_p]
        L.oracle_residual_rmsnorm.restype = None
        L.oracle_bf16_round_array.argtypes = [ctypes.c_void_p, ctypes.c_size_t,
                                              ctypes.c_void_p]
        L.oracle_bf16_round_array.restype = None
        L.oracle_bf16_value_array.argtypes = [ctypes.c_void_p, ctypes.c_size_t,
                                              ctypes.c_void_p]
        L.oracle_bf16_value_array.restype = None
        L.oracle_reduce_threads.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t,
                                            ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int]
        L.oracle_reduce_threads.restype = ctypes.c_int
        L.oracle_fp_env_ok.argtypes = []
        L.oracle_fp_env_ok.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def bf16_value(b: int) -> float:
    return lib().oracle_bf16_value(int(b) & 0xFFFF)


def bf16_round(x: float) -> int:
    return int(lib().oracle_bf16_round(float(x)))


def bf16_round_array(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    lib().oracle_bf16_round_array(_ptr(x), x.size, _ptr(out))
    return out


def bf16_value_array(b: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    out = np.empty(b.shape, dtype=np.float64)
    lib().oracle_bf16_value_array(_ptr(b), b.size, _ptr(out))
    return out


def fp_env_ok() -> bool:
    return bool(lib().oracle_fp_env_ok())


def reduce(x: np.ndarray) -> np.ndarray:
    """Fixed-order fp32 sum over axis 0 of bf16 bits ``x[N, ...]``, rounded to bf16."""
    x = np.ascontiguousarray(x, dtype=np.uint16)
    n = x.shape[0]
    count = x[0].size
    out = np.empty(x.shape[1:], dtype=np.uint16)
    lib().oracle_reduce(_ptr(x), n, count, count, _ptr(out))
    return out


def reduce_threads(x: np.ndarray, threads: int) -> np.ndarray:
    """``reduce`` computed by ``threads`` host threads, each running the same
    C reduction on a contiguous slice of the elements (bit-identical)."""
    x = np.ascontiguousarray(x, dtype=np.uint16)
    n = x.shape[0]
    count = x[0].size
    out = np.empty(x.shape[1:], dtype=np.uint16)
    used = lib().oracle_reduce_threads(_ptr(x), n, count, count, _ptr(out), int(threads))
    if used < 0:
        raise RuntimeError("oracle_reduce_threads could not start its threads")
    return out


def residual_rmsnorm(a: np.ndarray, res: np.ndarray, w: np.ndarray, eps: float):
    """Returns (res', y) for bf16 bits a[T, H], res[T, H], w[H]; res is not modified."""
    a = np.ascontiguousarray(a, dtype=np.uint16)
    r = np.array(res, dtype=np.uint16, copy=True, order="C")
    w = np.ascontiguousarray(w, dtype=np.uint16)
    T, H = a.shape
    y = np.empty_like(a)
    lib().oracle_residual_rmsnorm(_ptr(a), _ptr(r), _ptr(w), T, H, float(eps), _ptr(y))
    return r, y


def reduce_chain(pool: np.ndarray, epochs, tokens: int, epilogue=None):
    """Outputs of a chain of reduces, one per epoch g in ``epochs``.

    pool: uint16 [P][N][T_max][H]; epoch g reduces entry (g - 1) % P restricted
    to the first ``tokens`` tokens. With ``epilogue = (res0, w, eps)`` each
    reduce feeds the residual-add + RMSNorm chain and the function returns
    (a_list, res_list, y_list); otherwise the list of reduce outputs.
    """
    P = pool.shape[0]
    outs, ress, ys = [], [], []
    res = None if epilogue is None else np.array(epilogue[0], dtype=np.uint16, copy=True)
    for g in epochs:
        a = reduce(pool[(g - 1) % P][:, :tokens, :])
        outs.append(a)
        if epilogue is not None:
            res, y = residual_rmsnorm(a, res, epilogue[1], epilogue[2])
            ress.append(res)
            ys.append(y)
    if epilogue is None:
        return outs
    return outs, ress, ys
