"""Seeded synthetic router scores for the DO-loss workloads.

This module is shared test/bench infrastructure: both the CPU oracle and the
HIP path read the bytes it produces.  It contains no DO-loss arithmetic (no
top-k, no signatures, no distances), only counter-based random draws shaped
into the score distributions described in ``gen.c``.

bf16 scores are returned as ``numpy.uint16`` bit patterns; fp32 as
``numpy.float32``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None

F32, BF16 = 0, 1
DTYPE_NAME = {F32: "f32", BF16: "bf16"}

# Workload table (mirrors the table in gen.c; the C side is the authority).
WORKLOADS = {
    0: dict(name="e8_k2_n4096_f32", layers=1, n=4096, E=8, k=2, dtype=F32),
    1: dict(name="e64_k6_n65536_bf16_bias", layers=1, n=65536, E=64, k=6, dtype=BF16),
    2: dict(name="l48_e128_k8_n262144_bf16_idle16", layers=48, n=262144, E=128, k=8, dtype=BF16),
    3: dict(name="stream16x65536_e128_k8_bf16_zipf", layers=16, n=65536, E=128, k=8, dtype=BF16),
    4: dict(name="l8_e256_k8_n4194304_f32_softmax_clusters", layers=8, n=4194304, E=256, k=8, dtype=F32),
}


def build(force: bool = True) -> str:
    """Compile gen.c into libsynth.so (gcc, OpenMP, portable x86-64 flags)."""
    global _lib
    if not force and os.path.exists(_LIB_PATH):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp"
    cmd = ["gcc", "-O3", "-ffast-math", "-mavx2", "-mfma", "-fPIC", "-shared", "-fopenmp", "-std=c11", _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    _lib = None
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        i64, i32, u64, dbl, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p
        lib.synth_normal.argtypes = [u64, u64, ctypes.c_int, i64, i64, i32, dbl, dbl, vp, ctypes.c_int]
        lib.synth_int_ties.argtypes = [u64, u64, ctypes.c_int, i64, i32, i32, i32, vp, ctypes.c_int]
        lib.synth_config_fill.argtypes = [ctypes.c_int, ctypes.c_int, i64, i64, vp, ctypes.c_int]
        lib.synth_config_bias.argtypes = [ctypes.c_int, ctypes.c_int, vp]
        lib.synth_config_clusters.argtypes = [ctypes.c_int, vp]
        for f in ("synth_normal", "synth_int_ties", "synth_config_fill", "synth_config_bias", "synth_config_clusters"):
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
    return _lib


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _empty(n: int, E: int, dtype: int, out=None):
    np_dt = np.float32 if dtype == F32 else np.uint16
    if out is None:
        return np.empty((n, E), dtype=np_dt)
    assert out.dtype == np_dt and out.shape == (n, E) and out.flags.c_contiguous
    return out


def normal(seed: int, n: int, E: int, dtype: int = F32, mean: float = 0.0, std: float = 1.0,
           stream: int = 0, t0: int = 0, threads: int | None = None, out=None) -> np.ndarray:
    """i.i.d. normal scores, shape (n, E)."""
    a = _empty(n, E, dtype, out)
    rc = _load().synth_normal(seed, stream, dtype, t0, n, E, mean, std, a.ctypes.data, threads or default_threads())
    if rc:
        raise ValueError("synth_normal: bad arguments")
    return a


def int_ties(seed: int, n: int, E: int, lo: int, hi: int, dtype: int = F32, stream: int = 0,
             threads: int | None = None) -> np.ndarray:
    """Integer-valued scores uniform on [lo, hi]: many exact ties per row."""
    a = _empty(n, E, dtype)
    rc = _load().synth_int_ties(seed, stream, dtype, n, E, lo, hi, a.ctypes.data, threads or default_threads())
    if rc:
        raise ValueError("synth_int_ties: bad arguments")
    return a


def workload_fill(cfg: int, layer: int, t0: int = 0, n: int | None = None, threads: int | None = None,
                  out=None) -> np.ndarray:
    """Scores of tokens [t0, t0+n) of one layer (workload 3: one micro-batch) of a workload."""
    w = WORKLOADS[cfg]
    if n is None:
        n = w["n"] - t0
    a = _empty(n, w["E"], w["dtype"], out)
    rc = _load().synth_config_fill(cfg, layer, t0, n, a.ctypes.data, threads or default_threads())
    if rc:
        raise ValueError("synth_config_fill: bad arguments")
    return a


def workload_bias(cfg: int, layer: int = 0) -> np.ndarray:
    """Per-expert additive bias of workloads 1-3 (zeros otherwise)."""
    b = np.zeros(256, dtype=np.float64)
    _load().synth_config_bias(cfg, layer, b.ctypes.data)
    return b[: WORKLOADS[cfg]["E"]].copy()


def workload_clusters(layer: int) -> np.ndarray:
    """Favoured experts of workload 4, shape (32, 8)."""
    f = np.zeros((32, 8), dtype=np.int32)
    _load().synth_config_clusters(layer, f.ctypes.data)
    return f


def bf16_bits_to_f32(a: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32 values."""
    return (a.astype(np.uint32) << 16).view(np.float32)
