"""DO-loss reference oracle -- TEST INFRASTRUCTURE ONLY.

Plain CPU implementation (``doloss_oracle.c``) of what the DO-loss hot path
computes, written from the paper's definitions (arXiv 2609.32398):

* ``topk_signature``  -- Sec. 3.1.1, Eq. (1): the dense bool matrix F[E][N] of
  Top-K token assignments (ties to the lower expert index, -0 == +0, NaN
  ranks below -inf and NaNs tie).
* ``pack``            -- the binary load signature of each expert as 64-bit
  words, token t -> word t//64, bit t%64, tail bits zero.
* ``hamming``         -- Eq. (6) G_ij = ||F_i - F_j||_1 from its definition.
* ``loss``            -- Eq. (3) sum_{i!=j} G_ij^2 (fp64 and exact integer),
  with mean and population variance of the off-diagonal distances
  (App. C.1).
* ``surrogate``       -- Sec. 3.1.3, Eq. (6)-(7): the surrogate loss
  (scale/(N^2 k)) sum_ij G_ij C_ij, C_ij = sum_t p_it (f_it - f_jt), and its
  gradient with respect to the routing probabilities (G, F detached).
* ``surrogate_loss_blocked`` -- the same loss with the token sums inside C
  taken by a numpy matrix product, for inputs of millions of tokens.
* ``load_stats``      -- per-expert loads n_i (App. C.3), the Local-LBL loss
  sum_i f_i P_i of Sec. 4.2 and MaxVio (App. E) over a rank placement.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may use this package.  It shares no code with the HIP library.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "doloss_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

F32, BF16 = 0, 1
CFLAGS = ["-O3", "-fPIC", "-shared", "-fopenmp", "-std=c11"]


class _LossResult(ctypes.Structure):
    _fields_ = [("sum", ctypes.c_uint64), ("sumsq", ctypes.c_uint64), ("loss", ctypes.c_double),
                ("mean", ctypes.c_double), ("var", ctypes.c_double)]


class _LoadStatsResult(ctypes.Structure):
    _fields_ = [("total", ctypes.c_uint64), ("max_load", ctypes.c_uint32), ("min_load", ctypes.c_uint32),
                ("lbl", ctypes.c_double), ("maxvio", ctypes.c_double)]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O3, OpenMP; portable x86-64 code, no -march)."""
    global _lib
    if not force and os.path.exists(_LIB_PATH):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp"
    subprocess.run(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"], check=True)
    os.replace(tmp, _LIB_PATH)
    _lib = None
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        i64, i32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
        lib.oracle_topk_signature.argtypes = [vp, ctypes.c_int, i64, i32, i32, vp, ctypes.c_int]
        lib.oracle_pack.argtypes = [vp, i64, i32, vp]
        lib.oracle_hamming.argtypes = [vp, i64, i32, vp, ctypes.c_int]
        lib.oracle_loss.argtypes = [vp, i32, ctypes.POINTER(_LossResult)]
        lib.oracle_surrogate.argtypes = [vp, ctypes.c_int, i64, i32, i32, vp, vp, ctypes.c_double,
                                         ctypes.POINTER(ctypes.c_double), vp, ctypes.c_int]
        lib.oracle_load_stats.argtypes = [vp, i64, i32, i32, vp, ctypes.c_int, vp, i32, vp,
                                          ctypes.POINTER(_LoadStatsResult)]
        for f in ("oracle_topk_signature", "oracle_pack", "oracle_hamming", "oracle_loss", "oracle_surrogate",
                  "oracle_load_stats"):
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
    return _lib


def threads() -> int:
    """Host threads the oracle uses (all available cores, capped at 16)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _dtype_of(scores: np.ndarray) -> int:
    if scores.dtype == np.float32:
        return F32
    if scores.dtype == np.uint16:
        return BF16
    raise TypeError("scores must be float32 values or uint16 bf16 bit patterns")


def topk_signature(scores: np.ndarray, k: int, nthreads: int | None = None) -> np.ndarray:
    """Eq. (1): dense F[E][N] (uint8 0/1) for scores of shape (N, E)."""
    scores = np.ascontiguousarray(scores)
    N, E = scores.shape
    F = np.empty((E, N), dtype=np.uint8)
    rc = _load().oracle_topk_signature(scores.ctypes.data, _dtype_of(scores), N, E, k, F.ctypes.data,
                                       nthreads or threads())
    if rc:
        raise ValueError(f"oracle_topk_signature: bad arguments N={N} E={E} k={k}")
    return F


def pack(F: np.ndarray) -> np.ndarray:
    """Signature words[E][ceil(N/64)] (uint64) of a dense F[E][N]."""
    F = np.ascontiguousarray(F, dtype=np.uint8)
    E, N = F.shape
    W = (N + 63) // 64
    words = np.empty((E, W), dtype=np.uint64)
    _load().oracle_pack(F.ctypes.data, N, E, words.ctypes.data)
    return words


def hamming(F: np.ndarray, nthreads: int | None = None) -> np.ndarray:
    """Eq. (6) G_ij = ||F_i - F_j||_1 as uint32 D[E][E]."""
    F = np.ascontiguousarray(F, dtype=np.uint8)
    E, N = F.shape
    D = np.empty((E, E), dtype=np.uint32)
    rc = _load().oracle_hamming(F.ctypes.data, N, E, D.ctypes.data, nthreads or threads())
    if rc:
        raise ValueError("oracle_hamming: bad arguments")
    return D


def loss(D: np.ndarray) -> dict:
    """Eq. (3) and statistics of the off-diagonal distances."""
    D = np.ascontiguousarray(D, dtype=np.uint32)
    E = D.shape[0]
    r = _LossResult()
    _load().oracle_loss(D.ctypes.data, E, ctypes.byref(r))
    return dict(sum=int(r.sum), sumsq=int(r.sumsq), loss=float(r.loss), mean=float(r.mean), var=float(r.var))


def surrogate(p: np.ndarray, F: np.ndarray, G: np.ndarray, k: int, scale: float = 1.0, want_grad: bool = True,
              nthreads: int | None = None):
    """Eq. (7) loss and dL/dp (G, F detached) for p of shape (N, E) (float32 or
    bf16 bit patterns), F[E][N] 0/1 and G[E][E].  Returns (loss, grad or None)."""
    p = np.ascontiguousarray(p)
    N, E = p.shape
    F = np.ascontiguousarray(F, dtype=np.uint8)
    G = np.ascontiguousarray(G, dtype=np.uint32)
    assert F.shape == (E, N) and G.shape == (E, E)
    grad = np.empty((N, E), dtype=np.float64) if want_grad else None
    loss = ctypes.c_double()
    rc = _load().oracle_surrogate(p.ctypes.data, _dtype_of(p), N, E, k, F.ctypes.data, G.ctypes.data, scale,
                                  ctypes.byref(loss), grad.ctypes.data if want_grad else None, nthreads or threads())
    if rc:
        raise ValueError(f"oracle_surrogate: bad arguments N={N} E={E} k={k}")
    return float(loss.value), grad


def surrogate_loss_blocked(p: np.ndarray, F: np.ndarray, G: np.ndarray, k: int, scale: float = 1.0,
                           block: int = 1 << 18) -> float:
    """Eq. (7) loss alone for large N: the same definition as ``surrogate``,
    with the sum over tokens inside C_ij taken by a library matrix product.
    C_ij = sum_t p_it f_it - sum_t p_it f_jt = a_i - B_ij, where a_i is the
    probability mass expert i receives from its own tokens and B = (F p)^T
    (fp64, accumulated over blocks of tokens).  Then
    loss = scale / (N^2 k) * sum_ij G_ij C_ij."""
    N, E = p.shape
    assert F.shape == (E, N) and G.shape == (E, E)
    a = np.zeros(E, dtype=np.float64)
    B = np.zeros((E, E), dtype=np.float64)
    for t0 in range(0, N, block):
        pb = np.ascontiguousarray(p[t0:t0 + block])
        pb = (pb.astype(np.uint32) << 16).view(np.float32) if pb.dtype == np.uint16 else pb
        pb = pb.astype(np.float64)
        Fb = F[:, t0:t0 + block].astype(np.float64)
        a += (pb * Fb.T).sum(axis=0)
        B += (Fb @ pb).T
    C = a[:, None] - B
    return float(scale / (float(N) * float(N) * k) * (G.astype(np.float64) * C).sum())


def load_stats(F: np.ndarray, k: int, p: np.ndarray | None = None, rank=None, R: int = 0):
    """Loads n_i, Local-LBL and MaxVio of F[E][N] (p of shape (N, E) or None;
    rank: expert -> rank list/array or None for one expert per rank).
    Returns (loads uint32[E], dict)."""
    F = np.ascontiguousarray(F, dtype=np.uint8)
    E, N = F.shape
    loads = np.empty(E, dtype=np.uint32)
    pp = None
    dt = F32
    if p is not None:
        pp = np.ascontiguousarray(p)
        assert pp.shape == (N, E)
        dt = _dtype_of(pp)
    rk = None if rank is None else np.ascontiguousarray(rank, dtype=np.int32)
    r = _LoadStatsResult()
    rc = _load().oracle_load_stats(F.ctypes.data, N, E, k, pp.ctypes.data if pp is not None else None, dt,
                                   rk.ctypes.data if rk is not None else None, R, loads.ctypes.data,
                                   ctypes.byref(r))
    if rc:
        raise ValueError(f"oracle_load_stats: bad arguments N={N} E={E} k={k} R={R}")
    return loads, dict(total=int(r.total), max_load=int(r.max_load), min_load=int(r.min_load),
                       lbl=float(r.lbl), maxvio=float(r.maxvio))


def run(scores: np.ndarray, k: int, nthreads: int | None = None):
    """Whole path for one layer: (F, words, D, loss dict)."""
    F = topk_signature(scores, k, nthreads)
    D = hamming(F, nthreads)
    return F, pack(F), D, loss(D)


def run_stream(micro_batches, k: int, nthreads: int | None = None):
    """Streaming history: the micro-batches' tokens concatenated in order, then the whole path."""
    Fs = [topk_signature(s, k, nthreads) for s in micro_batches]
    F = np.concatenate(Fs, axis=1)
    D = hamming(F, nthreads)
    return F, pack(F), D, loss(D)
