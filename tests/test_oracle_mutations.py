"""Planted mistakes in the oracle must be caught by its pins.

Each mutant is a copy of oracle/doloss_oracle.c with one plausible mistake
(a reversed tie rule, a dropped term, a wrong index, a wrong bit order ...),
compiled on the CPU into a temporary library.  The pins used here are the
same independent facts as in test_oracle_pins.py: the worked examples,
numpy's stable argsort, Eq. (2), the App. C.3 identity and exact integer
sums.  A mutant that survives them all fails this test.
"""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle as oracle_pkg
from golden_io import load

SRC = os.path.join(os.path.dirname(oracle_pkg.__file__), "doloss_oracle.c")

MUTANTS = {
    "tie_to_higher_index": ("  return a < b; /* equal values", "  return a > b; /* equal values"),
    "nan_ranks_first": ("  if (na) return 0;\n  if (nb) return 1;", "  if (na) return 1;\n  if (nb) return 0;"),
    "strict_order_flipped": ("  if (va > vb) return 1;\n  if (va < vb) return 0;", "  if (va < vb) return 1;\n  if (va > vb) return 0;"),
    "one_fewer_pick": ("for (int32_t r = 0; r < k; ++r)", "for (int32_t r = 1; r < k; ++r)"),
    "bf16_wrong_shift": ("(uint32_t)((const uint16_t*)scores)[idx] << 16", "(uint32_t)((const uint16_t*)scores)[idx] << 15"),
    "pack_msb_first": ("(uint64_t)1 << (t % 64)", "(uint64_t)1 << (63 - t % 64)"),
    "hamming_and_not_xor": ("d += (uint64_t)(fi[t] != fj[t]);", "d += (uint64_t)(fi[t] & fj[t]);"),
    "hamming_wrong_row": ("const uint8_t* fj = F + (int64_t)j * N;", "const uint8_t* fj = F + (int64_t)i * N;"),
    "loss_not_squared": ("f2 += (double)d * (double)d;", "f2 += (double)d;"),
    "var_wrong_divisor": ("out->var = acc / P;", "out->var = acc / (P - 1.0);"),
    "mean_wrong": ("double mean = f1 / P;", "double mean = f1 / (double)E;"),
}


class _Res(ctypes.Structure):
    _fields_ = [("sum", ctypes.c_uint64), ("sumsq", ctypes.c_uint64), ("loss", ctypes.c_double),
                ("mean", ctypes.c_double), ("var", ctypes.c_double)]


class _Oracle:
    """Minimal binding of a compiled oracle variant."""

    def __init__(self, path):
        lib = ctypes.CDLL(path)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        lib.oracle_topk_signature.argtypes = [vp, ctypes.c_int, i64, i32, i32, vp, ctypes.c_int]
        lib.oracle_pack.argtypes = [vp, i64, i32, vp]
        lib.oracle_hamming.argtypes = [vp, i64, i32, vp, ctypes.c_int]
        lib.oracle_loss.argtypes = [vp, i32, ctypes.POINTER(_Res)]
        self.lib = lib

    def topk(self, x, k):
        x = np.ascontiguousarray(x)
        N, E = x.shape
        F = np.empty((E, N), np.uint8)
        self.lib.oracle_topk_signature(x.ctypes.data, 0 if x.dtype == np.float32 else 1, N, E, k, F.ctypes.data, 1)
        return F

    def pack(self, F):
        E, N = F.shape
        w = np.empty((E, (N + 63) // 64), np.uint64)
        self.lib.oracle_pack(np.ascontiguousarray(F).ctypes.data, N, E, w.ctypes.data)
        return w

    def hamming(self, F):
        E, N = F.shape
        D = np.empty((E, E), np.uint32)
        self.lib.oracle_hamming(np.ascontiguousarray(F).ctypes.data, N, E, D.ctypes.data, 1)
        return D

    def loss(self, D):
        r = _Res()
        self.lib.oracle_loss(np.ascontiguousarray(D, dtype=np.uint32).ctypes.data, D.shape[0], ctypes.byref(r))
        return dict(sum=r.sum, sumsq=r.sumsq, loss=r.loss, mean=r.mean, var=r.var)


def _pins_hold(o, syn) -> bool:
    """True iff every pin holds for oracle variant `o`."""
    for name in ("equidistant_e4_k2_n6.txt", "collapse_e4_k2_n8.txt"):
        g = load(name)
        F = o.topk(g["scores"], g["k"])
        D = o.hamming(F)
        L = o.loss(D)
        if not (np.array_equal(F, g["F"]) and np.array_equal(D, g["D"])):
            return False
        if L["sum"] != g["sum"] or L["sumsq"] != g["sumsq"]:
            return False
        if abs(L["loss"] - g["loss"]) > 1e-9 or abs(L["mean"] - g["mean"]) > 1e-9 or abs(L["var"] - g["var"]) > 1e-9:
            return False
    # NaN rule (hand case) and stable argsort on tie-heavy bf16 inputs
    xn = np.array([[np.nan, -np.inf, 1.0, np.nan]], np.float32)
    if o.topk(xn, 2)[:, 0].tolist() != [0, 1, 1, 0]:
        return False
    xb = syn.int_ties(5, 300, 12, -2, 2, 1)
    xf = syn.bf16_bits_to_f32(xb).astype(np.float64)
    idx = np.argsort(-xf, axis=1, kind="stable")[:, :3]
    Fr = np.zeros((12, 300), np.uint8)
    Fr[idx.T, np.arange(300)[None, :]] = 1
    F = o.topk(xb, 3)
    if not np.array_equal(F, Fr):
        return False
    w = o.pack(F)
    ref = np.packbits(np.pad(F, ((0, 0), (0, 320 - 300))), axis=1, bitorder="little").view("<u8")
    if not np.array_equal(w, ref):
        return False
    D = o.hamming(F).astype(np.int64)
    if D.sum() != 2 * 300 * 3 * 9:
        return False
    C = F.astype(np.int64) @ F.T.astype(np.int64)
    n = np.diag(C)
    off = ~np.eye(12, dtype=bool)
    if not np.array_equal(D[off], (n[:, None] + n[None, :] - 2 * C)[off]):
        return False
    L = o.loss(D)
    P = 12 * 11
    s1 = int(D[off].sum())
    s2 = int((D[off] ** 2).sum())
    return (L["sum"] == s1 and L["sumsq"] == s2 and abs(L["mean"] - s1 / P) < 1e-9
            and abs(L["var"] - (s2 * P - s1 * s1) / P / P) < 1e-6)


def _compile(src_text, tmp_path, tag):
    c = tmp_path / f"oracle_{tag}.c"
    so = tmp_path / f"liboracle_{tag}.so"
    c.write_text(src_text)
    subprocess.run(["gcc", "-O1", "-fPIC", "-shared", "-std=c11", str(c), "-o", str(so), "-lm"], check=True)
    return str(so)


def test_unmutated_oracle_passes_the_pins(syn, tmp_path):
    src = open(SRC).read()
    assert _pins_hold(_Oracle(_compile(src, tmp_path, "orig")), syn)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(syn, tmp_path, name):
    src = open(SRC).read()
    old, new = MUTANTS[name]
    assert old in src, f"mutation anchor for {name} not found"
    assert not _pins_hold(_Oracle(_compile(src.replace(old, new, 1), tmp_path, name)), syn)
