"""Pins for the oracle's load statistics: per-expert loads (App. C.3), the
Local-LBL loss of Sec. 4.2 and MaxVio (App. E).

Each check is independent of the oracle's own loops:

* the loads sum to N k (every token sets exactly k bits, Eq. 1-2);
* the loads follow from the oracle's distance matrix alone through the row-sum
  identity R_i = (E - 2k) n_i + N k (App. C.3 with Eq. 2), a different route
  (XOR counts) from the one the oracle takes;
* the equidistant fixture (App. C.3: ||F_i||_1 = N k / E) and the collapse
  fixture give the loads, Local-LBL and MaxVio worked out by hand below;
* MaxVio of App. E's own example: the busiest rank 10 % above the mean reads 0.1;
* Local-LBL closed forms: uniform probabilities give 1/E; with k = 1 and the
  probabilities equal to the assignments it is sum_i (n_i / N)^2.

Planted mistakes in a copy of the oracle must fail these pins.
"""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle as oracle_pkg
from golden_io import load as load_golden


def _case(syn, orc, seed, N, E, k):
    x = syn.normal(seed, N, E, 0)
    return x, orc.topk_signature(x, k)


@pytest.mark.parametrize("N,E,k", [(1, 1, 1), (37, 5, 2), (500, 16, 3), (1000, 64, 8), (257, 130, 7)])
def test_loads_sum_to_N_k(syn, orc, N, E, k):
    _, F = _case(syn, orc, 3 + N, N, E, k)
    loads, st = orc.load_stats(F, k)
    assert int(loads.astype(np.int64).sum()) == N * k == st["total"]
    assert st["max_load"] == loads.max() and st["min_load"] == loads.min()


@pytest.mark.parametrize("N,E,k", [(300, 8, 2), (777, 32, 5), (1000, 64, 8), (640, 128, 8)])
def test_loads_from_the_distance_row_sums(syn, orc, N, E, k):
    # App. C.3: D_ij = n_i + n_j - 2 c_ij; with Eq. 2 the row sums are
    # R_i = (E - 2k) n_i + N k, so n_i follows from D whenever E != 2k.
    _, F = _case(syn, orc, 11 + E, N, E, k)
    D = orc.hamming(F).astype(np.int64)
    n_from_D = (D.sum(axis=1) - N * k) // (E - 2 * k)
    assert np.array_equal((D.sum(axis=1) - N * k) % (E - 2 * k), np.zeros(E, np.int64))
    loads, _ = orc.load_stats(F, k)
    assert np.array_equal(loads.astype(np.int64), n_from_D)


def test_equidistant_fixture():
    # App. C.3: at equidistance every load is N k / E = 6 * 2 / 4 = 3, so
    # every placement of two experts per rank has L_r = 6 = tau and MaxVio 0;
    # with p uniform (1/4) Local-LBL = sum_i (3/12) (1/4) = 1/4.
    g = load_golden("equidistant_e4_k2_n6.txt")
    loads, st = oracle_pkg.load_stats(g["F"], g["k"], p=np.full((6, 4), 0.25, np.float32), rank=[1, 0, 0, 1], R=2)
    assert loads.tolist() == [3, 3, 3, 3]
    assert st["maxvio"] == 0.0 and st["lbl"] == 0.25 and st["total"] == 12


def test_collapse_fixture():
    # All tokens pick experts 0 and 1 (N = 8, k = 2): loads 8, 8, 0, 0.
    # One expert per rank: tau = 16 / 4 = 4, |8/4 - 1| = |0/4 - 1| = 1, MaxVio 1.
    # Ranks {0, 2} and {1, 3}: L = 8, 8, MaxVio 0.  Ranks {0, 1} and {2, 3}:
    # L = 16, 0, tau 8, MaxVio 1.  Local-LBL with p = 1/2 on experts 0 and 1 and
    # 0 elsewhere: f = (1/2, 1/2, 0, 0), P = (1/2, 1/2, 0, 0), sum 1/2.
    g = load_golden("collapse_e4_k2_n8.txt")
    F = g["F"]
    loads, st = oracle_pkg.load_stats(F, 2)
    assert loads.tolist() == [8, 8, 0, 0] and st["maxvio"] == 1.0
    assert oracle_pkg.load_stats(F, 2, rank=[0, 1, 0, 1], R=2)[1]["maxvio"] == 0.0
    assert oracle_pkg.load_stats(F, 2, rank=[0, 0, 1, 1], R=2)[1]["maxvio"] == 1.0
    p = np.tile(np.array([0.5, 0.5, 0.0, 0.0], np.float32), (8, 1))
    assert oracle_pkg.load_stats(F, 2, p=p)[1]["lbl"] == 0.5


def test_maxvio_example_of_the_appendix():
    # App. E: "a MaxVio value of 0.1" means the busiest rank carries 10 % more
    # tokens than the ideal average.  Four ranks of one expert each with loads
    # 11, 10, 10, 9 (mean 10): MaxVio = 11/10 - 1 = 0.1 (the lightest rank is
    # 0.1 below, which ties).
    N, E, k = 40, 4, 1
    F = np.zeros((E, N), np.uint8)
    start = 0
    for e, n in enumerate([11, 10, 10, 9]):
        F[e, start:start + n] = 1
        start += n
    _, st = oracle_pkg.load_stats(F, k)
    assert st["maxvio"] == pytest.approx(0.1, abs=1e-15)
    # a rank with 13 of 40 (mean 10): 0.3
    F2 = np.zeros((E, N), np.uint8)
    start = 0
    for e, n in enumerate([13, 9, 9, 9]):
        F2[e, start:start + n] = 1
        start += n
    assert oracle_pkg.load_stats(F2, k)[1]["maxvio"] == pytest.approx(0.3, abs=1e-15)
    # the definition takes |.|: an almost idle rank (2 of mean 10) reads 0.8,
    # more than the busiest one (13: 0.3)
    F3 = np.zeros((E, N), np.uint8)
    start = 0
    for e, n in enumerate([2, 12, 13, 13]):
        F3[e, start:start + n] = 1
        start += n
    assert oracle_pkg.load_stats(F3, k)[1]["maxvio"] == pytest.approx(0.8, abs=1e-15)


@pytest.mark.parametrize("N,E,k", [(200, 8, 2), (513, 64, 6)])
def test_lbl_uniform_probabilities(syn, orc, N, E, k):
    _, F = _case(syn, orc, 5 + E, N, E, k)
    p = np.full((N, E), 1.0 / E, np.float32)
    _, st = orc.load_stats(F, k, p=p)
    # sum_i f_i = 1, so sum_i f_i P_i = P = float32(1/E)
    assert st["lbl"] == pytest.approx(float(np.float32(1.0 / E)), rel=1e-12)


def test_lbl_top1_with_probabilities_equal_to_assignments(syn, orc):
    N, E, k = 999, 16, 1
    _, F = _case(syn, orc, 21, N, E, k)
    loads, st = orc.load_stats(F, k, p=F.T.astype(np.float32))
    assert st["lbl"] == pytest.approx(float(((loads / N) ** 2).sum()), rel=1e-12)


def test_bad_rank_is_rejected(orc):
    F = np.ones((2, 3), np.uint8)
    with pytest.raises(ValueError):
        orc.load_stats(F, 2, rank=[0, 2], R=2)


# ---------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------
SRC = os.path.join(os.path.dirname(oracle_pkg.__file__), "doloss_oracle.c")
MUTANTS = {
    "fraction_without_k": ("const double f = (double)loads[i] / ((double)N * (double)k);",
                           "const double f = (double)loads[i] / (double)N;"),
    "mean_probability_not_divided": ("      P /= (double)N;\n", "\n"),
    "maxvio_without_abs": ("const double v = fabs(Lr[r] / tau - 1.0);", "const double v = Lr[r] / tau - 1.0;"),
    "tau_is_the_sum": ("  tau /= (double)R;\n", "\n"),
    "load_counts_wrong_row": ("for (int64_t t = 0; t < N; ++t) n += F[(int64_t)i * N + t];",
                              "for (int64_t t = 0; t < N; ++t) n += F[(int64_t)((i + 1) % E) * N + t];"),
}


class _Res(ctypes.Structure):
    _fields_ = [("total", ctypes.c_uint64), ("max_load", ctypes.c_uint32), ("min_load", ctypes.c_uint32),
                ("lbl", ctypes.c_double), ("maxvio", ctypes.c_double)]


def _variant(tmp_path, tag, src):
    c = tmp_path / f"ls_{tag}.c"
    c.write_text(src)
    so = tmp_path / f"libls_{tag}.so"
    subprocess.run(["gcc", "-O1", "-fPIC", "-shared", "-fopenmp", "-std=c11", str(c), "-o", str(so), "-lm"], check=True)
    lib = ctypes.CDLL(str(so))
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    lib.oracle_load_stats.argtypes = [vp, i64, i32, i32, vp, ctypes.c_int, vp, i32, vp, ctypes.POINTER(_Res)]

    def stats(F, k, p=None, rank=None, R=0):
        F = np.ascontiguousarray(F, np.uint8)
        E, N = F.shape
        loads = np.empty(E, np.uint32)
        pp = None if p is None else np.ascontiguousarray(p, np.float32)
        rk = None if rank is None else np.ascontiguousarray(rank, np.int32)
        r = _Res()
        rc = lib.oracle_load_stats(F.ctypes.data, N, E, k, pp.ctypes.data if pp is not None else None, 0,
                                   rk.ctypes.data if rk is not None else None, R, loads.ctypes.data, ctypes.byref(r))
        if rc:
            raise ValueError(rc)
        return loads, dict(total=r.total, lbl=r.lbl, maxvio=r.maxvio)

    return stats


def _pins_hold(stats, syn, orc):
    try:
        N, E, k = 300, 8, 3
        x = syn.normal(31, N, E, 0)
        F = orc.topk_signature(x, k)
        D = orc.hamming(F).astype(np.int64)
        loads, st = stats(F, k)
        if st["total"] != N * k or not np.array_equal(loads.astype(np.int64), (D.sum(axis=1) - N * k) // (E - 2 * k)):
            return False
        g = load_golden("collapse_e4_k2_n8.txt")
        if stats(g["F"], 2)[1]["maxvio"] != 1.0 or stats(g["F"], 2, rank=[0, 0, 1, 1], R=2)[1]["maxvio"] != 1.0:
            return False
        Fm = np.zeros((4, 40), np.uint8)
        start = 0
        for e, n in enumerate([9, 10, 10, 11]):
            Fm[e, start:start + n] = 1
            start += n
        if abs(stats(Fm, 1)[1]["maxvio"] - 0.1) > 1e-12:
            return False
        Fl = np.zeros((4, 40), np.uint8)
        start = 0
        for e, n in enumerate([2, 12, 13, 13]):
            Fl[e, start:start + n] = 1
            start += n
        if abs(stats(Fl, 1)[1]["maxvio"] - 0.8) > 1e-12:
            return False
        p = np.full((N, E), 1.0 / E, np.float32)
        if abs(stats(F, k, p=p)[1]["lbl"] - float(np.float32(1.0 / E))) > 1e-12:
            return False
        return True
    except Exception:
        return False


def test_unmutated_load_stats_pass_the_pins(syn, orc, tmp_path):
    assert _pins_hold(_variant(tmp_path, "base", open(SRC).read()), syn, orc)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_load_stats_mistake_is_caught(syn, orc, tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert old in src, name
    assert not _pins_hold(_variant(tmp_path, name, src.replace(old, new)), syn, orc), f"mutant {name} survived"
