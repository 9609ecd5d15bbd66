"""Pins for the CPU oracle against what the paper and the mathematics fix.

Each check below is independent of the oracle's own code path: hand-derived
worked examples (tests/golden/), the paper's zero-sum identity (Eq. 2), the
Hamming/co-occurrence identity (App. C.3) evaluated with a numpy integer
matmul, the idle-expert property (App. C.2), library special cases (numpy's
stable argsort for Top-K), closed forms and brute force on tiny inputs.
"""
import itertools

import numpy as np
import pytest

from golden_io import load


def _zero_sum(N, E, k):
    # Eq. (2): sum over ordered pairs of ||F_i - F_j||_1 = 2 m K (n - K)
    return 2 * N * k * (E - k)


# ---------------------------------------------------------------------------
# worked examples
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["equidistant_e4_k2_n6.txt", "collapse_e4_k2_n8.txt"])
def test_golden_worked_examples(orc, name):
    g = load(name)
    F, words, D, L = orc.run(g["scores"], g["k"])
    np.testing.assert_array_equal(F, g["F"])
    np.testing.assert_array_equal(D, g["D"])
    assert L["sum"] == g["sum"] and L["sumsq"] == g["sumsq"]
    assert L["loss"] == pytest.approx(g["loss"], rel=1e-12)
    assert L["mean"] == pytest.approx(g["mean"], rel=1e-12)
    assert L["var"] == pytest.approx(g["var"], rel=1e-12, abs=1e-12)
    assert g["sum"] == _zero_sum(g["N"], g["E"], g["k"])


def test_equidistant_example_uniform_load_and_cooccurrence(orc):
    # App. C.3: at equidistance every load is mK/n and every c_ij = mK(K-1)/(n(n-1)).
    g = load("equidistant_e4_k2_n6.txt")
    F = orc.topk_signature(g["scores"], g["k"]).astype(np.int64)
    N, E, k = g["N"], g["E"], g["k"]
    C = F @ F.T
    assert np.all(np.diag(C) * E == N * k)
    off = C[~np.eye(E, dtype=bool)]
    assert np.all(off * E * (E - 1) == N * k * (k - 1))


# ---------------------------------------------------------------------------
# Top-K special cases
# ---------------------------------------------------------------------------
def _argsort_F(x, k):
    """Top-K by numpy's stable descending argsort (finite inputs only)."""
    N, E = x.shape
    idx = np.argsort(-x.astype(np.float64), axis=1, kind="stable")[:, :k]
    F = np.zeros((E, N), dtype=np.uint8)
    F[idx.T, np.arange(N)[None, :]] = 1
    return F


@pytest.mark.parametrize("E,k,N", [(8, 2, 300), (64, 6, 257), (128, 8, 130), (256, 8, 65), (5, 5, 40), (37, 1, 99)])
def test_topk_matches_stable_argsort_normal(orc, syn, E, k, N):
    x = syn.normal(11 + E, N, E, syn.F32)
    np.testing.assert_array_equal(orc.topk_signature(x, k), _argsort_F(x, k))
    xb = syn.normal(12 + E, N, E, syn.BF16)
    np.testing.assert_array_equal(orc.topk_signature(xb, k), _argsort_F(syn.bf16_bits_to_f32(xb), k))


@pytest.mark.parametrize("dtype", [0, 1])
def test_topk_matches_stable_argsort_ties(orc, syn, dtype):
    x = syn.int_ties(5, 500, 24, -3, 3, dtype)
    xf = x if dtype == 0 else syn.bf16_bits_to_f32(x)
    for k in (1, 3, 8, 23, 24):
        np.testing.assert_array_equal(orc.topk_signature(x, k), _argsort_F(xf, k))


def test_topk_signed_zero_ties(orc):
    x = np.array([[-0.0, 0.0, 0.0, -0.0]], dtype=np.float32)
    F = orc.topk_signature(x, 2)
    assert F[:, 0].tolist() == [1, 1, 0, 0]
    x = np.array([[0.0, -0.0, -1.0, -0.0]], dtype=np.float32)
    assert orc.topk_signature(x, 3)[:, 0].tolist() == [1, 1, 0, 1]


def test_topk_nan_and_inf_rules(orc):
    nan, inf = np.nan, np.inf
    x = np.array([[nan, -inf, 1.0, nan]], dtype=np.float32)
    assert orc.topk_signature(x, 1)[:, 0].tolist() == [0, 0, 1, 0]
    assert orc.topk_signature(x, 2)[:, 0].tolist() == [0, 1, 1, 0]
    # NaNs rank below -inf and tie with each other (lower index wins)
    assert orc.topk_signature(x, 3)[:, 0].tolist() == [1, 1, 1, 0]
    x = np.array([[inf, nan, inf, -inf, 0.0]], dtype=np.float32)
    assert orc.topk_signature(x, 2)[:, 0].tolist() == [1, 0, 1, 0, 0]
    assert orc.topk_signature(x, 4)[:, 0].tolist() == [1, 0, 1, 1, 1]
    # a negative NaN payload behaves like any other NaN
    bits = np.array([[0xFFC0, 0x7FC0, 0xFF80, 0x3F80]], dtype=np.uint16)  # -nan, nan, -inf, 1.0 (bf16)
    assert orc.topk_signature(bits, 2)[:, 0].tolist() == [0, 0, 1, 1]
    assert orc.topk_signature(bits, 3)[:, 0].tolist() == [1, 0, 1, 1]


def test_every_token_sets_exactly_k_bits(orc, syn):
    # Sec. 3.1.1: exactly k bits are set per token
    for dtype in (0, 1):
        x = syn.int_ties(9, 777, 19, -2, 2, dtype)
        for k in (1, 4, 19):
            F = orc.topk_signature(x, k)
            assert np.all(F.sum(axis=0) == k)


# ---------------------------------------------------------------------------
# signature packing
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("N", [1, 63, 64, 65, 200])
def test_pack_layout_lsb_first_tail_zero(orc, syn, N):
    x = syn.normal(3, N, 8, syn.F32)
    F = orc.topk_signature(x, 3)
    words = orc.pack(F)
    W = (N + 63) // 64
    assert words.shape == (8, W)
    ref = np.packbits(np.pad(F, ((0, 0), (0, W * 64 - N))), axis=1, bitorder="little").view("<u8")
    np.testing.assert_array_equal(words, ref)


# ---------------------------------------------------------------------------
# distance matrix
# ---------------------------------------------------------------------------
CASES = [(8, 2, 4096, 0), (64, 6, 3000, 1), (128, 8, 1000, 1), (256, 8, 300, 0), (7, 3, 101, 0), (3, 1, 50, 1)]


@pytest.mark.parametrize("E,k,N,dtype", CASES)
def test_distance_invariants(orc, syn, E, k, N, dtype):
    x = syn.normal(100 + E, N, E, dtype)
    F = orc.topk_signature(x, k)
    D = orc.hamming(F).astype(np.int64)
    # symmetric, zero diagonal
    assert np.array_equal(D, D.T) and np.all(np.diag(D) == 0)
    # Eq. (2) zero-sum identity
    assert D.sum() == _zero_sum(N, E, k)
    # App. C.3: ||F_i - F_j|| = ||F_i|| + ||F_j|| - 2 c_ij, with c = F F^T by integer matmul
    Fi = F.astype(np.int64)
    C = Fi @ Fi.T
    n = np.diag(C)
    np.testing.assert_array_equal(D, n[:, None] + n[None, :] - 2 * C * (1 - np.eye(E, dtype=np.int64)) - 2 * np.diag(n))
    # row sums: R_i = (E - 2k) n_i + N k (App. C.3 summed over j with sum_j c_ij = k n_i)
    np.testing.assert_array_equal(D.sum(axis=1), (E - 2 * k) * n + N * k)


def test_distance_ties_heavy(orc, syn):
    x = syn.int_ties(21, 2000, 32, 0, 4, 1)
    F = orc.topk_signature(x, 8)
    D = orc.hamming(F).astype(np.int64)
    assert D.sum() == _zero_sum(2000, 32, 8)
    Fi = F.astype(np.int64)
    C = Fi @ Fi.T
    n = np.diag(C)
    off = ~np.eye(32, dtype=bool)
    np.testing.assert_array_equal(D[off], (n[:, None] + n[None, :] - 2 * C)[off])


def test_idle_expert_rows_equal_loads(orc, syn):
    # App. C.2: an idle expert's distance to expert j equals ||F_j||_1
    N, E, k = 3000, 32, 4
    x = syn.normal(77, N, E, syn.F32)
    idle = [3, 10, 11, 30]
    x[:, idle] -= 100.0
    F = orc.topk_signature(x, k)
    D = orc.hamming(F).astype(np.int64)
    loads = F.sum(axis=1).astype(np.int64)
    assert np.all(loads[idle] == 0)
    for i in idle:
        np.testing.assert_array_equal(D[i], loads)
    assert np.all(D[np.ix_(idle, idle)] == 0)


def test_additivity_over_token_splits(orc, syn):
    x = syn.normal(5, 1000, 16, syn.F32)
    F = orc.topk_signature(x, 4)
    D = orc.hamming(F).astype(np.int64)
    D1 = orc.hamming(F[:, :377]).astype(np.int64)
    D2 = orc.hamming(F[:, 377:]).astype(np.int64)
    np.testing.assert_array_equal(D, D1 + D2)
    F_s, _, D_s, _ = orc.run_stream([x[:377], x[377:]], 4)
    np.testing.assert_array_equal(D_s, D)
    np.testing.assert_array_equal(F_s, F)


def test_complement_symmetry(orc, syn):
    # with no ties, Top-(E-k) of -s is the complement of Top-k of s, so D is equal
    x = syn.normal(8, 500, 12, syn.F32)
    F = orc.topk_signature(x, 5)
    Fc = orc.topk_signature(-x, 7)
    np.testing.assert_array_equal(F, 1 - Fc)
    np.testing.assert_array_equal(orc.hamming(F), orc.hamming(Fc))


# ---------------------------------------------------------------------------
# loss
# ---------------------------------------------------------------------------
def test_k1_closed_form(orc, syn):
    # k = 1: c_ij = 0 for i != j, so loss = 2(E-2) sum n_i^2 + 2 N^2
    N, E = 1234, 10
    x = syn.normal(4, N, E, syn.F32)
    F = orc.topk_signature(x, 1)
    n = F.sum(axis=1).astype(np.int64)
    L = orc.loss(orc.hamming(F))
    assert L["sumsq"] == 2 * (E - 2) * int((n * n).sum()) + 2 * N * N


def test_loss_exact_vs_fp64(orc, syn):
    x = syn.normal(6, 50000, 64, syn.BF16)
    F, _, D, L = orc.run(x, 6)
    d = D.astype(object)
    off = ~np.eye(64, dtype=bool)
    s2 = sum(int(v) * int(v) for v in D[off])
    assert L["sumsq"] == s2 and L["sum"] == int(D[off].astype(np.int64).sum())
    assert abs(L["loss"] - s2) <= 1e-12 * s2
    P = 64 * 63
    var_exact = (s2 * P - L["sum"] ** 2) / (P * P)
    assert L["var"] == pytest.approx(var_exact, rel=1e-10)
    assert L["mean"] == pytest.approx(L["sum"] / P, rel=1e-14)
    del d


def test_single_expert_is_all_zero(orc):
    x = np.ones((10, 1), dtype=np.float32)
    F, _, D, L = orc.run(x, 1)
    assert D.tolist() == [[0]] and L == dict(sum=0, sumsq=0, loss=0.0, mean=0.0, var=0.0)


def test_k_equals_E_gives_zero_distances(orc, syn):
    x = syn.normal(1, 100, 6, syn.F32)
    F, _, D, L = orc.run(x, 6)
    assert np.all(D == 0) and L["sumsq"] == 0


def test_exhaustive_tiny_assignments(orc):
    # Brute force over every Top-2 pattern of N=4 tokens among E=4 experts
    # (6^4 assignments): exactly-k bits, Eq. (2), symmetry, App. C.3 identity,
    # and App. C.1's equivalence of min sum-of-squares and min variance.
    E, k, N = 4, 2, 4
    pairs = list(itertools.combinations(range(E), k))
    seen = []
    for choice in itertools.product(range(len(pairs)), repeat=N):
        x = np.zeros((N, E), dtype=np.float32)
        for t, c in enumerate(choice):
            x[t, list(pairs[c])] = 1.0
        F = orc.topk_signature(x, k)
        for t, c in enumerate(choice):
            assert sorted(np.nonzero(F[:, t])[0].tolist()) == list(pairs[c])
        D = orc.hamming(F).astype(np.int64)
        assert D.sum() == _zero_sum(N, E, k) and np.array_equal(D, D.T)
        C = F.astype(np.int64) @ F.T.astype(np.int64)
        n = np.diag(C)
        off = ~np.eye(E, dtype=bool)
        assert np.array_equal(D[off], (n[:, None] + n[None, :] - 2 * C)[off])
        L = orc.loss(D)
        seen.append((L["sumsq"], L["var"]))
    s2 = np.array([a for a, _ in seen], dtype=np.float64)
    var = np.array([b for _, b in seen])
    # fixed total => variance is an increasing affine function of the sum of squares
    order = np.argsort(s2, kind="stable")
    assert np.all(np.diff(var[order]) >= -1e-12)
    assert np.argmin(s2) in set(np.nonzero(var == var.min())[0].tolist())
