"""Pins for the oracle's surrogate loss (Sec. 3.1.3, Eq. 6-7) and its gradient.

Each check is independent of the oracle's own loops:

* the gradient of the paper's DO-STE loss (Sec. 3.1.2, Eq. 5), accumulated
  here term by term from that equation, is 4x the surrogate's gradient
  (the surrogate keeps G detached, so the factor 2 of the square and the
  factor 2 of the symmetric pair sum both drop out);
* the loss is linear in p, so a finite difference equals the gradient's
  inner product with the perturbation;
* with G = 1 off the diagonal the loss has the closed form
  sum_t (E s_K(t) - k sum_i p_it) / (N^2 k), s_K(t) the selected mass;
* an idle expert's gradient is never positive (App. C.2, anti-collapse);
* the loss scales linearly with `scale`, and a worked E=2 example.

Planted mistakes in a copy of the oracle must fail these pins.
"""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle as oracle_pkg


def _setup(syn, orc, seed, N, E, k, normalize=True):
    x = syn.normal(seed, N, E, 0)
    F = orc.topk_signature(x, k)
    D = orc.hamming(F)
    p = np.exp(x.astype(np.float64))
    if normalize:
        p /= p.sum(axis=1, keepdims=True)
    return p.astype(np.float32), F, D


def _ste_gradient(p, F, G):
    """Coefficient of dp_at in Eq. (5), accumulated literally over i != j and t:
    sum_{i!=j} 2 G_ij sum_t (f_it - f_jt) (dp_it - dp_jt)."""
    N, E = p.shape
    f = F.astype(np.float64)
    g = np.zeros((N, E))
    for i in range(E):
        for j in range(E):
            if i == j:
                continue
            w = 2.0 * float(G[i, j]) * (f[i] - f[j])  # over t
            g[:, i] += w
            g[:, j] -= w
    return g


@pytest.mark.parametrize("N,E,k", [(60, 6, 2), (200, 16, 4), (96, 8, 1)])
def test_gradient_is_a_quarter_of_the_ste_gradient(syn, orc, N, E, k):
    p, F, D = _setup(syn, orc, 11 + E, N, E, k)
    _, grad = orc.surrogate(p, F, D, k)
    ste = _ste_gradient(p, F, D)
    np.testing.assert_allclose(grad * (N * N * k), ste / 4.0, rtol=1e-12, atol=1e-9)


@pytest.mark.parametrize("N,E,k", [(80, 8, 2), (150, 12, 3)])
def test_loss_is_linear_in_p(syn, orc, N, E, k):
    p, F, D = _setup(syn, orc, 21 + E, N, E, k)
    L0, grad = orc.surrogate(p, F, D, k)
    rng = np.random.default_rng(5)
    delta = (rng.standard_normal(p.shape) * 0.01).astype(np.float32)
    L1, _ = orc.surrogate((p.astype(np.float64) + delta).astype(np.float32), F, D, k, want_grad=False)
    p1 = (p.astype(np.float64) + delta).astype(np.float32).astype(np.float64)
    step = p1 - p.astype(np.float64)
    assert L1 - L0 == pytest.approx(float((step * grad).sum()), rel=1e-9, abs=1e-15)


@pytest.mark.parametrize("normalize", [True, False])
def test_closed_form_with_unit_distances(syn, orc, normalize):
    N, E, k = 120, 10, 3
    p, F, _ = _setup(syn, orc, 31, N, E, k, normalize)
    G = np.ones((E, E), np.uint32) - np.eye(E, dtype=np.uint32)
    L, _ = orc.surrogate(p, F, G, k, want_grad=False)
    pd = p.astype(np.float64)
    sK = (pd * F.T.astype(np.float64)).sum(axis=1)
    expect = (E * sK - k * pd.sum(axis=1)).sum() / (N * N * k)
    assert L == pytest.approx(expect, rel=1e-12, abs=1e-15)


def test_idle_expert_gradient_is_not_positive(syn, orc):
    N, E, k = 300, 8, 2
    x = syn.normal(41, N, E, 0)
    x[:, 5] -= 100.0  # expert 5 never selected
    F = orc.topk_signature(x, k)
    assert not F[5].any()
    D = orc.hamming(F)
    p = np.exp(x.astype(np.float64))
    p = (p / p.sum(axis=1, keepdims=True)).astype(np.float32)
    _, grad = orc.surrogate(p, F, D, k)
    assert (grad[:, 5] <= 0).all() and (grad[:, 5] < 0).any()


def test_scale_is_linear(syn, orc):
    p, F, D = _setup(syn, orc, 51, 64, 8, 2)
    L1, g1 = orc.surrogate(p, F, D, 2, scale=1.0)
    L2, g2 = orc.surrogate(p, F, D, 2, scale=0.25)
    assert L2 == pytest.approx(0.25 * L1, rel=1e-14)
    np.testing.assert_allclose(g2, 0.25 * g1, rtol=1e-14)


def test_worked_example_two_experts(orc):
    # E=2, k=1, N=2: token 0 picks expert 0, token 1 picks expert 1, so
    # G = [[0, 2], [2, 0]].  C_01 = p_00 - p_01 (t=0: f_00 - f_10 = 1; t=1: -1),
    # C_10 = -p_10 + p_11, and L = (G_01 C_01 + G_10 C_10) / (N^2 k)
    #   = 2 (p_00 - p_01 - p_10 + p_11) / 4.
    p = np.array([[0.75, 0.25], [0.5, 0.5]], np.float32)  # rows: tokens, cols: experts
    F = np.array([[1, 0], [0, 1]], np.uint8)               # F[e][t]
    G = np.array([[0, 2], [2, 0]], np.uint32)
    L, grad = orc.surrogate(p, F, G, 1)
    assert L == pytest.approx(2 * (0.75 - 0.5 - 0.25 + 0.5) / 4, rel=1e-15)
    # dL/dp_it = (1/4) sum_j G_ij (f_it - f_jt)
    expect = np.array([[2 * (1 - 0), 2 * (0 - 1)], [2 * (0 - 1), 2 * (1 - 0)]]) / 4.0
    np.testing.assert_allclose(grad, expect, rtol=1e-15)


# ---------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------
SRC = os.path.join(os.path.dirname(oracle_pkg.__file__), "doloss_oracle.c")
MUTANTS = {
    "direction_sign_flipped": (
        "score_at(p, dtype, t * E + i) * ((double)F[(int64_t)i * N + t] - (double)F[(int64_t)j * N + t]);",
        "score_at(p, dtype, t * E + i) * ((double)F[(int64_t)j * N + t] - (double)F[(int64_t)i * N + t]);"),
    "direction_uses_p_of_j": (
        "c += score_at(p, dtype, t * E + i) *", "c += score_at(p, dtype, t * E + j) *"),
    "normalisation_without_square": (
        "const double norm = scale / ((double)N * (double)N * (double)k);",
        "const double norm = scale / ((double)N * (double)k);"),
    "gradient_drops_own_term": (
        "g += (double)G[(int64_t)i * E + j] * ((double)F[(int64_t)i * N + t] - (double)F[(int64_t)j * N + t]);",
        "g += (double)G[(int64_t)i * E + j] * (0.0 - (double)F[(int64_t)j * N + t]);"),
    "gradient_sign_flipped": ("grad[t * E + i] = norm * g;", "grad[t * E + i] = -norm * g;"),
}


def _variant(tmp_path, tag, src):
    c = tmp_path / f"surr_{tag}.c"
    c.write_text(src)
    so = tmp_path / f"libsurr_{tag}.so"
    subprocess.run(["gcc", "-O1", "-fPIC", "-shared", "-fopenmp", "-std=c11", str(c), "-o", str(so), "-lm"], check=True)
    lib = ctypes.CDLL(str(so))
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    lib.oracle_surrogate.argtypes = [vp, ctypes.c_int, i64, i32, i32, vp, vp, ctypes.c_double,
                                     ctypes.POINTER(ctypes.c_double), vp, ctypes.c_int]

    def surrogate(p, F, G, k, scale=1.0):
        p = np.ascontiguousarray(p, np.float32)
        N, E = p.shape
        F = np.ascontiguousarray(F, np.uint8)
        G = np.ascontiguousarray(G, np.uint32)
        grad = np.empty((N, E))
        loss = ctypes.c_double()
        lib.oracle_surrogate(p.ctypes.data, 0, N, E, k, F.ctypes.data, G.ctypes.data, scale, ctypes.byref(loss),
                             grad.ctypes.data, 1)
        return loss.value, grad

    return surrogate


def _pins_hold(sur, syn, orc):
    try:
        N, E, k = 60, 6, 2
        p, F, D = _setup(syn, orc, 17, N, E, k)
        _, grad = sur(p, F, D, k)
        if not np.allclose(grad * (N * N * k), _ste_gradient(p, F, D) / 4.0, rtol=1e-10, atol=1e-9):
            return False
        G = np.ones((E, E), np.uint32) - np.eye(E, dtype=np.uint32)
        L, _ = sur(p, F, G, k)
        pd = p.astype(np.float64)
        sK = (pd * F.T.astype(np.float64)).sum(axis=1)
        if not np.isclose(L, (E * sK - k * pd.sum(axis=1)).sum() / (N * N * k), rtol=1e-10):
            return False
        L0, g0 = sur(p, F, D, k)
        p1 = p.copy()
        p1[3, 1] = np.float32(p[3, 1] + np.float32(0.125))
        step = float(p1[3, 1]) - float(p[3, 1])
        L1, _ = sur(p1, F, D, k)
        return bool(np.isclose(L1 - L0, step * g0[3, 1], rtol=1e-8, atol=1e-14))
    except Exception:
        return False


def test_unmutated_surrogate_passes_the_pins(syn, orc, tmp_path):
    assert _pins_hold(_variant(tmp_path, "base", open(SRC).read()), syn, orc)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_surrogate_mistake_is_caught(syn, orc, tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert old in src, name
    assert not _pins_hold(_variant(tmp_path, name, src.replace(old, new)), syn, orc), f"mutant {name} survived"


# ---------------------------------------------------------------------------
# surrogate_loss_blocked: the same Eq. (7) loss with the token sums of C taken
# by a matrix product over token blocks.  Pinned to the pins above: the worked
# E=2 example, the closed form at unit distances, and the looped oracle on
# random inputs (fp32 and bf16 p, blocks that split the tokens unevenly).
# ---------------------------------------------------------------------------
def test_blocked_loss_worked_example(orc):
    p = np.array([[0.75, 0.25], [0.5, 0.5]], np.float32)
    F = np.array([[1, 0], [0, 1]], np.uint8)
    G = np.array([[0, 2], [2, 0]], np.uint32)
    assert orc.surrogate_loss_blocked(p, F, G, 1, block=1) == pytest.approx(2 * (0.75 - 0.5 - 0.25 + 0.5) / 4,
                                                                           rel=1e-15)


def test_blocked_loss_closed_form_with_unit_distances(syn, orc):
    N, E, k = 120, 10, 3
    p, F, _ = _setup(syn, orc, 31, N, E, k)
    G = np.ones((E, E), np.uint32) - np.eye(E, dtype=np.uint32)
    pd = p.astype(np.float64)
    sK = (pd * F.T.astype(np.float64)).sum(axis=1)
    expect = (E * sK - k * pd.sum(axis=1)).sum() / (N * N * k)
    assert orc.surrogate_loss_blocked(p, F, G, k, block=37) == pytest.approx(expect, rel=1e-12, abs=1e-15)


@pytest.mark.parametrize("N,E,k,bf16,block", [(500, 16, 4, False, 64), (333, 24, 3, True, 100),
                                              (1000, 8, 2, False, 1 << 18)])
def test_blocked_loss_matches_the_looped_oracle(syn, orc, N, E, k, bf16, block):
    p, F, D = _setup(syn, orc, 61 + E, N, E, k)
    if bf16:
        p = (p.view(np.uint32) >> 16).astype(np.uint16)  # truncated bf16 patterns of the probabilities
    L, _ = orc.surrogate(p, F, D, k, scale=0.5, want_grad=False)
    assert orc.surrogate_loss_blocked(p, F, D, k, scale=0.5, block=block) == pytest.approx(L, rel=1e-11)
