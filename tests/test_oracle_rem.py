"""Pins for the REM scheduler oracle (Sec. 3.2.1 Benefit Score; App. B,
Alg. 1 replica allocation and Alg. 2 token dispatching).

* hand-worked examples (tests/golden/rem_*.txt, each with its derivation);
* the Benefit Score's cases at their boundaries, from the equation;
* properties of any run: loads and volumes are conserved, every move is
  positive and within the expert's volume, no rank takes more than D
  replicas, and an Alg. 1 move never raises the busiest rank's load nor
  lowers the idlest's, so MaxVio (App. E) never grows;
* planted mistakes in a copy of the oracle must fail these pins.
"""
import importlib.util
import os
import random

import pytest

from oracle import rem

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
SRC = rem.__file__


def load_rem(name):
    g = {"move": [], "replica": []}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            if key == "alg":
                g[key] = vals[0]
            elif key in ("move", "replica"):
                g[key].append(tuple(int(v) for v in vals))
            elif key in ("R", "D"):
                g[key] = int(vals[0])
            else:
                g[key] = [int(v) for v in vals]
    return g


GOLDEN_FILES = sorted(f for f in os.listdir(GOLDEN) if f.startswith("rem_"))


def run_golden(mod, g):
    if g["alg"] == "allocate":
        return mod.allocate(g["rank_load"], g["tokens"], g["home"], g["D"])
    return mod.dispatch(g["replica"], g["tokens"], g["home"], g["R"], g["D"])


@pytest.mark.parametrize("name", GOLDEN_FILES)
def test_worked_examples(name):
    g = load_rem(name)
    moves, L, T = run_golden(rem, g)
    assert moves == g["move"]
    assert L == g["final_load"]
    assert T == g["final_tokens"]


def test_benefit_score_cases():
    # total 30 over 3 ranks: tau = 10
    assert rem.benefit(100, 25, 4, 30, 3) == min(10 - 4, 100, 25 - 10)      # first case
    assert rem.benefit(3, 25, 4, 30, 3) == 3                                # limited by T_e
    assert rem.benefit(100, 11, 4, 30, 3) == 1                              # limited by L_s - tau
    assert rem.benefit(100, 10, 4, 30, 3) == -1                             # sender at tau, receiver below
    assert rem.benefit(100, 17, 10, 30, 3) == 3                             # receiver at tau: floor(7/2)
    assert rem.benefit(2, 17, 12, 30, 3) == 2                               # second case limited by T_e
    assert rem.benefit(100, 12, 12, 30, 3) == -1                            # sender not heavier
    assert rem.benefit(100, 9, 12, 30, 3) == -1
    # fractional tau = 31/3: 10 < tau < 11, differences rounded down
    assert rem.benefit(100, 20, 10, 31, 3) == min(0, 100, 9)               # tau - 10 = 1/3 -> 0
    assert rem.benefit(100, 20, 9, 31, 3) == min(1, 100, 9)                # 4/3 -> 1, 29/3 -> 9
    assert rem.benefit(100, 11, 9, 31, 3) == 0                             # 11 - tau = 2/3 -> 0
    assert rem.benefit(100, 10, 9, 31, 3) == -1                            # sender below tau


def _rand_case(seed):
    rng = random.Random(seed)
    R = rng.randint(2, 9)
    E = rng.randint(R, 40)
    home = [rng.randrange(R) for _ in range(E)]
    T = [int(rng.paretovariate(1.2) * 100) if rng.random() < 0.9 else 0 for _ in range(E)]
    D = rng.randint(1, 4)
    return R, E, home, T, D


def _rank_loads(T, home, R):
    L = [0] * R
    for e, t in enumerate(T):
        L[home[e]] += t
    return L


@pytest.mark.parametrize("seed", range(40))
def test_allocation_properties(seed):
    R, E, home, T0, D = _rand_case(seed)
    L0 = _rank_loads(T0, home, R)
    moves, L, T = rem.allocate(L0, T0, home, D)
    # replay the moves one at a time
    Lc, Tc, used = list(L0), list(T0), [0] * R
    mv = rem.max_violation(Lc)
    for e, r_s, r_r, d in moves:
        assert d > 0 and r_s == home[e] and r_s != r_r
        assert d <= Tc[e]
        hi, lo = max(Lc), min(Lc)
        Lc[r_r] += d
        Lc[r_s] -= d
        Tc[e] -= d
        used[r_r] += 1
        assert used[r_r] <= D
        assert max(Lc) <= hi and min(Lc) >= lo
        nv = rem.max_violation(Lc)
        assert nv <= mv + 1e-12
        mv = nv
    assert Lc == L and Tc == T
    assert sum(L) == sum(L0) and all(t >= 0 for t in T)


@pytest.mark.parametrize("seed", range(40))
def test_dispatch_properties(seed):
    R, E, home, T0, D = _rand_case(seed)
    moves, _, _ = rem.allocate(_rank_loads(T0, home, R), T0, home, D)
    rng = random.Random(1000 + seed)
    Tm = [max(0, t + rng.randint(-t // 2 - 1, t // 2 + 1)) for t in T0]  # this micro-batch's volumes
    routes, Q, T = rem.dispatch(moves, Tm, home, R, D)
    reps = {(e, r_s, r) for e, r_s, r, _ in moves}
    Qc, Tc = _rank_loads(Tm, home, R), list(Tm)
    for e, r_s, r, d in routes:
        assert (e, r_s, r) in reps and d > 0 and d <= Tc[e]
        Qc[r] += d
        Qc[r_s] -= d
        Tc[e] -= d
    assert Qc == Q and Tc == T and sum(Q) == sum(Tm)
    # at most one route per rank and pass
    assert len(routes) <= R * D


def _mutant(tmp_path, old, new):
    text = open(SRC).read()
    assert text.count(old) == 1, old
    p = tmp_path / "rem_mutant.py"
    p.write_text(text.replace(old, new))
    spec = importlib.util.spec_from_file_location("rem_mutant", p)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


MUTANTS = {
    "receiver_most_loaded": ("r_r = min(free, key=lambda r: (L[r], r))", "r_r = max(free, key=lambda r: (L[r], r))"),
    "no_floor_difference": ("return min((L_s - L_r) // 2, T_e)", "return min(L_s - L_r, T_e)"),
    "tie_to_last_expert": ("if best is None or s > best:\n                best, best_e = s, e",
                           "if best is None or s >= best:\n                best, best_e = s, e"),
    "volume_not_reduced": ("        T[best_e] -= best\n", "\n"),
    "no_slot_limit": ("free = [r for r in range(R) if used[r] < D]", "free = list(range(R))"),
    "first_case_without_sender_bound": ("return min((total - R * L_r) // R, T_e, (R * L_s - total) // R)",
                                        "return min((total - R * L_r) // R, T_e)"),
    "strict_second_case": ("if R * L_r >= total and L_s > L_r:", "if R * L_r > total and L_s > L_r:"),
    "dispatch_sorted_descending": ("for r in sorted(range(R), key=lambda r: (Q[r], r)):",
                                   "for r in sorted(range(R), key=lambda r: (-Q[r], r)):"),
    "dispatch_sender_not_updated": ("            Q[r_s] -= best\n", "\n"),
    "dispatch_single_pass": ("for _ in range(D):", "for _ in range(1):"),
}


def _pins_pass(mod):
    try:
        for name in GOLDEN_FILES:
            g = load_rem(name)
            moves, L, T = run_golden(mod, g)
            if moves != g["move"] or L != g["final_load"] or T != g["final_tokens"]:
                return False
        for seed in range(40):
            R, E, home, T0, D = _rand_case(seed)
            L0 = _rank_loads(T0, home, R)
            moves, L, T = mod.allocate(L0, T0, home, D)
            if sum(L) != sum(L0) or any(t < 0 for t in T):
                return False
            used = [0] * R
            for m in moves:
                used[m[2]] += 1
            if any(u > D for u in used):
                return False
    except AssertionError:
        return False
    return True


def test_unmutated_rem_passes_the_pins(tmp_path):
    assert _pins_pass(_mutant(tmp_path, "def benefit(", "def benefit("))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_rem_mistake_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    assert not _pins_pass(_mutant(tmp_path, old, new)), f"mutant {name} survived the pins"
