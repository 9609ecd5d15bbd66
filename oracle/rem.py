"""REM scheduler oracle -- TEST INFRASTRUCTURE ONLY.

Plain Python (exact integers) of the Replica Expert Mechanism's two greedy
steps (arXiv 2609.32398, Sec. 3.2.1 and App. B):

* ``benefit``   -- the Benefit Score S(e, r_s, r_r, tau) of the Benefit Score
  equation (Sec. 3.2.1).
* ``allocate``  -- global-batch replica allocation (App. B, Alg. 1): while
  some rank has a free replica slot, the least-loaded such rank receives a
  replica of the expert with the largest benefit, and the loads move.
* ``dispatch``  -- micro-batch token dispatching (App. B, Alg. 2): D passes;
  each pass orders the ranks by queue depth and lets every rank, lightest
  first, pull tokens through its best replica.

Readings where the paper leaves a choice open (each one is listed in the
design notes):

* tau, the mean load, is a rational number; comparisons with it are made
  exactly (R * L against the total) and the two differences tau - L_r and
  L_s - tau are rounded down to whole tokens;
* an expert's tokens are sent from its home rank (the rank the expert is
  placed on), so the pair (e, r_s) of Alg. 1 is (e, home(e)) with
  home(e) != r_r;
* ties: the least-loaded receiver with the lowest rank index; the largest
  benefit with the lowest expert index (Alg. 1) or the earliest replica in
  the assignment (Alg. 2); Alg. 2 sorts the ranks by queue depth, ties by
  rank index;
* Alg. 2 records and applies a move only when its benefit is positive (the
  listing applies Delta unconditionally, which for Delta = -1 would move a
  token backwards);
* tau stays as computed at the start (moves keep the total unchanged).

It shares no code with the HIP library.
"""
from __future__ import annotations


def benefit(T_e: int, L_s: int, L_r: int, total: int, R: int) -> int:
    """Benefit Score S(e, r_s, r_r, tau), tau = total / R (Sec. 3.2.1)."""
    if R * L_r < total and R * L_s > total:  # L_r < tau < L_s
        return min((total - R * L_r) // R, T_e, (R * L_s - total) // R)
    if R * L_r >= total and L_s > L_r:       # L_r >= tau, sender heavier
        return min((L_s - L_r) // 2, T_e)
    return -1


def allocate(rank_load, expert_tokens, home, D: int):
    """Alg. 1.  rank_load: historical loads L_r (R ints); expert_tokens: T_e
    (E ints); home: home rank of each expert; D: replica slots per rank.
    Returns (moves, L, T): moves = [(e, r_s, r_r, Delta), ...] in order, and
    the loads and token volumes after the last move."""
    L = [int(v) for v in rank_load]
    T = [int(v) for v in expert_tokens]
    R, E = len(L), len(T)
    total = sum(L)
    used = [0] * R
    moves = []
    while True:
        free = [r for r in range(R) if used[r] < D]
        if not free:
            break  # every rank is full
        r_r = min(free, key=lambda r: (L[r], r))
        best, best_e = None, None
        for e in range(E):
            r_s = home[e]
            if r_s == r_r:
                continue
            s = benefit(T[e], L[r_s], L[r_r], total, R)
            if best is None or s > best:
                best, best_e = s, e
        if best is None or best <= 0:
            break
        r_s = home[best_e]
        moves.append((best_e, r_s, r_r, best))
        used[r_r] += 1
        L[r_r] += best
        L[r_s] -= best
        T[best_e] -= best
    return moves, L, T


def dispatch(assignment, expert_tokens, home, R: int, D: int):
    """Alg. 2.  assignment: replicas (e, r_s, r, ...) as allocate returns them
    (only the first three fields are used); expert_tokens: this micro-batch's
    T_e; home: home rank of each expert; R ranks, D passes.
    Returns (routes, Q, T): routes = [(e, r_s, r, Delta), ...] in order (Delta
    tokens of expert e go from its home r_s to its replica on rank r), and the
    queue depths and remaining volumes after the last pass."""
    T = [int(v) for v in expert_tokens]
    Q = [0] * R
    for e, t in enumerate(T):
        Q[home[e]] += t
    total = sum(Q)
    routes = []
    for _ in range(D):
        for r in sorted(range(R), key=lambda r: (Q[r], r)):
            best, pick = None, None
            for rep in assignment:
                e, r_s, r_dst = rep[0], rep[1], rep[2]
                if r_dst != r:
                    continue
                s = benefit(T[e], Q[r_s], Q[r], total, R)
                if best is None or s > best:
                    best, pick = s, (e, r_s)
            if best is None or best <= 0:
                continue
            e, r_s = pick
            routes.append((e, r_s, r, best))
            Q[r] += best
            Q[r_s] -= best
            T[e] -= best
    return routes, Q, T


def max_violation(loads) -> float:
    """MaxVio (App. E) of rank loads: max_r |L_r / tau - 1|, 0 when tau is 0."""
    R = len(loads)
    tau = sum(loads) / R
    if tau == 0:
        return 0.0
    return max(abs(l / tau - 1.0) for l in loads)
