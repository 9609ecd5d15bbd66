"""REM scheduling on the GPU (do_rem_allocate: App. B, Alg. 1; do_rem_dispatch:
App. B, Alg. 2; Benefit Score of Sec. 3.2.1) against the oracle in
oracle/rem.py, move by move: the hand-worked fixtures, random problems of
many shapes (several layers per call, up to 1024 experts and ranks), loads
measured from GPU signatures of a Zipf-popular score stream, and the
device-side rejection of invalid volumes and assignments.
"""
import random

import numpy as np
import pytest
import torch

from oracle import rem
from test_oracle_rem import GOLDEN_FILES, load_rem

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dl():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32398_amd as p

    p.lib()
    return p


def pack_moves(layers, S):
    """Host lists of (e, src, dst, tokens) -> int64 [L, S, 3] records and counts."""
    rec = np.zeros((len(layers), S, 3), dtype=np.int64)
    for l, moves in enumerate(layers):
        for i, (e, rs, rd, t) in enumerate(moves):
            rec[l, i] = (e | (rs << 32), rd, t)
    n = torch.tensor([len(m) for m in layers], dtype=torch.int32, device="cuda")
    return torch.from_numpy(rec).cuda(), n


def dev64(rows):
    return torch.tensor(rows, dtype=torch.int64, device="cuda")


@pytest.mark.parametrize("name", GOLDEN_FILES)
def test_worked_examples_on_the_gpu(dl, name):
    g = load_rem(name)
    R, D, home = g["R"] if "R" in g else len(g["rank_load"]), g["D"], g["home"]
    if g["alg"] == "allocate":
        m, n, lo, to = dl.do_rem_allocate(dev64([g["tokens"]]), home, R, D, rank_load=dev64([g["rank_load"]]))
    else:
        reps, nr = pack_moves([[(e, rs, rd, 0) for e, rs, rd in g["replica"]]], max(1, len(g["replica"])))
        m, n, lo, to = dl.do_rem_dispatch(reps, nr, dev64([g["tokens"]]), home, R, D)
    torch.cuda.synchronize()
    assert dl.rem_records(m, n)[0] == g["move"]
    assert lo[0].tolist() == g["final_load"] and to[0].tolist() == g["final_tokens"]


def _problem(seed, E, R, L, given_loads):
    rng = random.Random(seed)
    home = [rng.randrange(R) for _ in range(E)]
    T = [[int(rng.paretovariate(1.1) * 1000) if rng.random() < 0.95 else 0 for _ in range(E)] for _ in range(L)]
    if given_loads:  # historical loads differ from this batch's volumes (a moving average)
        Ld = []
        for l in range(L):
            base = [0] * R
            for e in range(E):
                base[home[e]] += T[l][e]
            Ld.append([max(0, b + rng.randint(-b // 4 - 1, b // 4 + 1)) for b in base])
    else:
        Ld = None
    return home, T, Ld


@pytest.mark.parametrize("E,R,D,L,given", [(8, 2, 1, 3, False), (64, 8, 2, 4, False), (128, 8, 2, 5, True),
                                           (256, 16, 4, 2, False), (37, 5, 3, 3, True), (1024, 64, 4, 2, False),
                                           (1024, 1024, 4, 1, False), (300, 1000, 1, 2, True), (16, 4, 64, 2, False)])
def test_allocate_and_dispatch_match_the_oracle(dl, E, R, D, L, given):
    print(f"[case] rem E={E} R={R} D={D} L={L} given={given}", flush=True)
    home, T, Ld = _problem(E * 1000 + R * 10 + D, E, R, L, given)
    m, n, lo, to = dl.do_rem_allocate(dev64(T), home, R, D, rank_load=dev64(Ld) if given else None)
    torch.cuda.synchronize()
    got = dl.rem_records(m, n)
    refs = []
    for l in range(L):
        base = Ld[l] if given else [sum(T[l][e] for e in range(E) if home[e] == r) for r in range(R)]
        ref_moves, ref_L, ref_T = rem.allocate(base, T[l], home, D)
        refs.append(ref_moves)
        assert got[l] == ref_moves, f"layer {l}: placements differ"
        assert lo[l].tolist() == ref_L and to[l].tolist() == ref_T, f"layer {l}: loads after placement differ"
    # the next micro-batch's volumes, routed through those replicas
    rng = random.Random(7 + E)
    Tm = [[max(0, t + rng.randint(-t // 3 - 1, t // 3 + 1)) for t in row] for row in T]
    r2, n2, qo, to2 = dl.do_rem_dispatch(m, n, dev64(Tm), home, R, D)
    torch.cuda.synchronize()
    got2 = dl.rem_records(r2, n2)
    for l in range(L):
        ref_routes, ref_Q, ref_T = rem.dispatch(refs[l], Tm[l], home, R, D)
        assert got2[l] == ref_routes, f"layer {l}: routes differ"
        assert qo[l].tolist() == ref_Q and to2[l].tolist() == ref_T, f"layer {l}: queues differ"


def test_rem_on_loads_of_gpu_signatures(dl, orc, syn):
    # loads of a Zipf-popular bf16 score stream (128 experts, top-8), measured
    # from the GPU's signatures, placed on 8 ranks of 16 consecutive experts
    E, k, N, R, D = 128, 8, 65_536, 8, 2
    w = syn.WORKLOADS[3]
    xs = [syn.workload_fill(3, b) for b in range(2)]
    loads = []
    for x in xs:
        t = torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()
        bits = dl.do_topk_signature(t, k)
        ld, _ = dl.do_load_stats(bits, N, k)
        torch.cuda.synchronize()
        loads.append(ld[0].long())
        assert ld[0].cpu().numpy().astype(np.int64).tolist() == orc.topk_signature(x, k).sum(axis=1).tolist()
    home = [e * R // E for e in range(E)]
    m, n, lo, to = dl.do_rem_allocate(loads[0].unsqueeze(0).contiguous(), home, R, D)
    r2, n2, qo, _ = dl.do_rem_dispatch(m, n, loads[1].unsqueeze(0).contiguous(), home, R, D)
    torch.cuda.synchronize()
    T0, T1 = loads[0].tolist(), loads[1].tolist()
    base = [sum(T0[e] for e in range(E) if home[e] == r) for r in range(R)]
    ref_moves, ref_L, _ = rem.allocate(base, T0, home, D)
    assert dl.rem_records(m, n)[0] == ref_moves and lo[0].tolist() == ref_L
    ref_routes, ref_Q, _ = rem.dispatch(ref_moves, T1, home, R, D)
    assert dl.rem_records(r2, n2)[0] == ref_routes and qo[0].tolist() == ref_Q
    # the placement balances the skewed loads: MaxVio (App. E) falls
    assert rem.max_violation(ref_L) < rem.max_violation(base)
    assert w["E"] == E


def test_invalid_inputs_fail_only_their_layer(dl):
    home = [0, 0, 1, 1]
    T = [[5, 6, 1, 0], [5, -1, 1, 0], [5, 1 << 40, 1, 0]]
    m, n, _, _ = dl.do_rem_allocate(dev64(T), home, 2, 1)
    torch.cuda.synchronize()
    recs = dl.rem_records(m, n)
    assert recs[0] == rem.allocate([11, 1], T[0], home, 1)[0]
    assert recs[1] is None and recs[2] is None
    # a replica whose source is not its expert's home rank
    reps, nr = pack_moves([[(0, 0, 1, 0)], [(0, 1, 1, 0)]], 1)
    r2, n2, _, _ = dl.do_rem_dispatch(reps, nr, dev64([T[0], T[0]]), home, 2, 1)
    torch.cuda.synchronize()
    got = dl.rem_records(r2, n2)
    assert got[0] == rem.dispatch([(0, 0, 1)], T[0], home, 2, 1)[0] and got[1] is None
