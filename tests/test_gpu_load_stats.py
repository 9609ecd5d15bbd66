"""Load statistics (per-expert loads, Local-LBL of Sec. 4.2, MaxVio of App. E)
on the GPU against the oracle, through the C ABI.

Bar: loads, total, max and min bit-exact; MaxVio within 1e-12 relative (the
GPU divides exact integers once, the oracle divides per rank); Local-LBL within
1e-9 relative (fp64 sums in a different order).
"""
import numpy as np
import pytest
import torch

from gpu_util import to_dev, units_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dl():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32398_amd as p

    p.lib()
    return p


def _probs(x, dtype):
    z = np.exp(x.astype(np.float64) - x.max(axis=1, keepdims=True))
    p = (z / z.sum(axis=1, keepdims=True)).astype(np.float32)
    if dtype == 1:
        u = p.view(np.uint32).astype(np.uint64)
        return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    return p


def _compare(got_loads, rec, ref_loads, ref, label):
    assert np.array_equal(got_loads, ref_loads), label
    assert rec["total"] == ref["total"] and rec["max_load"] == ref["max_load"] and rec["min_load"] == ref["min_load"], \
        (label, rec, ref)
    assert rec["maxvio"] == pytest.approx(ref["maxvio"], rel=1e-12, abs=1e-15), (label, rec, ref)
    assert rec["lbl"] == pytest.approx(ref["lbl"], rel=1e-9, abs=1e-300), (label, rec, ref)


CASES = [(1, 1, 1, 1), (100, 8, 2, 2), (4097, 64, 6, 1), (1000, 37, 5, 3), (777, 128, 8, 2), (3000, 256, 8, 1),
         (300, 300, 8, 1), (129, 1024, 4, 1)]


@pytest.mark.parametrize("N,E,k,L", CASES)
@pytest.mark.parametrize("with_p", [False, True])
@pytest.mark.parametrize("dtype", [0, 1])
def test_load_stats_match_oracle(dl, orc, syn, N, E, k, L, with_p, dtype):
    xs = [syn.normal(900 + 13 * E + l, N, E, 0) for l in range(L)]
    Fs = [orc.topk_signature(x, k) for x in xs]
    bits = units_dev(np.stack([orc.pack(F) for F in Fs]))
    ps = [_probs(x, dtype) for x in xs] if with_p else None
    rng = np.random.default_rng(E + N)
    R = max(1, E // 4)
    rank = rng.integers(0, R, size=E).tolist()
    for use_rank in (False, True):
        print(f"[case] load stats N={N} E={E} k={k} L={L} p={with_p} dtype={dtype} rank={use_rank}", flush=True)
        p_dev = to_dev(np.stack(ps)) if with_p else None
        loads, out = dl.do_load_stats(bits, N, k, p=p_dev, expert_rank=rank if use_rank else None, R=R)
        torch.cuda.synchronize()
        got = loads.cpu().numpy().view(np.uint32)
        recs = dl.load_stats_records(out)
        for l in range(L):
            ref_loads, ref = orc.load_stats(Fs[l], k, p=ps[l] if with_p else None,
                                            rank=rank if use_rank else None, R=R if use_rank else 0)
            _compare(got[l], recs[l], ref_loads, ref, f"layer {l}")


def test_load_stats_of_fused_signatures_and_empty_ranks(dl, orc, syn):
    # signatures written by do_fused (workload-1 shape), a placement with empty ranks
    x = syn.workload_fill(1, 0)
    k = 6
    bits, _, _ = dl.do_fused(to_dev(x), k, want_bits=True)
    rank = [i % 3 for i in range(64)]
    loads, out = dl.do_load_stats(bits, x.shape[0], k, expert_rank=rank, R=5)  # ranks 3 and 4 are empty
    torch.cuda.synchronize()
    F = orc.topk_signature(x, k)
    ref_loads, ref = orc.load_stats(F, k, rank=rank, R=5)
    _compare(loads.cpu().numpy().view(np.uint32)[0], dl.load_stats_records(out)[0], ref_loads, ref, "fused")
    assert ref["maxvio"] == 1.0  # an empty rank sits at |0 / tau - 1| = 1


def test_load_stats_of_a_stream_history(dl, orc, syn):
    # the history holds more units than ceil(N/512): ld = its padded words per expert
    E, k = 64, 6
    s = dl.DoStream(E, k, 50_000)
    mbs = [syn.normal(70 + b, n, E, 1) for b, n in enumerate([1000, 777, 4096])]
    for m in mbs:
        s.append(to_dev(m))
    N = s.tokens
    loads, out = dl.do_load_stats(None, N, k, bits_ptr=s.bits_ptr(), E=E, L=1, ld=s.words_per_expert)
    torch.cuda.synchronize()
    F = np.concatenate([orc.topk_signature(m, k) for m in mbs], axis=1)
    ref_loads, ref = orc.load_stats(F, k)
    _compare(loads.cpu().numpy().view(np.uint32)[0], dl.load_stats_records(out)[0], ref_loads, ref, "stream")
    s.close()


def test_load_stats_full_workload4_layer_against_properties(dl, orc, syn):
    # 4 Mi tokens, 256 experts: loads against the oracle's on one layer, LBL
    # against the oracle, and total = N k
    x = syn.workload_fill(4, 0)
    N, E, k = x.shape[0], x.shape[1], 8
    xd = to_dev(x)
    bits = dl.do_topk_signature(xd, k)
    loads, out = dl.do_load_stats(bits, N, k, p=xd.view(1, N, E))
    torch.cuda.synchronize()
    F = orc.topk_signature(x, k)
    ref_loads, ref = orc.load_stats(F, k, p=x)
    _compare(loads.cpu().numpy().view(np.uint32)[0], dl.load_stats_records(out)[0], ref_loads, ref, "workload 4")
    assert ref["total"] == N * k
