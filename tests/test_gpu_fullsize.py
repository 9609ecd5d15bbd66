"""The large workloads at their full sizes, in the launch configuration the
benchmark times (one do_fused call over all layers with signatures written;
the stream as reset + one append_many of all micro-batches + finalize).

Workloads 2, 3 and 4 are compared with the oracle element by element in full
(every layer: signatures, distances, loss record).  The surrogate loss
(Eq. 7) on workload 4 is compared with the oracle's loss on every layer, and
sampled gradients with the oracle's gradient.  Every unit schedule the
library can choose and both Gram kinds are run at full size and must give
bit-identical results; so must repeated calls while the schedule tuner
measures its candidates.
"""
import time

import numpy as np
import pytest
import torch

from gpu_util import D_np, bits_at, bits_np, check_invariants, loss_close, to_dev, upload_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dl():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32398_amd as p

    p.lib()
    return p


def _same_results(dl, scores, k, ref, label):
    """do_fused into fresh buffers must equal the oracle-checked `ref` bit for bit."""
    bits, D, out = dl.do_fused(scores, k, want_bits=True)
    torch.cuda.synchronize()
    assert torch.equal(bits, ref[0]), f"{label}: signatures differ"
    assert torch.equal(D, ref[1]), f"{label}: distances differ"
    assert torch.equal(out, ref[2]), f"{label}: loss records differ"


def _schedules_and_grams_agree(dl, scores, k, ref, name):
    """Both fixed unit schedules, the popcount Gram, and eight calls with the
    run-time choice (from 100 ms after a shape's first launch the schedule
    tuner measures each candidate three times, then keeps one) all reproduce
    `ref`."""
    try:
        for opt, val, label in ((dl.DO_OPT_SCHEDULE, 0, "XCD-partitioned schedule"),
                                (dl.DO_OPT_SCHEDULE, 1, "contiguous schedule")):
            dl.set_option(opt, val)
            print(f"[case] {name}: {label}", flush=True)
            _same_results(dl, scores, k, ref, f"{name} {label}")
        dl.set_option(dl.DO_OPT_SCHEDULE, -1)
        dl.set_option(dl.DO_OPT_GRAM, 1)
        print(f"[case] {name}: popcount Gram", flush=True)
        _same_results(dl, scores, k, ref, f"{name} popcount Gram")
        dl.set_option(dl.DO_OPT_GRAM, 0)
        time.sleep(0.15)  # the tuner measures from 100 ms after a shape's first launch
        for rep in range(8):
            print(f"[case] {name}: tuned call {rep}", flush=True)
            _same_results(dl, scores, k, ref, f"{name} tuned call {rep}")
    finally:
        dl.set_option(dl.DO_OPT_SCHEDULE, -1)
        dl.set_option(dl.DO_OPT_GRAM, 0)


def test_workload2_full(dl, orc, syn):
    w = syn.WORKLOADS[2]
    L, N, E, k = w["layers"], w["n"], w["E"], w["k"]
    print(f"[case] {w['name']} full, L={L} N={N} E={E} k={k}", flush=True)
    scores, _ = upload_workload(syn, 2, L)
    bits, D, out = dl.do_fused(scores, k, want_bits=True)
    torch.cuda.synchronize()
    got_bits, got_D, recs = bits_np(bits, N), D_np(D), dl.loss_records(out)
    for l in range(L):
        x = syn.workload_fill(2, l)
        F, ref_bits, ref_D, ref_L = orc.run(x, k)
        assert np.array_equal(got_bits[l], ref_bits), f"layer {l}: signatures differ"
        np.testing.assert_array_equal(got_D[l], ref_D, err_msg=f"layer {l}")
        loss_close(recs[l], ref_L)
        # the 16 experts biased by -10 are idle; their rows hold the loads (App. C.2)
        idle = np.flatnonzero(syn.workload_bias(2, l) < -5)
        loads = F.sum(axis=1, dtype=np.int64)
        assert len(idle) == 16 and not loads[idle].any()
        for i in idle:
            assert np.array_equal(got_D[l][i].astype(np.int64), np.where(np.arange(E) == i, 0, loads))
    # 48 x 512 = 24,576 work units: the run-time schedule choice applies
    _schedules_and_grams_agree(dl, scores, k, (bits, D, out), w["name"])


def test_workload3_stream_full(dl, orc, syn):
    w = syn.WORKLOADS[3]
    nmb, N, E, k = w["layers"], w["n"], w["E"], w["k"]
    print(f"[case] {w['name']} full, {nmb} x {N} tokens, E={E} k={k}", flush=True)
    mbs = [syn.workload_fill(3, b) for b in range(nmb)]
    dev = [to_dev(x) for x in mbs]
    _, ref_bits, ref_D, ref_L = orc.run_stream(mbs, k)
    s = dl.DoStream(E, k, nmb * N)
    try:
        for rep in range(2):  # the benchmark resets and re-appends every step
            s.reset()
            s.append_many(dev)
            D, out = s.finalize()
            torch.cuda.synchronize()
            assert s.tokens == nmb * N
            assert np.array_equal(bits_np(s.history(), nmb * N), ref_bits), f"rep {rep}: history differs"
            np.testing.assert_array_equal(D_np(D), ref_D)
            loss_close(dl.loss_records(out)[0], ref_L)
    finally:
        s.close()


def test_workload4_full(dl, orc, syn):
    w = syn.WORKLOADS[4]
    L, N, E, k = w["layers"], w["n"], w["E"], w["k"]
    print(f"[case] {w['name']} full, L={L} N={N} E={E} k={k}", flush=True)
    scores, _ = upload_workload(syn, 4, L)
    bits, D, out = dl.do_fused(scores, k, want_bits=True)
    torch.cuda.synchronize()
    _schedules_and_grams_agree(dl, scores, k, (bits, D, out), w["name"])
    # the surrogate loss (Eq. 7) and its gradient on the same tokens: the
    # scores of this workload are per-token probabilities
    print(f"[case] surrogate on the full workload L={L} N={N} E={E}", flush=True)
    sloss, grad = dl.do_surrogate(scores, k, bits, D)
    torch.cuda.synchronize()
    sloss = sloss.cpu().numpy()
    del scores
    torch.cuda.empty_cache()
    recs = dl.loss_records(out)
    got_D = D_np(D)
    rng = np.random.default_rng(44)
    for l in range(L):
        print(f"[case] {w['name']} layer {l}: full oracle", flush=True)
        words = bits_np(bits[l], N)
        x = syn.workload_fill(4, l)
        F, ref_bits, ref_D, ref_L = orc.run(x, k)
        assert np.array_equal(words, ref_bits), f"layer {l}: signatures differ"
        np.testing.assert_array_equal(got_D[l], ref_D, err_msg=f"layer {l}")
        loss_close(recs[l], ref_L)
        check_invariants(words, got_D[l], recs[l], N, k, f"layer {l}")
        # surrogate: the loss against the oracle's, sampled gradients against its gradient
        ref_s = orc.surrogate_loss_blocked(x, F, ref_D, k)
        assert sloss[l] == pytest.approx(ref_s, rel=1e-6), (l, sloss[l], ref_s)
        tok = np.sort(rng.choice(N, 256, replace=False))
        # the oracle's 1/(n^2 k) for n sampled tokens, rescaled to the full N
        _, ref_g = orc.surrogate(x[tok], F[:, tok], ref_D, k, scale=(len(tok) / N) ** 2)
        got_g = grad[l][torch.from_numpy(tok).cuda()].cpu().numpy().astype(np.float64)
        tol = 1e-5 * np.abs(ref_g) + 1e-6 * np.abs(ref_g).max()
        assert (np.abs(got_g - ref_g) <= tol).all(), f"layer {l}: sampled gradients differ"
        del x, F


def test_more_than_2_31_tokens(dl, orc):
    # token indices, signature words and sums past 32 bits: E = 2, k = 1 and
    # N = 2^31 + 100 (the largest expert count the overflow check allows at this
    # N).  Every token selects exactly one of the two experts, so the rows are
    # complements, D_01 = N and the loss is 2 N^2.  Sampled tokens are compared
    # with the oracle's Top-K of those rows.
    N, E, k = (1 << 31) + 100, 2, 1
    print(f"[case] N={N} E={E} k={k} fp32", flush=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(0x32398)
    x = torch.randn((N, E), dtype=torch.float32, device="cuda", generator=g)
    x[N - 7] = 0.5  # a tie near the end: the lower index wins
    bits, D, out = dl.do_fused(x, k, want_bits=True)
    torch.cuda.synchronize()
    W = (N + 63) // 64
    b = bits[0].permute(1, 0, 2).reshape(E, -1)[:, :W]  # expert-major rows (a device copy of the unit-major layout)
    full = W - 1
    assert bool(torch.all((b[0, :full] ^ b[1, :full]) == -1)), "rows are not complements"
    assert bool(torch.all((b[0] & b[1]) == 0)), "a token selected both experts"
    tail = (1 << (N % 64)) - 1
    assert int(b[0, full] ^ b[1, full]) & ((1 << 64) - 1) == tail, "tail word"
    lut = torch.tensor([bin(i).count("1") for i in range(256)], dtype=torch.int64, device="cuda")
    n0 = int(lut[b[0].contiguous().view(torch.uint8).long()].sum())
    assert n0 == int((x[:, 0] >= x[:, 1]).sum()), "load of expert 0"
    assert D.view(E, E).cpu().numpy().view(np.uint32).astype(np.int64).tolist() == [[0, N], [N, 0]]
    D2 = dl.do_pairwise_hamming(bits, N)  # the stored-signature Gram over 2^25 words per row
    torch.cuda.synchronize()
    assert D2.view(E, E).cpu().numpy().view(np.uint32).astype(np.int64).tolist() == [[0, N], [N, 0]]
    rec = dl.loss_records(out)[0]
    assert rec["sum"] == 2 * N and rec["sumsq"] == 2 * N * N
    assert rec["loss"] == float(2 * N * N) and rec["mean"] == float(N) and rec["var"] == 0.0
    rng = np.random.default_rng(7)
    ts = np.unique(np.concatenate([rng.integers(0, N, 2000), [0, 63, 64, (1 << 31) - 1, 1 << 31, N - 7, N - 1]]))
    rows = x[torch.from_numpy(ts).cuda()].cpu().numpy()
    F = orc.topk_signature(rows, k)  # [E][len(ts)] booleans of the sampled rows
    words = b[:, torch.from_numpy(ts // 64).cuda()].cpu().numpy().view(np.uint64)
    got = ((words >> (ts % 64).astype(np.uint64)) & np.uint64(1)).astype(bool)
    assert np.array_equal(got, np.asarray(F, dtype=bool)), "sampled tokens differ from the oracle"
    del x, bits


def test_maximum_layer_count(dl):
    # L = 65535 layers (1,024 launches of 64 layers; one finalize block per
    # layer) of one token each, E = 2, k = 1: in every layer the token selects
    # the expert with the larger score (expert 0 on a tie), so D_01 = 1 and
    # the loss is 2.
    L, N, E, k = 65535, 1, 2, 1
    print(f"[case] L={L} N={N} E={E} k={k} fp32", flush=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(65535)
    x = torch.randn((L, N, E), dtype=torch.float32, device="cuda", generator=g)
    x[100, 0, :] = -1.25  # a tie
    bits, D, out = dl.do_fused(x, k, want_bits=True)
    torch.cuda.synchronize()
    b = bits[:, 0, :, 0].cpu().numpy()  # word 0 of each expert: [layer][unit 0][expert][word 0]
    assert not bool(bits[:, 0, :, 1:].any()), "padding words of the last unit are not zero"
    want0 = (x[:, 0, 0] >= x[:, 0, 1]).cpu().numpy()
    assert np.array_equal(b[:, 0], want0.astype(np.int64)), "expert 0 bits"
    assert np.array_equal(b[:, 1], (~want0).astype(np.int64)), "expert 1 bits"
    Dn = D.view(L, E, E).cpu().numpy()
    assert np.all(Dn[:, 0, 1] == 1) and np.all(Dn[:, 1, 0] == 1) and np.all(Dn[:, 0, 0] == 0) and np.all(Dn[:, 1, 1] == 0)
    recs = dl.loss_records(out)
    assert len(recs) == L
    assert all(r["sum"] == 2 and r["sumsq"] == 2 and r["loss"] == 2.0 and r["var"] == 0.0 for r in recs)
