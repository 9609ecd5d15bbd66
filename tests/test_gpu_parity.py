"""HIP path vs the CPU oracle, element by element, through the C ABI.

Bar: signatures and distances bit-exact; loss sums exact, the fp64 loss,
mean and variance within 1e-5 relative of the oracle (spec tolerance).
"""
import numpy as np
import pytest
import torch

from gpu_util import D_np, bits_np, loss_close, to_dev, units_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dl():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32398_amd as p

    p.lib()
    return p


def _check_layer(dl, orc, scores_np, k, bits, D, rec, label=""):
    F = orc.topk_signature(scores_np, k)
    ref_bits = orc.pack(F)
    ref_D = orc.hamming(F)
    ref_L = orc.loss(ref_D)
    if bits is not None:
        got = bits_np(bits, scores_np.shape[0])
        if not np.array_equal(got, ref_bits):
            bad = np.argwhere(got != ref_bits)
            raise AssertionError(f"{label}: {len(bad)} signature words differ, first {bad[:4].tolist()}")
    np.testing.assert_array_equal(D_np(D), ref_D, err_msg=label)
    loss_close(rec, ref_L)


def _run_all_entry_points(dl, orc, x, k, label):
    """do_topk_signature, do_pairwise_hamming, do_loss and do_fused on one layer."""
    print(f"[case] {label} shape={x.shape} dtype={x.dtype} k={k}", flush=True)
    xd = to_dev(x)
    N, E = x.shape
    bits = dl.do_topk_signature(xd, k)
    D = dl.do_pairwise_hamming(bits, N)
    out = dl.do_loss(D)
    torch.cuda.synchronize()
    _check_layer(dl, orc, x, k, bits[0], D[0], dl.loss_records(out)[0], label + " (separate)")
    fb, fD, fout = dl.do_fused(xd, k, want_bits=True)
    torch.cuda.synchronize()
    _check_layer(dl, orc, x, k, fb[0], fD[0], dl.loss_records(fout)[0], label + " (fused)")
    _, fD2, fout2 = dl.do_fused(xd, k, want_bits=False)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(D_np(fD2), D_np(fD))
    assert dl.loss_records(fout2) == dl.loss_records(fout)


# ---------------------------------------------------------------------------
# the small workloads at full size
# ---------------------------------------------------------------------------
def test_workload0_e8_k2_n4096_f32(dl, orc, syn):
    x = syn.workload_fill(0, 0)
    _run_all_entry_points(dl, orc, x, 2, "workload0")


def test_workload1_e64_k6_n65536_bf16(dl, orc, syn):
    x = syn.workload_fill(1, 0)
    _run_all_entry_points(dl, orc, x, 6, "workload1")


# ---------------------------------------------------------------------------
# shapes, ties and special values
# ---------------------------------------------------------------------------
SHAPES = [
    (1, 1, 1), (3, 1, 5), (3, 3, 64), (5, 2, 63), (8, 8, 65), (13, 4, 100), (16, 1, 129), (24, 7, 1000),
    (37, 8, 257), (64, 8, 4097), (100, 3, 333), (128, 8, 3000), (200, 5, 1234), (256, 8, 2500), (256, 1, 700),
]


@pytest.mark.parametrize("E,k,N", SHAPES)
@pytest.mark.parametrize("dtype", [0, 1])
def test_random_shapes_normal(dl, orc, syn, E, k, N, dtype):
    x = syn.normal(1000 + 7 * E + N, N, E, dtype)
    _run_all_entry_points(dl, orc, x, k, f"normal E={E} k={k} N={N}")


# Unit-aligned launches (token counts and offsets multiples of 512, rows of
# whole 128-byte chunks) run a specialization of the score pass up to 128
# experts: fp32 rows of 32, 64, 96, 128 experts, bf16 rows of 64 and 128;
# several layers, every entry point, normal and tie-heavy scores.
@pytest.mark.parametrize("E,k,N,dtype", [(32, 1, 512, 0), (64, 8, 1536, 0), (96, 5, 2048, 0), (128, 8, 4608, 0),
                                         (64, 6, 512, 1), (128, 8, 3584, 1), (128, 1, 1024, 1),
                                         (160, 8, 1536, 0), (256, 8, 2048, 0), (256, 3, 512, 0),
                                         (192, 5, 1024, 1), (256, 8, 2560, 1)])
def test_unit_aligned_layers(dl, orc, syn, E, k, N, dtype):
    x = syn.normal(4000 + E + N, N, E, dtype)
    _run_all_entry_points(dl, orc, x, k, f"aligned normal E={E} k={k} N={N}")
    t = syn.int_ties(4100 + E, N, E, -3, 3, dtype)
    _run_all_entry_points(dl, orc, t, k, f"aligned ties E={E} k={k} N={N}")
    print(f"[case] aligned 3 layers E={E} k={k} N={N}", flush=True)
    layers = [syn.normal(4200 + E + l, N, E, dtype) for l in range(3)]
    xd = to_dev(np.stack(layers))
    bits, D, out = dl.do_fused(xd, k, want_bits=True)
    torch.cuda.synchronize()
    recs = dl.loss_records(out)
    for l, xl in enumerate(layers):
        _check_layer(dl, orc, xl, k, bits[l], D[l], recs[l], f"aligned layer {l}")


@pytest.mark.parametrize("E,k,dtype", [(128, 8, 1), (64, 6, 0)])
def test_stream_unit_aligned_and_unaligned_appends(dl, orc, syn, E, k, dtype):
    # aligned appends (the specialization), then an unaligned one, then
    # aligned again at an unaligned offset (the general kernel), one history
    print(f"[case] stream aligned/unaligned E={E} k={k} dtype={dtype}", flush=True)
    sizes = [2048, 512, 512, 1000, 512, 1536]
    parts = [syn.normal(4300 + i, n, E, dtype) for i, n in enumerate(sizes)]
    s = dl.DoStream(E, k, sum(sizes))
    s.append(to_dev(parts[0]))
    s.append_many([to_dev(parts[1]), to_dev(parts[2])])
    s.append(to_dev(parts[3]))
    s.append_many([to_dev(parts[4])])
    s.append(to_dev(parts[5]))
    D, out = s.finalize()
    hist = s.history()
    torch.cuda.synchronize()
    F, words, ref_D, ref_L = orc.run_stream(parts, k)
    np.testing.assert_array_equal(D_np(D), ref_D)
    loss_close(dl.loss_records(out)[0], ref_L)
    np.testing.assert_array_equal(bits_np(hist)[:, : words.shape[1]], words)
    s.close()


@pytest.mark.parametrize("E,k,N", [(8, 2, 500), (24, 8, 700), (64, 6, 999), (128, 8, 1500), (256, 8, 640),
                                   (40, 3, 128), (96, 8, 200)])
@pytest.mark.parametrize("dtype", [0, 1])
def test_tie_heavy_integer_scores(dl, orc, syn, E, k, N, dtype):
    x = syn.int_ties(77 + E, N, E, -3, 3, dtype)
    _run_all_entry_points(dl, orc, x, k, f"ties E={E} k={k} N={N}")


@pytest.mark.parametrize("E,k,N", [(12, 9, 300), (64, 20, 200), (33, 33, 100), (300, 8, 150), (1024, 12, 70),
                                   (520, 1, 90)])
def test_slow_paths_large_k_and_wide_E(dl, orc, syn, E, k, N):
    x = syn.normal(5 + E, N, E, 0)
    print(f"[case] slow E={E} k={k} N={N}", flush=True)
    xd = to_dev(x)
    bits = dl.do_topk_signature(xd, k)
    D = dl.do_pairwise_hamming(bits, N)
    out = dl.do_loss(D)
    fb, fD, fout = dl.do_fused(xd, k, want_bits=True)
    torch.cuda.synchronize()
    _check_layer(dl, orc, x, k, bits[0], D[0], dl.loss_records(out)[0], "slow separate")
    _check_layer(dl, orc, x, k, fb[0], fD[0], dl.loss_records(fout)[0], "slow fused")


def _special_rows(dtype, E, N, seed):
    rng = np.random.default_rng(seed)
    vals32 = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1.0, -1.0, 1e-40, -1e-40, 3.5], dtype=np.float32)
    x = rng.standard_normal((N, E)).astype(np.float32)
    mask = rng.random((N, E)) < 0.3
    x[mask] = rng.choice(vals32, size=mask.sum())
    x[0, :] = -0.0
    x[1, :] = np.nan
    x[2, ::2] = np.inf
    x[3, :] = 0.0
    x[3, ::3] = -0.0
    x[4, :] = -np.inf
    x[4, 1] = np.nan
    if dtype == 0:
        return x
    b = x.view(np.uint32)
    return (b >> 16).astype(np.uint16)  # truncation keeps every special value (and makes more ties)


@pytest.mark.parametrize("E,k,N", [(8, 2, 300), (16, 8, 200), (64, 6, 256), (256, 8, 128), (40, 5, 100)])
@pytest.mark.parametrize("dtype", [0, 1])
def test_special_values(dl, orc, E, k, N, dtype):
    x = _special_rows(dtype, E, N, E * 31 + k)
    _run_all_entry_points(dl, orc, x, k, f"specials E={E} k={k}")


@pytest.mark.parametrize("dtype", [0, 1])
def test_negative_and_bucket_ties_fp32(dl, orc, syn, dtype):
    # all-negative scores (threshold below zero) and fp32 values that share
    # their top 24 bits (force the exact re-rank)
    x = syn.normal(9, 2000, 64, dtype, mean=-20.0)
    _run_all_entry_points(dl, orc, x, 8, "negative")
    if dtype == 0:
        base = syn.normal(10, 1000, 32, 0)
        bits = base.view(np.uint32) & np.uint32(0xFFFFFF00)
        bits = bits | (np.arange(32, dtype=np.uint32)[None, ::-1] & np.uint32(0xFF))
        _run_all_entry_points(dl, orc, bits.view(np.float32), 5, "bucket ties")


def _key_switch_rows(seed):
    """bf16 rows of 128 experts around the in-row switch to positive keys.

    Scores come from a small set (many equal values, both zeros) and words of
    64 tokens take turns: (0) every token has 12 positive scores among experts
    0-63, so the wave switches after its first chunk; (1) as (0), but one token
    has 5 positives there and 1 after, so its top-8 holds tied negative scores
    and the wave must keep general keys; (2) 7 positives and a +0 among
    experts 0-63 (the 8th key is not positive: no switch)."""
    rng = np.random.default_rng(seed)
    N, E = 64 * 24 + 37, 128
    pos = np.array([0.25, 0.5, 1.0, 2.0, 3.0], np.float32)
    neg = np.array([-8.0, -3.0, -2.5, -1.0, -0.5, -0.0], np.float32)
    both = np.concatenate([pos, neg, np.array([0.0], np.float32)])
    x = np.empty((N, E), np.float32)
    for t in range(N):
        w, lane = divmod(t, 64)
        kind = w % 3
        row = np.empty(E, np.float32)
        npos = 12 if kind < 2 else 7
        if kind == 1 and lane == (w * 7) % 64:
            npos = 5
        first = rng.choice(neg, 64)
        first[rng.choice(64, npos, replace=False)] = rng.choice(pos, npos)
        if kind == 2:
            first[rng.choice(np.flatnonzero(first < 0), 1)] = 0.0
        row[:64] = first
        if kind == 1 and lane == (w * 7) % 64:
            second = rng.choice(neg, 64)
            second[rng.integers(64)] = rng.choice(pos)
        else:
            second = rng.choice(both, 64)
        row[64:] = second
        x[t] = row
    return (x.view(np.uint32) >> 16).astype(np.uint16)


@pytest.mark.parametrize("k", [8, 3])
def test_bf16_rows_switching_to_positive_keys(dl, orc, k):
    x = _key_switch_rows(77 + k)
    _run_all_entry_points(dl, orc, x, k, f"bf16 key switch k={k}")


def _bucket_tie_rows(rng, N, E, k, sign):
    """fp32 rows whose k-th and (k+1)-th largest values share their top 24
    bits: a cluster of 2..k+3 values b with random low bytes (some exactly
    equal) sits at random positions among clearly larger and smaller values."""
    x = rng.normal(size=(N, E)).astype(np.float32)
    for t in range(N):
        above = rng.integers(0, k)  # values clearly above the cluster
        m = int(rng.integers(max(2, k - above + 1), k - above + 4))
        m = min(m, E - above)
        pos = rng.permutation(E)
        b = np.float32(sign * rng.uniform(0.5, 4.0))
        bb = np.uint32(b.view(np.uint32)) & np.uint32(0xFFFFFF00)
        low = rng.integers(0, 256, size=m).astype(np.uint32)
        if m >= 3:
            low[1] = low[2]  # an exact duplicate inside the bucket
        cl = (bb | low).view(np.float32)
        x[t, pos[:m]] = cl
        x[t, pos[m:m + above]] = np.abs(b) * 4 + 1 + rng.random(above).astype(np.float32)
        x[t, pos[m + above:]] = -np.abs(b) * 4 - 1 - rng.random(E - m - above).astype(np.float32)
    return x


@pytest.mark.parametrize("E,k", [(32, 1), (32, 5), (100, 8), (256, 8), (256, 3)])
@pytest.mark.parametrize("sign", [1.0, -1.0])
def test_fp32_bucket_ties_resolved(dl, orc, E, k, sign):
    # keys keep 24 value bits: the low 8 bits must still decide the Top-K
    rng = np.random.default_rng(1000 + E + k)
    x = _bucket_tie_rows(rng, 700, E, k, sign)
    _run_all_entry_points(dl, orc, x, k, f"bucket cluster E={E} k={k} sign={sign}")


def test_misaligned_scores_take_the_exact_path(dl, orc, syn):
    N, E, k = 500, 64, 6
    x = syn.normal(3, N, E, 0)
    buf = torch.zeros(N * E + 1, dtype=torch.float32, device="cuda")
    buf[1:] = torch.from_numpy(x.reshape(-1)).cuda()
    xd = buf[1:].view(N, E)
    assert xd.data_ptr() % 16 != 0
    bits = dl.do_topk_signature(xd, k)
    _, D, out = dl.do_fused(xd, k)
    torch.cuda.synchronize()
    _check_layer(dl, orc, x, k, bits[0], D[0], dl.loss_records(out)[0], "misaligned")


def test_multi_layer_batching_beyond_one_launch(dl, orc, syn):
    L, N, E, k = 70, 130, 16, 3
    x = np.stack([syn.normal(40 + l, N, E, 1) for l in range(L)])
    xd = to_dev(x.reshape(L * N, E)).view(L, N, E)
    fb, fD, fout = dl.do_fused(xd, k, want_bits=True)
    bits = dl.do_topk_signature(xd, k)
    torch.cuda.synchronize()
    recs = dl.loss_records(fout)
    for l in (0, 1, 63, 64, 69):
        _check_layer(dl, orc, x[l], k, fb[l], fD[l], recs[l], f"layer {l}")
    np.testing.assert_array_equal(bits_np(bits, N), bits_np(fb, N))


def test_loss_of_arbitrary_matrices(dl):
    rng = np.random.default_rng(0)
    for E in (1, 2, 7, 300):
        D = rng.integers(0, 1 << 20, size=(3, E, E), dtype=np.uint32)
        out = dl.do_loss(torch.from_numpy(D.view(np.int32)).cuda())
        torch.cuda.synchronize()
        recs = dl.loss_records(out)
        for l in range(3):
            off = ~np.eye(E, dtype=bool)
            v = D[l][off].astype(object)
            s1 = int(sum(v)) if E > 1 else 0
            s2 = int(sum(a * a for a in v)) if E > 1 else 0
            P = E * (E - 1)
            assert recs[l]["sum"] == s1 and recs[l]["sumsq"] == s2
            if E > 1:
                assert recs[l]["mean"] == pytest.approx(s1 / P, rel=1e-12)
                assert recs[l]["var"] == pytest.approx((s2 * P - s1 * s1) / (P * P), rel=1e-9)
            else:
                assert recs[l] == dict(sum=0, sumsq=0, loss=0.0, mean=0.0, var=0.0)
    # one column past a 128-column load batch, and the largest E: exact sums in
    # uint64 (entries < 2^20, so the sum of squares stays below 2^60)
    for E in (129, 1024):
        D = rng.integers(0, 1 << 20, size=(1, E, E), dtype=np.uint32)
        out = dl.do_loss(torch.from_numpy(D.view(np.int32)).cuda())
        torch.cuda.synchronize()
        rec = dl.loss_records(out)[0]
        v = D[0][~np.eye(E, dtype=bool)].astype(np.uint64)
        assert rec["sum"] == int(v.sum()) and rec["sumsq"] == int((v * v).sum()), f"E={E}"


@pytest.mark.parametrize("E,hi", [(2, (1 << 32) - 1), (64, (1 << 32) - 1), (300, 3_000_000_000), (1024, (1 << 32) - 1),
                                  (5, 1 << 30)])
def test_loss_of_matrices_with_entries_near_2_32(dl, E, hi):
    # Any uint32 entries: the sum of squares is exact in 128 bits, `sumsq`
    # saturates at 2^64 - 1 once it does not fit, `loss` is the exact sum in
    # fp64 and `var` the exact population variance, both pinned here with
    # Python integers (E = 5 with entries < 2^30 stays below 2^64: exact sumsq).
    rng = np.random.default_rng(E)
    D = rng.integers(hi // 2, hi, size=(2, E, E), dtype=np.uint64).astype(np.uint32)
    D[1, 0, 1 % E] = hi  # the largest entry, once
    out = dl.do_loss(torch.from_numpy(D.view(np.int32)).cuda())
    torch.cuda.synchronize()
    for l, rec in enumerate(dl.loss_records(out)):
        v = [int(a) for a in D[l][~np.eye(E, dtype=bool)]]
        P = E * (E - 1)
        s1, s2 = sum(v), sum(a * a for a in v)
        assert rec["sum"] == s1
        assert rec["sumsq"] == (s2 if s2 < (1 << 64) else (1 << 64) - 1), (E, s2)
        assert rec["loss"] == pytest.approx(float(s2), rel=4.5e-16)
        assert rec["mean"] == pytest.approx(s1 / P, rel=1e-15)
        var = (s2 * P - s1 * s1) / (P * P)  # exact rational, rounded once
        assert rec["var"] == pytest.approx(var, rel=1e-12)


def test_hamming_of_oracle_signatures(dl, orc, syn):
    x = syn.normal(12, 5000, 96, 1)
    F = orc.topk_signature(x, 7)
    words = orc.pack(F)
    D = dl.do_pairwise_hamming(units_dev(words), 5000)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(D_np(D)[0], orc.hamming(F))


def test_determinism_bit_identical_reruns(dl, syn):
    x = to_dev(syn.normal(2, 20000, 128, 1))
    a = dl.do_fused(x, 8, want_bits=True)
    b = dl.do_fused(x, 8, want_bits=True)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1]) and torch.equal(a[2], b[2])


@pytest.mark.parametrize("E,k,dtype", [(64, 6, 1), (256, 8, 0), (130, 8, 0)])
def test_fused_distances_not_8_byte_aligned(dl, orc, syn, E, k, dtype):
    """D only 4-byte aligned: the co-occurrence counts take 32-bit atomics."""
    L, N = 3, 3001
    x = np.stack([syn.normal(500 + 3 * E + l, N, E, dtype) for l in range(L)])
    xd = to_dev(x)
    big = torch.empty(L * E * E + 1, dtype=torch.int32, device="cuda")
    D = big[1:].view(L, E, E)
    assert D.data_ptr() % 8 == 4
    bits, D, out = dl.do_fused(xd, k, want_bits=True, D=D)
    torch.cuda.synchronize()
    recs = dl.loss_records(out)
    for l in range(L):
        _check_layer(dl, orc, x[l], k, bits[l], D[l], recs[l], f"layer {l}")


# ---------------------------------------------------------------------------
# streaming history
# ---------------------------------------------------------------------------
def test_stream_unaligned_appends_equal_one_batch(dl, orc, syn):
    E, k = 64, 6
    sizes = [1000, 37, 64, 1, 4096, 130, 63]
    parts = [syn.normal(500 + i, n, E, 1) for i, n in enumerate(sizes)]
    s = dl.DoStream(E, k, 10000)
    for p in parts:
        s.append(to_dev(p))
    assert s.tokens == sum(sizes)
    D, out = s.finalize()
    torch.cuda.synchronize()
    F, words, ref_D, ref_L = orc.run_stream(parts, k)
    np.testing.assert_array_equal(D_np(D), ref_D)
    loss_close(dl.loss_records(out)[0], ref_L)
    hist = s.history()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bits_np(hist)[:, : words.shape[1]], words)
    assert not bits_np(hist)[:, words.shape[1]:].any()  # never-used words are zero before any reset
    # finalize twice gives the same answer; after a reset nothing is counted
    D2, out2 = s.finalize()
    torch.cuda.synchronize()
    assert torch.equal(D, D2) and torch.equal(out, out2)
    s.reset()
    D3, out3 = s.finalize()
    torch.cuda.synchronize()
    assert s.tokens == 0 and int(D3.abs().sum()) == 0
    assert dl.loss_records(out3)[0]["sum"] == 0
    # the old bits stay in the history after the reset; unaligned appends that
    # follow must not OR into them: a new epoch with another split of fewer
    # tokens gives the oracle's words over the tokens it holds
    sizes2 = [70, 1, 129, 64, 500]
    parts2 = [syn.normal(700 + i, n, E, 1) for i, n in enumerate(sizes2)]
    for p in parts2:
        s.append(to_dev(p))
    D4, out4 = s.finalize()
    hist4 = s.history()
    torch.cuda.synchronize()
    F2, words2, ref_D2, ref_L2 = orc.run_stream(parts2, k)
    np.testing.assert_array_equal(D_np(D4), ref_D2)
    loss_close(dl.loss_records(out4)[0], ref_L2)
    np.testing.assert_array_equal(bits_np(hist4)[:, : words2.shape[1]], words2)
    s.close()


@pytest.mark.parametrize("E,k,dtype", [(128, 8, 1), (256, 8, 0), (40, 5, 1)])
def test_stream_finalize_between_appends_and_resets(dl, orc, syn, E, k, dtype):
    """The handle's running totals: finalize after each append (the counts of
    all tokens so far), appends after a finalize, a reset right after appends
    (counters not yet finalized) and a reset right after a finalize."""
    print(f"[case] stream epochs E={E} k={k} dtype={dtype}", flush=True)
    sizes = [4096, 128, 960, 64 * 9]
    parts = [syn.normal(1300 + 17 * i + E, n, E, dtype) for i, n in enumerate(sizes)]
    dev = [to_dev(p) for p in parts]
    s = dl.DoStream(E, k, sum(sizes))
    try:
        for epoch in range(2):
            for upto in range(1, len(parts) + 1):
                s.append(dev[upto - 1])
                D, out = s.finalize()
                torch.cuda.synchronize()
                _, words, ref_D, ref_L = orc.run_stream(parts[:upto], k)
                np.testing.assert_array_equal(D_np(D), ref_D, err_msg=f"epoch {epoch}, {upto} appends")
                loss_close(dl.loss_records(out)[0], ref_L)
                np.testing.assert_array_equal(bits_np(s.history())[:, : words.shape[1]], words)
            s.reset()  # right after a finalize
        # appends, then a reset before any finalize, then one aligned append
        s.append_many(dev[:1])
        s.append(dev[1])
        s.reset()
        s.append(dev[3])
        D, out = s.finalize()
        torch.cuda.synchronize()
        _, words, ref_D, ref_L = orc.run_stream(parts[3:4], k)
        np.testing.assert_array_equal(D_np(D), ref_D)
        loss_close(dl.loss_records(out)[0], ref_L)
        np.testing.assert_array_equal(bits_np(s.history())[:, : words.shape[1]], words)
    finally:
        s.close()


@pytest.mark.parametrize("E,k,sizes", [(128, 8, [1000, 4096, 333]), (40, 5, [64, 700]), (300, 8, [513, 1024])])
def test_stream_history_prefix_is_a_signature_array(dl, orc, syn, E, k, sizes):
    # the history's first ceil(tokens/512) units are the signature array of the
    # appended tokens: do_pairwise_hamming over them gives the finalize's D
    print(f"[case] history prefix E={E} k={k} sizes={sizes}", flush=True)
    parts = [syn.normal(1500 + 11 * i + E, n, E, 1) for i, n in enumerate(sizes)]
    s = dl.DoStream(E, k, 4 * sum(sizes))
    try:
        for p in parts:
            s.append(to_dev(p))
        N = s.tokens
        D, _ = s.finalize()
        hist = s.history()[: (N + 511) // 512].contiguous()
        D2 = dl.do_pairwise_hamming(hist, N)
        torch.cuda.synchronize()
        _, words, ref_D, _ = orc.run_stream(parts, k)
        np.testing.assert_array_equal(D_np(D2)[0], ref_D)
        assert torch.equal(D2[0], D)
        np.testing.assert_array_equal(bits_np(hist, N), words)
    finally:
        s.close()


def test_stream_append_many_and_capacity(dl, orc, syn):
    E, k, nmb = 128, 8, 5
    parts = [syn.normal(900 + i, 777, E, 1) for i in range(nmb)]
    s = dl.DoStream(E, k, 777 * nmb)
    s.append_many([to_dev(p) for p in parts])
    D, out = s.finalize()
    torch.cuda.synchronize()
    F, words, ref_D, ref_L = orc.run_stream(parts, k)
    np.testing.assert_array_equal(D_np(D), ref_D)
    loss_close(dl.loss_records(out)[0], ref_L)
    with pytest.raises(dl.DoLossError) as ei:
        s.append(to_dev(parts[0][:1]))
    assert ei.value.status == dl.DO_ERR_CAPACITY
    assert s.tokens == 777 * nmb
    s.close()


def test_stream_wide_E_gram_at_finalize(dl, orc, syn):
    E, k = 300, 4
    parts = [syn.normal(60 + i, n, E, 0) for i, n in enumerate([100, 65, 300])]
    s = dl.DoStream(E, k, 465)
    for p in parts:
        s.append(to_dev(p))
    D, out = s.finalize()
    torch.cuda.synchronize()
    F, words, ref_D, ref_L = orc.run_stream(parts, k)
    np.testing.assert_array_equal(D_np(D), ref_D)
    loss_close(dl.loss_records(out)[0], ref_L)
    s.close()


@pytest.mark.parametrize("E,k,L,N,offset", [(256, 8, 3, 70_001, 0), (37, 5, 2, 5_000, 1), (128, 8, 5, 100_000, 1),
                                            (2, 1, 4, 64, 0), (64, 6, 1, 1_000_003, 0)])
def test_pairwise_hamming_of_stored_layers(dl, orc, syn, E, k, L, N, offset):
    """do_pairwise_hamming over several layers of oracle signatures; with
    offset 1 the distances are only 4-byte aligned (32-bit count atomics)."""
    print(f"[case] hamming E={E} k={k} L={L} N={N} offset={offset}", flush=True)
    Fs = [orc.topk_signature(syn.normal(900 + 7 * E + l, N, E, 1), k) for l in range(L)]
    words = np.stack([orc.pack(F) for F in Fs])
    big = torch.empty(L * E * E + offset, dtype=torch.int32, device="cuda")
    D = big[offset:].view(L, E, E)
    dl.do_pairwise_hamming(units_dev(words), N, D=D)
    torch.cuda.synchronize()
    got = D_np(D)
    for l in range(L):
        np.testing.assert_array_equal(got[l], orc.hamming(Fs[l]), err_msg=f"layer {l}")


def test_stream_append_of_zero_tokens_changes_nothing(dl, orc, syn):
    E, k = 64, 6
    print(f"[case] stream zero-token appends E={E} k={k}", flush=True)
    x = syn.normal(4242, 3000, E, 1)
    xd = to_dev(x)
    s = dl.DoStream(E, k, 5000)
    s.append(xd[:0])  # a zero-length view: valid pointer, no tokens
    assert s.tokens == 0
    s.append(xd[:1234])
    s.append(xd[1234:1234])
    s.append_many([xd[:0], xd[5:5]])
    s.append(xd[1234:])
    assert s.tokens == 3000
    D, out = s.finalize()
    torch.cuda.synchronize()
    F = orc.topk_signature(x, k)
    np.testing.assert_array_equal(D_np(D), orc.hamming(F))
    s.close()
