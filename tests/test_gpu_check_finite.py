"""The check-finite mode (do_set_option DO_OPT_CHECK_FINITE): the calls that
rank scores return DO_ERR_NONFINITE on a NaN score without writing anything,
accept +-inf, and give the same results as without the mode otherwise.
"""
import numpy as np
import pytest
import torch

from gpu_util import D_np, bits_np, loss_close, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dl():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32398_amd as p

    p.lib()
    return p


@pytest.fixture
def check_mode(dl):
    dl.set_option(dl.DO_OPT_CHECK_FINITE, 1)
    try:
        yield
    finally:
        dl.set_option(dl.DO_OPT_CHECK_FINITE, 0)


NAN_BITS = {0: [0x7FC00000, 0xFFC00001, 0x7F800001], 1: [0x7FC0, 0xFF81, 0x7F81]}


def _with_nan(x, pos, pattern):
    y = x.copy()
    flat = y.reshape(-1).view(np.uint32 if y.dtype == np.float32 else np.uint16)
    flat[pos] = pattern
    return y


def _offset_view(x, offset):
    """A device tensor holding x that starts `offset` elements into its allocation
    (aligned to the element size, not to 16 bytes when offset is odd)."""
    xd = to_dev(x)
    big = torch.empty(xd.numel() + offset, dtype=xd.dtype, device=xd.device)
    v = big[offset:].view(xd.shape)
    v.copy_(xd)
    return v


@pytest.mark.parametrize("dtype", [0, 1])
@pytest.mark.parametrize("offset", [0, 1, 3])
def test_nan_anywhere_is_reported_and_nothing_written(dl, syn, check_mode, dtype, offset):
    E, k, N, L = 40, 5, 1_001, 2
    x = np.stack([syn.normal(900 + l, N, E, dtype) for l in range(L)])
    n = x.size
    # first and last elements (head and tail of the scan) and a middle one
    for pos, pattern in [(0, NAN_BITS[dtype][0]), (n - 1, NAN_BITS[dtype][1]), (n // 2 + 7, NAN_BITS[dtype][2])]:
        print(f"[case] check-finite dtype={dtype} offset={offset} pos={pos}", flush=True)
        xd = _offset_view(_with_nan(x, pos, pattern), offset)
        bits = dl.alloc_bits(L, N, E, "cuda").fill_(7)
        D = torch.full((L, E, E), 5, dtype=torch.int32, device="cuda")
        out = dl.alloc_out(L, "cuda").fill_(3)
        with pytest.raises(dl.DoLossError) as ei:
            dl.do_fused(xd, k, bits=bits, D=D, out=out)
        assert ei.value.status == dl.DO_ERR_NONFINITE
        with pytest.raises(dl.DoLossError) as ei:
            dl.do_topk_signature(xd, k, bits=bits)
        assert ei.value.status == dl.DO_ERR_NONFINITE
        torch.cuda.synchronize()
        assert bool((bits == 7).all()) and bool((D == 5).all()) and bool((out == 3).all()), "a buffer was written"


@pytest.mark.parametrize("dtype", [0, 1])
def test_infinities_pass_and_results_match_the_unchecked_call(dl, orc, syn, dtype):
    E, k, N = 64, 6, 3_000
    x = syn.normal(911, N, E, dtype)
    flat = x.reshape(-1).view(np.uint32 if dtype == 0 else np.uint16)
    inf, ninf = (0x7F800000, 0xFF800000) if dtype == 0 else (0x7F80, 0xFF80)
    flat[5] = inf
    flat[E * 10 + 3] = ninf
    flat[-1] = inf
    xd = _offset_view(x, 1)
    ref_bits, ref_D, ref_out = dl.do_fused(xd, k, want_bits=True)
    torch.cuda.synchronize()
    dl.set_option(dl.DO_OPT_CHECK_FINITE, 1)
    try:
        bits, D, out = dl.do_fused(xd, k, want_bits=True)
        torch.cuda.synchronize()
    finally:
        dl.set_option(dl.DO_OPT_CHECK_FINITE, 0)
    assert torch.equal(bits, ref_bits) and torch.equal(D, ref_D) and torch.equal(out, ref_out)
    F = orc.topk_signature(x, k)
    np.testing.assert_array_equal(bits_np(bits[0], N), orc.pack(F))
    ref = orc.hamming(F)
    np.testing.assert_array_equal(D_np(D[0]), ref)
    loss_close(dl.loss_records(out)[0], orc.loss(ref))


def test_stream_append_with_nan_leaves_the_handle_unchanged(dl, orc, syn, check_mode):
    E, k, n = 128, 8, 4_096
    a = syn.normal(921, n, E, 1)
    b = syn.normal(922, n, E, 1)
    s = dl.DoStream(E, k, 4 * n)
    try:
        s.append(to_dev(a))
        bad = to_dev(_with_nan(b, 3 * E + 1, 0x7FC0))
        with pytest.raises(dl.DoLossError) as ei:
            s.append(bad)
        assert ei.value.status == dl.DO_ERR_NONFINITE
        with pytest.raises(dl.DoLossError) as ei:
            s.append_many([to_dev(b), bad])
        assert ei.value.status == dl.DO_ERR_NONFINITE
        s.append(to_dev(b))
        D, out = s.finalize()
        torch.cuda.synchronize()
        F = orc.topk_signature(np.concatenate([a, b]), k)
        ref = orc.hamming(F)
        np.testing.assert_array_equal(D_np(D), ref)
        loss_close(dl.loss_records(out)[0], orc.loss(ref))
    finally:
        s.close()


def test_check_mode_refuses_stream_capture(dl, syn, check_mode):
    E, k, N = 32, 4, 2_000
    xd = to_dev(syn.normal(931, N, E, 0))
    bits, D, out = dl.do_fused(xd, k, want_bits=True)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        with pytest.raises(dl.DoLossError) as ei:
            dl.do_fused(xd, k, bits=bits, D=D, out=out)
    assert ei.value.status == dl.DO_ERR_INVALID_ARG
