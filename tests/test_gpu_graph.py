"""The fused pass and the separate calls under HIP-graph capture.

The library launches only kernels on the caller's stream (its buffers are
cleared with fill kernels, not memsets), so a captured do_fused replays to the
same bits, distances and loss as an eager call.  Every replay is checked, with
eager work and synchronisations between the replays.
"""
import time

import numpy as np
import pytest
import torch

from gpu_util import to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dl():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32398_amd as p

    p.lib()
    return p


@pytest.mark.parametrize("E,k,N,L,dtype", [(256, 8, 70_000, 3, 0), (128, 8, 100_001, 2, 1), (37, 5, 5_000, 2, 0)])
def test_fused_pass_replays_from_a_graph(dl, syn, E, k, N, L, dtype):
    print(f"[case] graph E={E} k={k} N={N} L={L} dtype={dtype}", flush=True)
    x = np.stack([syn.normal(4000 + 17 * l + E, N, E, dtype) for l in range(L)])
    xd = to_dev(x)
    ref_bits, ref_D, ref_out = dl.do_fused(xd, k, want_bits=True)
    torch.cuda.synchronize()
    bits = torch.zeros_like(ref_bits)
    D = torch.zeros_like(ref_D)
    out = torch.zeros_like(ref_out)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm the launch path outside the capture
        dl.do_fused(xd, k, bits=bits, D=D, out=out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        dl.do_fused(xd, k, bits=bits, D=D, out=out)
    for rep in range(3):
        bits.zero_()
        D.fill_(-1)
        out.zero_()
        y = torch.randn(1 << 20, device="cuda").sum()  # unrelated eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(bits, ref_bits), f"replay {rep}: signatures differ"
        assert torch.equal(D, ref_D), f"replay {rep}: distances differ"
        assert torch.equal(out, ref_out), f"replay {rep}: loss records differ"
        del y


def test_separate_calls_replay_from_a_graph(dl, syn):
    E, k, N = 64, 6, 30_000
    x = syn.normal(77, N, E, 1)
    xd = to_dev(x)
    ref_bits = dl.do_topk_signature(xd, k)
    ref_D = dl.do_pairwise_hamming(ref_bits, N)
    ref_out = dl.do_loss(ref_D)
    torch.cuda.synchronize()
    bits = torch.zeros_like(ref_bits)
    D = torch.zeros_like(ref_D)
    out = torch.zeros_like(ref_out)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        dl.do_topk_signature(xd, k, bits=bits)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        dl.do_topk_signature(xd, k, bits=bits)
        dl.do_pairwise_hamming(bits, N, D=D)
        dl.do_loss(D, out=out)
    for rep in range(3):
        bits.zero_()
        D.zero_()
        out.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(bits, ref_bits) and torch.equal(D, ref_D) and torch.equal(out, ref_out), rep


@pytest.mark.parametrize("E,k", [(128, 8), (300, 8)])
def test_stream_reset_append_finalize_replays_from_a_graph(dl, syn, E, k):
    # the stream finalize keeps its cross-block sums in the handle and clears
    # them itself: repeated finalize calls and graph replays give one result
    # (E = 300: the history's Gram is taken at finalize by the popcount kernel)
    n, nmb = 5_000, 4
    print(f"[case] graph stream E={E} k={k} n={n} x{nmb}", flush=True)
    mbs = [to_dev(syn.normal(300 + b, n, E, 1)) for b in range(nmb)]
    s = dl.DoStream(E, k, nmb * n)
    s.append_many(mbs)
    ref_D, ref_out = s.finalize()
    torch.cuda.synchronize()
    D2, out2 = s.finalize()
    torch.cuda.synchronize()
    assert torch.equal(D2, ref_D) and torch.equal(out2, ref_out), "second finalize differs"
    D = torch.zeros_like(ref_D)
    out = torch.zeros_like(ref_out)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        s.reset()
        s.append_many(mbs)
        s.finalize(D, out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        s.reset()
        s.append_many(mbs)
        s.finalize(D, out)
    for rep in range(3):
        D.fill_(-1)
        out.zero_()
        y = torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(D, ref_D), f"replay {rep}: distances differ"
        assert torch.equal(out, ref_out), f"replay {rep}: loss records differ"
        del y
    s.close()


def test_capture_while_the_schedule_tuner_is_measuring(dl, syn):
    # 4,194,304 tokens = 8,192 work units: the run-time schedule choice
    # applies.  The first eager call of the shape is unmeasured; the tuner
    # measures only from 100 ms after it, so after a pause the second call
    # leaves a measured trial pending and the capture happens while the tuner
    # is mid-way; a captured launch must not touch the measurement events and
    # must replay to the eager result, and eager calls after the capture
    # (which finish the measurement) must agree too.
    E, k, N = 16, 2, 1 << 22
    print(f"[case] graph during tuning E={E} k={k} N={N}", flush=True)
    xd = to_dev(syn.normal(909, N, E, 1))
    ref = dl.do_fused(xd, k, want_bits=True)
    torch.cuda.synchronize()
    time.sleep(0.15)
    again = dl.do_fused(xd, k, want_bits=True)  # a measured trial
    bits = torch.zeros_like(ref[0])
    D = torch.zeros_like(ref[1])
    out = torch.zeros_like(ref[2])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        dl.do_fused(xd, k, bits=bits, D=D, out=out)
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(again, ref)), "second eager call differs"
    for rep in range(3):
        bits.zero_()
        D.fill_(-1)
        out.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(bits, ref[0]) and torch.equal(D, ref[1]) and torch.equal(out, ref[2]), rep
        more = dl.do_fused(xd, k, want_bits=True)  # eager calls complete the measurement
        torch.cuda.synchronize()
        assert all(torch.equal(a, b) for a, b in zip(more, ref)), f"eager call {rep} after capture differs"
