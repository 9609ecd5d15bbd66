"""do_profile_next: the caller's timing events bound to the Top-K dispatch.

The events must complete with a positive interval, and a timed call must give
the same signatures, distances and loss records as an untimed one.
"""
import numpy as np
import pytest
import torch

from gpu_util import D_np, bits_np, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dl():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32398_amd as p

    p.lib()
    return p


def _events():
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()  # materialise the handles
    b.record()
    torch.cuda.synchronize()
    return a, b


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_timed_fused_call_matches_untimed(dl, dtype):
    print(f"[case] profiled do_fused {dtype}", flush=True)
    rng = np.random.default_rng(11)
    x = rng.standard_normal((3, 7000, 128)).astype(np.float32)
    if dtype == "bf16":
        x = (x.view(np.uint32) >> 16).astype(np.uint16)
    xd = to_dev(x)
    b0, D0, o0 = dl.do_fused(xd, 8, want_bits=True)
    a, b = _events()
    dl.do_profile_next(a, b)
    b1, D1, o1 = dl.do_fused(xd, 8, want_bits=True)
    torch.cuda.synchronize()
    assert a.query() and b.query()
    assert 0.0 < a.elapsed_time(b) < 1000.0
    np.testing.assert_array_equal(bits_np(b1, 7000), bits_np(b0, 7000))
    np.testing.assert_array_equal(D_np(D1), D_np(D0))
    assert dl.loss_records(o1) == dl.loss_records(o0)


def test_timed_stream_append_and_noalloc_batch(dl):
    print("[case] profiled stream append_many and global batch", flush=True)
    rng = np.random.default_rng(12)
    E, k, n, count = 128, 8, 3000, 4
    mbs = [to_dev(rng.standard_normal((n, E)).astype(np.float32)) for _ in range(count)]
    s = dl.DoStream(E, k, n * count)
    s.append_many(mbs)
    D0, o0 = s.finalize()
    s.reset()
    a, b = _events()
    dl.do_profile_next(a, b)
    s.append_many(mbs)
    D1, o1 = s.finalize()
    torch.cuda.synchronize()
    assert 0.0 < a.elapsed_time(b) < 1000.0
    np.testing.assert_array_equal(D_np(D1), D_np(D0))
    assert dl.loss_records(o1) == dl.loss_records(o0)
    s.close()
    c, d = _events()
    dl.do_profile_next(c, d)
    _, D2, o2 = dl.do_global_batch_noalloc(mbs, k)
    torch.cuda.synchronize()
    assert 0.0 < c.elapsed_time(d) < 1000.0
    np.testing.assert_array_equal(D_np(D2), D_np(D0))
    assert dl.loss_records(o2) == dl.loss_records(o0)
