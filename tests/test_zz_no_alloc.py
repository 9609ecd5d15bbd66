"""do_global_batch_noalloc (the global batch without any library allocation)
against the handle-based stream (do_stream_create + do_stream_append_many +
do_stream_finalize) on the same micro-batches: history, distances and loss
record must be identical.  Two calls in a row share the static buffer; the
second is smaller (fewer experts, fewer and unaligned micro-batches), so a
count left over from the first call would show."""
import ctypes

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


def _via_handle(dl, mbs, E, k):
    s = dl.DoStream(E, k, len(mbs) * mbs[0].shape[0])
    try:
        s.append_many(mbs)
        D, out = s.finalize()
        torch.cuda.synchronize()
        return s.history(), D, out
    finally:
        s.close()


def _via_c_abi(dl, mbs, E, k):
    """The new entry point called through the C ABI directly (ctypes)."""
    n = mbs[0].shape[0]
    U = (len(mbs) * n + 511) // 512  # 512-token units of the signature layout
    hist = torch.full((U, E, 8), -1, dtype=torch.int64, device="cuda")  # garbage: the call must overwrite it
    D = torch.full((E, E), -1, dtype=torch.int32, device="cuda")
    out = torch.zeros((1, 40), dtype=torch.uint8, device="cuda")
    ptrs = (ctypes.c_void_p * len(mbs))(*[t.data_ptr() for t in mbs])
    st = dl.lib().do_global_batch_noalloc(ptrs, 1 if mbs[0].dtype == torch.bfloat16 else 0, n, len(mbs), E, k,
                                          hist.data_ptr(), D.data_ptr(), out.data_ptr(),
                                          ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, dl.lib().do_last_error()
    torch.cuda.synchronize()
    return hist, D, out


@pytest.mark.parametrize("first,second", [((128, 8, 16_384, 6, 1), (64, 6, 3_001, 3, 0)),
                                          ((256, 8, 9_000, 4, 0), (32, 5, 777, 2, 1))])
def test_noalloc_global_batch_matches_the_stream_handle(dl, syn, first, second):
    for call, (E, k, n, count, dt) in enumerate((first, second)):
        print(f"[case] noalloc call {call}: E={E} k={k} n={n} count={count} dtype={dt}", flush=True)
        mbs = [to_dev(syn.normal(5000 + 31 * b + E, n, E, dt)) for b in range(count)]
        ref = _via_handle(dl, mbs, E, k)
        got = _via_c_abi(dl, mbs, E, k)
        assert torch.equal(got[0], ref[0]), f"call {call}: history differs"
        assert torch.equal(got[1], ref[1]), f"call {call}: distances differ"
        assert torch.equal(got[2], ref[2]), f"call {call}: loss records differ"
        rec = dl.loss_records(got[2])[0]
        assert rec["sum"] == 2 * count * n * k * (E - k)  # Eq. 2 on the whole global batch
