"""Helpers for the GPU parity tests: host arrays <-> device tensors."""
import numpy as np
import torch


def to_dev(scores: np.ndarray) -> torch.Tensor:
    """float32 values or uint16 bf16 bit patterns -> contiguous CUDA tensor."""
    if scores.dtype == np.float32:
        return torch.from_numpy(np.ascontiguousarray(scores)).cuda()
    if scores.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(scores).view(np.int16)).view(torch.bfloat16).cuda()
    raise TypeError(scores.dtype)


def bits_np(bits: torch.Tensor) -> np.ndarray:
    """int64 device tensor of uint64 words -> numpy uint64."""
    return bits.cpu().numpy().view(np.uint64)


def D_np(D: torch.Tensor) -> np.ndarray:
    return D.cpu().numpy().view(np.uint32)


def loss_close(got: dict, ref: dict, rel: float = 1e-5):
    """Exact integer sums, floats within `rel` (variance with an absolute floor)."""
    assert got["sum"] == ref["sum"], (got, ref)
    assert got["sumsq"] == ref["sumsq"], (got, ref)
    for f in ("loss", "mean"):
        assert abs(got[f] - ref[f]) <= rel * abs(ref[f]) + 1e-12, (f, got, ref)
    assert abs(got["var"] - ref["var"]) <= rel * abs(ref["var"]) + 1e-9 * max(1.0, ref["mean"] ** 2), (got, ref)
