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


def bits_np(bits: torch.Tensor, N: int | None = None) -> np.ndarray:
    """Signatures in the library's unit-major layout ([..., U, E, 8] int64 on the device)
    -> expert-major numpy uint64 [..., E, W]: W = ceil(N/64) words when N is given (the
    words past it in the last unit are never written), else all 8 U."""
    a = bits.cpu().numpy().view(np.uint64)
    assert a.shape[-1] == 8, a.shape
    a = np.swapaxes(a, -3, -2)  # [..., E, U, 8]
    a = a.reshape(a.shape[:-2] + (a.shape[-2] * 8,))
    return np.ascontiguousarray(a if N is None else a[..., : (N + 63) // 64])


def units_dev(words: np.ndarray) -> torch.Tensor:
    """Expert-major signature words [..., E, W] (numpy uint64, e.g. the oracle's pack) ->
    the library's unit-major layout [..., U, E, 8] on the device, zero words past W."""
    W = words.shape[-1]
    U = (W + 7) // 8
    pad = np.zeros(words.shape[:-1] + (8 * U,), dtype=np.uint64)
    pad[..., :W] = words
    a = pad.reshape(words.shape[:-1] + (U, 8))
    a = np.ascontiguousarray(np.swapaxes(a, -3, -2))  # [..., U, E, 8]
    return torch.from_numpy(a.view(np.int64)).cuda()


def D_np(D: torch.Tensor) -> np.ndarray:
    return D.cpu().numpy().view(np.uint32)


def loss_close(got: dict, ref: dict, rel: float = 1e-5):
    """Exact integer sums, floats within `rel` (variance with an absolute floor)."""
    assert got["sum"] == ref["sum"], (got, ref)
    assert got["sumsq"] == ref["sumsq"], (got, ref)
    for f in ("loss", "mean"):
        assert abs(got[f] - ref[f]) <= rel * abs(ref[f]) + 1e-12, (f, got, ref)
    assert abs(got["var"] - ref["var"]) <= rel * abs(ref["var"]) + 1e-9 * max(1.0, ref["mean"] ** 2), (got, ref)


def upload_workload(syn, cfg: int, layers: int, keep=()) -> tuple:
    """Device tensor [layers][N][E] of a synthetic workload, generated one layer at
    a time on the host; host copies of the layers listed in `keep` are returned too."""
    w = syn.WORKLOADS[cfg]
    N, E = w["n"], w["E"]
    tdt = torch.float32 if w["dtype"] == 0 else torch.bfloat16
    dev = torch.empty((layers, N, E), dtype=tdt, device="cuda")
    kept = {}
    for l in range(layers):
        x = syn.workload_fill(cfg, l)
        if l in keep:
            kept[l] = x
        t = torch.from_numpy(x) if w["dtype"] == 0 else torch.from_numpy(x.view(np.int16)).view(torch.bfloat16)
        dev[l].copy_(t)
    torch.cuda.synchronize()
    return dev, kept


def bits_at(words: np.ndarray, tokens: np.ndarray) -> np.ndarray:
    """Dense 0/1 [E][len(tokens)] of the signature words [E][W] at the given token positions."""
    w = words[:, tokens >> 6]
    return ((w >> (tokens & 63).astype(np.uint64)) & np.uint64(1)).astype(np.uint8)


def check_invariants(words: np.ndarray, D: np.ndarray, rec: dict, N: int, k: int, label: str):
    """Properties that hold at any size (Eq. 2, App. C.2/C.3 row sums, exact loss of D)."""
    E = D.shape[0]
    loads = np.bitwise_count(words).sum(axis=1, dtype=np.int64)
    assert loads.sum() == N * k, f"{label}: {loads.sum()} selections, expected {N * k}"
    assert np.array_equal(D, D.T), f"{label}: D not symmetric"
    assert not np.diagonal(D).any(), f"{label}: nonzero diagonal"
    Di = D.astype(np.int64)
    assert Di.sum() == 2 * N * k * (E - k), f"{label}: zero-sum identity violated"
    rows = Di.sum(axis=1)
    assert np.array_equal(rows, (E - 2 * k) * loads + N * k), f"{label}: row sums differ from (E-2k) n_i + N k"
    assert rec["sum"] == int(Di.sum())
    assert rec["sumsq"] == int((Di * Di).sum())  # < 2^63 for every workload here
    return loads
