"""DO-loss hot path on MI355X: Python binding of the C ABI in include/doloss.h.

Argument marshalling only: every step of the path runs in the HIP kernels of
``libdoloss.so``.  torch is used for device memory and the current stream.
There is no CPU fallback; if the library is missing the import of the
binding's functions raises.

Functions keep the C names:

* ``do_topk_signature(scores, k)``  -> bits  [L][U][E][8] int64 (uint64 bit patterns), U = ceil(N/512):
  word w of expert e is bits[l, w // 8, e, w % 8] (the library's unit-major signature layout)
* ``do_pairwise_hamming(bits, N)``   -> D     [L][E][E] int32 (uint32 values)
* ``do_loss(D)``                     -> out   [L][5] (sum, sumsq, loss, mean, var) as a dict list
* ``do_fused(scores, k, want_bits)`` -> (bits or None, D, out)
* ``do_surrogate(p, k, bits, D)``    -> (loss [L] float64, dloss/dp [L][N][E] float32)
* ``DoStream``                       -> streaming history (do_stream_*)
* ``do_rem_allocate`` / ``do_rem_dispatch`` -> REM replica placement and token routes

``scores`` is a CUDA tensor of shape [N, E] or [L, N, E], float32 or bfloat16.
"""
from __future__ import annotations

import ctypes
import os

import torch

from .hipbuild import LIB_PATH, build  # noqa: F401

DO_OK, DO_ERR_INVALID_ARG, DO_ERR_UNSUPPORTED_DTYPE, DO_ERR_CAPACITY, DO_ERR_OVERFLOW, DO_ERR_HIP, DO_ERR_NONFINITE = range(7)
DO_F32, DO_BF16 = 0, 1
DO_OPT_SCHEDULE, DO_OPT_GRAM, DO_OPT_CHECK_FINITE = 0, 1, 2

LOSS_RESULT_BYTES = 40
LOSS_FIELDS = ("sum", "sumsq", "loss", "mean", "var")
LOAD_STATS_BYTES = 32


class DoLossError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        super().__init__(f"{where}: status {status} ({msg})")
        self.status = status


_lib = None


def lib():
    """The loaded libdoloss.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        st = ctypes.c_int
        sigs = {
            "do_topk_signature": ([vp, st, i64, i32, i32, i32, vp, vp], st),
            "do_pairwise_hamming": ([vp, i64, i32, i32, vp, vp], st),
            "do_loss": ([vp, i32, i32, vp, vp], st),
            "do_fused": ([vp, st, i64, i32, i32, i32, vp, vp, vp, vp], st),
            "do_surrogate": ([vp, st, i64, i32, i32, i32, vp, vp, ctypes.c_double, vp, vp, vp], st),
            "do_load_stats": ([vp, i64, i64, i32, i32, i32, vp, st, vp, i32, vp, vp, vp], st),
            "do_stream_create": ([i32, i32, i64, ctypes.POINTER(vp)], st),
            "do_stream_append": ([vp, vp, st, i64, vp], st),
            "do_stream_append_many": ([vp, ctypes.POINTER(vp), st, i64, i32, vp], st),
            "do_stream_finalize": ([vp, vp, vp, vp], st),
            "do_stream_reset": ([vp, vp], st),
            "do_stream_destroy": ([vp], st),
            "do_stream_bits": ([vp], vp),
            "do_stream_tokens": ([vp], i64),
            "do_stream_words_per_expert": ([vp], i64),
            "do_status_string": ([st], ctypes.c_char_p),
            "do_last_error": ([], ctypes.c_char_p),
            "do_version": ([], i32),
            "do_profile_next": ([vp, vp], st),
            "do_set_option": ([st, i32], st),
            "do_global_batch_noalloc": ([ctypes.POINTER(vp), st, i64, i32, i32, i32, vp, vp, vp, vp], st),
            "do_rem_allocate": ([vp, vp, vp, i32, i32, i32, i32, vp, vp, vp, vp, vp], st),
            "do_rem_dispatch": ([vp, vp, i32, vp, vp, i32, i32, i32, i32, vp, vp, vp, vp, vp], st),
        }
        for name, (args, res) in sigs.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


_hip = None


def _hip_copy_d2d(dst: int, src: int, nbytes: int) -> int:
    """Device-to-device copy on the current stream through the HIP runtime torch loaded."""
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so.7")
        _hip.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int,
                                        ctypes.c_void_p]
        _hip.hipMemcpyAsync.restype = ctypes.c_int
    rc = _hip.hipMemcpyAsync(dst, src, nbytes, 3, _stream())  # 3 = hipMemcpyDeviceToDevice
    return DO_OK if rc == 0 else DO_ERR_HIP


def _check(status: int, where: str):
    if status != DO_OK:
        raise DoLossError(status, where, lib().do_last_error().decode())


def _stream() -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return DO_F32
    if t.dtype == torch.bfloat16:
        return DO_BF16
    raise TypeError(f"unsupported score dtype {t.dtype}")


def _want(t: torch.Tensor, name: str, shape=None, dtypes=None, numel=None):
    """Checks a tensor argument before its pointer reaches the library: shape
    (or element count), dtype and contiguity first, then that it lives on the
    current GPU.  Every failure raises ValueError before any launch."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch.Tensor")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, at least {numel} are needed")
    if dtypes is not None and t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    why = _device_problem(t)
    if why:
        raise ValueError(f"{name} {why}")


def _device_problem(t: torch.Tensor) -> str | None:
    """Why `t` cannot be handed to the library as device memory, or None."""
    if not t.is_cuda:
        return "must be a device tensor"
    if t.device.index != torch.cuda.current_device():
        return f"is on {t.device}, not on the current device"
    return None


_SCORE_DTYPES = (torch.float32, torch.bfloat16)
_I64, _I32, _U8 = (torch.int64,), (torch.int32,), (torch.uint8,)


def _scores_3d(scores: torch.Tensor, name: str = "scores"):
    if not isinstance(scores, torch.Tensor) or scores.dim() not in (2, 3):
        raise ValueError(f"{name} must be a tensor of shape [N, E] or [L, N, E]")
    _want(scores, name, dtypes=_SCORE_DTYPES)
    if scores.dim() == 2:
        return 1, scores.shape[0], scores.shape[1]
    return scores.shape[0], scores.shape[1], scores.shape[2]


def _units(N: int) -> int:
    """512-token units of the signature layout."""
    return (N + 511) // 512


def set_option(option: int, value: int):
    """do_set_option: process-wide options (DO_OPT_SCHEDULE: -1 tuned, 0 XCD-partitioned,
    1 contiguous; DO_OPT_GRAM: 0 MFMA, 1 popcount; DO_OPT_CHECK_FINITE: 1 makes the
    score-ranking calls fail with DO_ERR_NONFINITE on a NaN score, 0 turns it off)."""
    _check(lib().do_set_option(int(option), int(value)), "do_set_option")


def loss_records(out: torch.Tensor) -> list[dict]:
    """Decode a [L, 40] uint8 tensor of do_loss_result records."""
    raw = out.detach().cpu().contiguous().view(torch.uint8).numpy().reshape(-1, LOSS_RESULT_BYTES)
    recs = []
    for r in raw:
        u = r[:16].view("<u8")
        d = r[16:].view("<f8")
        recs.append(dict(sum=int(u[0]), sumsq=int(u[1]), loss=float(d[0]), mean=float(d[1]), var=float(d[2])))
    return recs


def alloc_bits(L: int, N: int, E: int, device) -> torch.Tensor:
    """Signatures [L, U, E, 8], U = ceil(N/512) (see include/doloss.h)."""
    return torch.empty((L, _units(N), E, 8), dtype=torch.int64, device=device)


def alloc_D(L: int, E: int, device) -> torch.Tensor:
    return torch.empty((L, E, E), dtype=torch.int32, device=device)


def alloc_out(L: int, device) -> torch.Tensor:
    return torch.empty((L, LOSS_RESULT_BYTES), dtype=torch.uint8, device=device)


def do_topk_signature(scores: torch.Tensor, k: int, bits: torch.Tensor | None = None) -> torch.Tensor:
    L, N, E = _scores_3d(scores)
    if bits is None:
        bits = alloc_bits(L, N, E, scores.device)
    _want(bits, "bits", numel=L * E * 8 * _units(N), dtypes=_I64)
    _check(lib().do_topk_signature(scores.data_ptr(), _dtype_code(scores), N, E, k, L, bits.data_ptr(), _stream()),
           "do_topk_signature")
    return bits


def do_pairwise_hamming(bits: torch.Tensor, N: int, D: torch.Tensor | None = None) -> torch.Tensor:
    if not isinstance(bits, torch.Tensor) or bits.dim() not in (3, 4) or bits.shape[-1] != 8:
        raise ValueError("bits must be a tensor of shape [U, E, 8] or [L, U, E, 8]")
    if bits.dim() == 3:
        bits = bits.unsqueeze(0)
    L, U, E = bits.shape[0], bits.shape[1], bits.shape[2]
    if U != _units(N):
        raise ValueError(f"bits has {U} units, ceil(N/512) = {_units(N)} for N = {N}")
    _want(bits, "bits", dtypes=_I64)
    if D is None:
        D = alloc_D(L, E, bits.device)
    _want(D, "D", numel=L * E * E, dtypes=_I32)
    _check(lib().do_pairwise_hamming(bits.data_ptr(), N, E, L, D.data_ptr(), _stream()), "do_pairwise_hamming")
    return D


def do_loss(D: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
    if not isinstance(D, torch.Tensor) or D.dim() not in (2, 3) or D.shape[-1] != D.shape[-2]:
        raise ValueError("D must be a tensor of shape [E, E] or [L, E, E]")
    if D.dim() == 2:
        D = D.unsqueeze(0)
    L, E, _ = D.shape
    _want(D, "D", dtypes=_I32)
    if out is None:
        out = alloc_out(L, D.device)
    _want(out, "out", numel=L * LOSS_RESULT_BYTES, dtypes=_U8)
    _check(lib().do_loss(D.data_ptr(), E, L, out.data_ptr(), _stream()), "do_loss")
    return out


def do_fused(scores: torch.Tensor, k: int, want_bits: bool = False, bits: torch.Tensor | None = None,
             D: torch.Tensor | None = None, out: torch.Tensor | None = None):
    L, N, E = _scores_3d(scores)
    if want_bits and bits is None:
        bits = alloc_bits(L, N, E, scores.device)
    if D is None:
        D = alloc_D(L, E, scores.device)
    if out is None:
        out = alloc_out(L, scores.device)
    if bits is not None:
        _want(bits, "bits", numel=L * E * 8 * _units(N), dtypes=_I64)
    _want(D, "D", numel=L * E * E, dtypes=_I32)
    _want(out, "out", numel=L * LOSS_RESULT_BYTES, dtypes=_U8)
    _check(lib().do_fused(scores.data_ptr(), _dtype_code(scores), N, E, k, L,
                          bits.data_ptr() if bits is not None else None, D.data_ptr(), out.data_ptr(), _stream()),
           "do_fused")
    return bits, D, out


def do_surrogate(p: torch.Tensor, k: int, bits: torch.Tensor, D: torch.Tensor, scale: float = 1.0,
                 want_grad: bool = True, loss: torch.Tensor | None = None, grad: torch.Tensor | None = None):
    """Eq. (7) surrogate loss per layer (float64 [L]) and dloss/dp (float32 [L, N, E] or None)."""
    L, N, E = _scores_3d(p, "p")
    _want(bits, "bits", numel=L * E * 8 * _units(N), dtypes=_I64)
    _want(D, "D", numel=L * E * E, dtypes=_I32)
    if loss is None:
        loss = torch.empty(L, dtype=torch.float64, device=p.device)
    if want_grad and grad is None:
        grad = torch.empty((L, N, E), dtype=torch.float32, device=p.device)
    _want(loss, "loss", numel=L, dtypes=(torch.float64,))
    if grad is not None:
        _want(grad, "grad", numel=L * N * E, dtypes=(torch.float32,))
    _check(lib().do_surrogate(p.data_ptr(), _dtype_code(p), N, E, k, L, bits.data_ptr(), D.data_ptr(), float(scale),
                              loss.data_ptr(), grad.data_ptr() if grad is not None else None, _stream()),
           "do_surrogate")
    return loss, grad


def do_load_stats(bits: torch.Tensor, N: int, k: int, p: torch.Tensor | None = None, expert_rank=None,
                  R: int = 0, ld: int = 0, bits_ptr: int | None = None, E: int | None = None, L: int | None = None,
                  loads: torch.Tensor | None = None, out: torch.Tensor | None = None):
    """Per-expert loads (uint32 as int32 [L, E]) and per-layer statistics ([L, 32] bytes, see
    load_stats_records) of signatures `bits` [L, U, E, 8] with U >= ceil(N/512) (or a raw device
    pointer `bits_ptr` with E, L and ld given, e.g. a stream history).  p: routing probabilities
    [L, N, E] or None; expert_rank: host sequence of E ranks in [0, R) or None (one expert per rank)."""
    if bits_ptr is None:
        if not isinstance(bits, torch.Tensor) or bits.dim() not in (3, 4) or bits.shape[-1] != 8:
            raise ValueError("bits must be a tensor of shape [U, E, 8] or [L, U, E, 8]")
        if bits.dim() == 3:
            bits = bits.unsqueeze(0)
        L, E = bits.shape[0], bits.shape[2]
        if bits.shape[1] < _units(N):
            raise ValueError(f"bits has {bits.shape[1]} units, fewer than ceil(N/512) = {_units(N)}")
        if ld == 0:
            ld = 8 * bits.shape[1]  # the tensor's layer stride
        elif ld != 8 * bits.shape[1]:
            raise ValueError(f"ld = {ld} differs from the tensor's {8 * bits.shape[1]} words per expert (0 takes it)")
        _want(bits, "bits", dtypes=_I64)
        ptr = bits.data_ptr()
        dev = bits.device
    else:
        if E is None or L is None:
            raise ValueError("bits_ptr needs E and L")
        ptr = bits_ptr
        dev = torch.device("cuda", torch.cuda.current_device())
    if loads is None:
        loads = torch.empty((L, E), dtype=torch.int32, device=dev)
    if out is None:
        out = torch.empty((L, LOAD_STATS_BYTES), dtype=torch.uint8, device=dev)
    _want(loads, "loads", numel=L * E, dtypes=_I32)
    _want(out, "out", numel=L * LOAD_STATS_BYTES, dtypes=_U8)
    rk = None
    if expert_rank is not None:
        if len(expert_rank) != E:
            raise ValueError(f"expert_rank has {len(expert_rank)} entries, expected E = {E}")
        rk = (ctypes.c_int32 * E)(*[int(r) for r in expert_rank])
    if p is not None:
        _want(p, "p", shape=(L, N, E) if p.dim() == 3 else (N, E), dtypes=_SCORE_DTYPES)
        if p.dim() == 2 and L != 1:
            raise ValueError("p of shape [N, E] needs L = 1")
    pptr, pdt = (p.data_ptr(), _dtype_code(p)) if p is not None else (None, DO_F32)
    _check(lib().do_load_stats(ptr, N, ld, E, k, L, pptr, pdt, rk, R, loads.data_ptr(), out.data_ptr(), _stream()),
           "do_load_stats")
    return loads, out


def load_stats_records(out: torch.Tensor) -> list[dict]:
    """Decode a [L, 32] uint8 tensor of do_load_stats_result records."""
    raw = out.detach().cpu().contiguous().view(torch.uint8).numpy().reshape(-1, LOAD_STATS_BYTES)
    recs = []
    for r in raw:
        u = r[8:16].view("<u4")
        d = r[16:].view("<f8")
        recs.append(dict(total=int(r[:8].view("<u8")[0]), max_load=int(u[0]), min_load=int(u[1]), lbl=float(d[0]),
                         maxvio=float(d[1])))
    return recs


def do_profile_next(start: "torch.cuda.Event | None", stop: "torch.cuda.Event | None"):
    """Bracket the main kernel of this thread's next call with two (recorded-once) torch events."""
    a = ctypes.c_void_p(start.cuda_event) if start is not None else None
    b = ctypes.c_void_p(stop.cuda_event) if stop is not None else None
    _check(lib().do_profile_next(a, b), "do_profile_next")


def do_global_batch_noalloc(score_list, k: int, hist: torch.Tensor | None = None, D: torch.Tensor | None = None,
                            out: torch.Tensor | None = None):
    """do_global_batch_noalloc: the history, distances and loss of one global batch of
    micro-batches (each [n, E] on the device) in one call that allocates nothing in the
    library.  Returns (hist int64 [U, E, 8] with U = ceil(count n / 512), D int32 [E, E], out [1, 40])."""
    if not 1 <= len(score_list) <= 64:
        raise ValueError("do_global_batch_noalloc takes 1 to 64 micro-batches")
    first = score_list[0]
    if not isinstance(first, torch.Tensor) or first.dim() != 2:
        raise ValueError("each micro-batch must be a tensor of shape [n_tokens, E]")
    n, E = first.shape
    for i, t in enumerate(score_list):
        if not isinstance(t, torch.Tensor) or t.shape != first.shape or t.dtype != first.dtype:
            raise ValueError(f"scores[{i}] differs in shape or dtype from scores[0]")
        _want(t, f"scores[{i}]", dtypes=_SCORE_DTYPES)
    U = _units(len(score_list) * n)
    if hist is None:
        hist = torch.empty((U, E, 8), dtype=torch.int64, device=first.device)
    if D is None:
        D = torch.empty((E, E), dtype=torch.int32, device=first.device)
    if out is None:
        out = alloc_out(1, first.device)
    _want(hist, "hist", numel=E * 8 * U, dtypes=_I64)
    _want(D, "D", numel=E * E, dtypes=_I32)
    _want(out, "out", numel=LOSS_RESULT_BYTES, dtypes=_U8)
    ptrs = (ctypes.c_void_p * len(score_list))(*[t.data_ptr() for t in score_list])
    _check(lib().do_global_batch_noalloc(ptrs, _dtype_code(first), n, len(score_list), E, k, hist.data_ptr(),
                                         D.data_ptr(), out.data_ptr(), _stream()), "do_global_batch_noalloc")
    return hist, D, out


REM_MOVE_WORDS = 3  # do_rem_move: 24 bytes = 3 int64 words


def _rank_array(expert_rank, E: int):
    if expert_rank is None or len(expert_rank) != E:
        raise ValueError(f"expert_rank must list the home rank of each of the E = {E} experts")
    return (ctypes.c_int32 * E)(*[int(r) for r in expert_rank])


def do_rem_allocate(expert_tokens: torch.Tensor, expert_rank, R: int, D: int, rank_load: torch.Tensor | None = None,
                    want_state: bool = True):
    """REM Alg. 1 per layer.  expert_tokens: int64 [L, E] (or [E]); expert_rank: host
    sequence of E home ranks; rank_load: int64 [L, R] or None (sum of the volumes).
    Returns (moves int64 [L, R*D, 3] (see rem_records), n_moves int32 [L],
    load_out int64 [L, R] or None, tokens_out int64 [L, E] or None)."""
    if not isinstance(expert_tokens, torch.Tensor) or expert_tokens.dim() not in (1, 2):
        raise ValueError("expert_tokens must be a tensor of shape [E] or [L, E]")
    T = expert_tokens if expert_tokens.dim() == 2 else expert_tokens.unsqueeze(0)
    L, E = T.shape
    _want(T, "expert_tokens", dtypes=_I64)
    if rank_load is not None:
        rank_load = rank_load if rank_load.dim() == 2 else rank_load.unsqueeze(0)
        _want(rank_load, "rank_load", shape=(L, R), dtypes=_I64)
    rk = _rank_array(expert_rank, E)
    dev = T.device
    moves = torch.zeros((L, R * D, REM_MOVE_WORDS), dtype=torch.int64, device=dev)
    n = torch.empty(L, dtype=torch.int32, device=dev)
    lo = torch.empty((L, R), dtype=torch.int64, device=dev) if want_state else None
    to = torch.empty((L, E), dtype=torch.int64, device=dev) if want_state else None
    _check(lib().do_rem_allocate(rank_load.data_ptr() if rank_load is not None else None, T.data_ptr(), rk, E, R, D,
                                 L, moves.data_ptr(), n.data_ptr(), lo.data_ptr() if lo is not None else None,
                                 to.data_ptr() if to is not None else None, _stream()), "do_rem_allocate")
    return moves, n, lo, to


def do_rem_dispatch(replicas: torch.Tensor, n_replicas: torch.Tensor, expert_tokens: torch.Tensor, expert_rank,
                    R: int, D: int, want_state: bool = True):
    """REM Alg. 2 per layer.  replicas: int64 [L, S, 3] assignment records (e.g. the
    moves of do_rem_allocate) with n_replicas int32 [L] valid each; expert_tokens:
    int64 [L, E] volumes of this micro-batch.  Returns (routes int64 [L, R*D, 3],
    n_routes int32 [L], queue_out int64 [L, R] or None, tokens_out int64 [L, E] or None)."""
    if not isinstance(replicas, torch.Tensor) or replicas.dim() != 3 or replicas.shape[2] != REM_MOVE_WORDS:
        raise ValueError("replicas must be a tensor of shape [L, S, 3]")
    L, S = replicas.shape[0], replicas.shape[1]
    _want(replicas, "replicas", dtypes=_I64)
    _want(n_replicas, "n_replicas", shape=(L,), dtypes=_I32)
    T = expert_tokens if expert_tokens.dim() == 2 else expert_tokens.unsqueeze(0)
    if T.shape[0] != L:
        raise ValueError(f"expert_tokens has {T.shape[0]} layers, replicas {L}")
    E = T.shape[1]
    _want(T, "expert_tokens", dtypes=_I64)
    rk = _rank_array(expert_rank, E)
    dev = T.device
    routes = torch.zeros((L, R * D, REM_MOVE_WORDS), dtype=torch.int64, device=dev)
    n = torch.empty(L, dtype=torch.int32, device=dev)
    qo = torch.empty((L, R), dtype=torch.int64, device=dev) if want_state else None
    to = torch.empty((L, E), dtype=torch.int64, device=dev) if want_state else None
    _check(lib().do_rem_dispatch(replicas.data_ptr(), n_replicas.data_ptr(), S, T.data_ptr(), rk, E, R, D, L,
                                 routes.data_ptr(), n.data_ptr(), qo.data_ptr() if qo is not None else None,
                                 to.data_ptr() if to is not None else None, _stream()), "do_rem_dispatch")
    return routes, n, qo, to


def rem_records(moves: torch.Tensor, n: torch.Tensor) -> list:
    """Decode do_rem_move records: per layer a list of (expert, src_rank, dst_rank, tokens),
    or None for a layer whose count is -1 (invalid input)."""
    m = moves.detach().cpu().contiguous().numpy()
    cnt = n.detach().cpu().numpy()
    out = []
    for l in range(m.shape[0]):
        if cnt[l] < 0:
            out.append(None)
            continue
        w = m[l, :cnt[l]]
        out.append([(int(a) & 0xFFFFFFFF, (int(a) >> 32) & 0xFFFFFFFF, int(b) & 0xFFFFFFFF, int(c)) for a, b, c in w])
    return out


class DoStream:
    """Streaming global-batch signature history (do_stream_*)."""

    def __init__(self, E: int, k: int, capacity_tokens: int):
        h = ctypes.c_void_p()
        _check(lib().do_stream_create(E, k, capacity_tokens, ctypes.byref(h)), "do_stream_create")
        self.h, self.E, self.k, self.capacity = h, E, k, capacity_tokens

    def _micro_batch(self, scores: torch.Tensor, name: str = "scores") -> int:
        if not isinstance(scores, torch.Tensor) or scores.dim() != 2:
            raise ValueError(f"{name} must be a tensor of shape [n_tokens, E]")
        if scores.shape[1] != self.E:
            raise ValueError(f"{name} has {scores.shape[1]} experts, the history has E = {self.E}")
        _want(scores, name, dtypes=_SCORE_DTYPES)
        return scores.shape[0]

    def append(self, scores: torch.Tensor):
        N = self._micro_batch(scores)
        _check(lib().do_stream_append(self.h, scores.data_ptr(), _dtype_code(scores), N, _stream()),
               "do_stream_append")

    def append_many(self, score_list):
        if not 1 <= len(score_list) <= 64:
            raise ValueError("append_many takes 1 to 64 micro-batches")
        N = self._micro_batch(score_list[0], "scores[0]")
        for i, t in enumerate(score_list[1:], 1):
            self._micro_batch(t, f"scores[{i}]")
            if t.shape != score_list[0].shape or t.dtype != score_list[0].dtype:
                raise ValueError(f"scores[{i}] differs in shape or dtype from scores[0]")
        ptrs = (ctypes.c_void_p * len(score_list))(*[s.data_ptr() for s in score_list])
        _check(lib().do_stream_append_many(self.h, ptrs, _dtype_code(score_list[0]), N, len(score_list), _stream()),
               "do_stream_append_many")

    def finalize(self, D: torch.Tensor | None = None, out: torch.Tensor | None = None):
        # the caller's buffers are checked before any is allocated
        if D is not None:
            _want(D, "D", numel=self.E * self.E, dtypes=_I32)
        if out is not None:
            _want(out, "out", numel=LOSS_RESULT_BYTES, dtypes=_U8)
        if D is None:
            D = torch.empty((self.E, self.E), dtype=torch.int32, device=torch.cuda.current_device())
        if out is None:
            out = alloc_out(1, torch.device("cuda", torch.cuda.current_device()))
        _check(lib().do_stream_finalize(self.h, D.data_ptr(), out.data_ptr(), _stream()), "do_stream_finalize")
        return D, out

    def reset(self):
        _check(lib().do_stream_reset(self.h, _stream()), "do_stream_reset")

    @property
    def tokens(self) -> int:
        return int(lib().do_stream_tokens(self.h))

    @property
    def words_per_expert(self) -> int:
        return int(lib().do_stream_words_per_expert(self.h))

    def bits_ptr(self) -> int:
        return int(lib().do_stream_bits(self.h) or 0)

    def history(self) -> torch.Tensor:
        """Copy of the signature history [words_per_expert / 8, E, 8] (int64 words, signature layout)."""
        W = self.words_per_expert
        out = torch.empty((W // 8, self.E, 8), dtype=torch.int64,
                          device=torch.device("cuda", torch.cuda.current_device()))
        _check(_hip_copy_d2d(out.data_ptr(), self.bits_ptr(), self.E * W * 8), "history copy")
        return out

    def close(self):
        if self.h is not None and self.h.value:
            _check(lib().do_stream_destroy(self.h), "do_stream_destroy")
        self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
