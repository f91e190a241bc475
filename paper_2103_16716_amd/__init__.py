"""Balanced token-to-expert assignment of BASE layers on AMD Instinct MI355X.

Python binding of the C ABI in include/base.h (libbase_mi355x.so, built from
csrc/ by `python -m paper_2103_16716_amd.build`). The functions below only
marshal torch tensors into the C calls; every step of the path runs in the
library's HIP kernels. There is no fallback: if the library is missing or
fails to load, every call raises.

    S = affinity(H, W)                 # Sec. 3.1 / Eq. 2: S[t, e] = h_t . w_e
    res = assign(S)                    # Sec. 3.2.1 / Eq. 2: balanced assignment
    X = permute(H, res.perm)           # Fig. 2: rows grouped by expert
    Y = permute(X, res.perm, inverse=True)   # Sec. 3: back to token order
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbase_mi355x.so")

# Status codes and enums of include/base.h.
BASE_OK = 0
BASE_ERR_INVALID_ARG = -1
BASE_ERR_NOT_DIVISIBLE = -2
BASE_ERR_UNSUPPORTED_DTYPE = -3
BASE_ERR_NONFINITE = -4
BASE_ERR_NOT_CONVERGED = -5
BASE_ERR_WORKSPACE = -6
BASE_ERR_HIP = -7
BASE_ERR_RANGE = -8
BASE_ERR_INTERNAL = -9

BASE_F32 = 0
BASE_BF16 = 1
BASE_I16 = 2

BASE_ASSIGN_GREEDY_FALLBACK = 1
BASE_ASSIGN_SYNC_STATS = 2
BASE_ASSIGN_CHECK_FINITE = 4
BASE_ASSIGN_WARM_PRICES = 8
BASE_ASSIGN_FULL_SCHEDULE = 16

# Every symbol include/base.h declares.
EXPORTED = ("base_status_string", "base_affinity", "base_affinity_gather",
            "base_assign_workspace_size", "base_assign", "base_assign_batched_workspace_size",
            "base_assign_batched", "base_assign_status", "base_assign_noalloc", "base_permute", "base_permute_batched",
            "base_greedy_workspace_size", "base_greedy_assign", "base_gate_combine",
            "base_gate_combine_batched", "base_gate_backward", "base_timing_enable",
            "base_timing_read")


class AssignOpts(ctypes.Structure):
    _fields_ = [("eps_final", ctypes.c_double), ("eps_initial", ctypes.c_double),
                ("eps_factor", ctypes.c_double), ("max_rounds", ctypes.c_int32),
                ("flags", ctypes.c_uint32)]


class AssignStats(ctypes.Structure):
    _fields_ = [("phases", ctypes.c_int32), ("rounds", ctypes.c_int32), ("bids", ctypes.c_int64),
                ("eps_final", ctypes.c_double), ("fell_back", ctypes.c_int32),
                ("dual_gap", ctypes.c_double), ("converged", ctypes.c_int32),
                ("engine_bids", ctypes.c_int64), ("eps_last", ctypes.c_double),
                ("certified", ctypes.c_int32), ("augmentations", ctypes.c_int32)]


class BaseError(RuntimeError):
    """A non-zero status returned by the library."""

    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run `python -m paper_2103_16716_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        L.base_status_string.argtypes = [i32]
        L.base_status_string.restype = ctypes.c_char_p
        L.base_affinity.argtypes = [vp, vp, vp, i64, i64, i64, i32, vp]
        L.base_affinity.restype = i32
        L.base_affinity_gather.argtypes = [vp, i64, vp, vp, vp, i64, i64, i64, i32, vp]
        L.base_affinity_gather.restype = i32
        L.base_assign_workspace_size.argtypes = [i64, i64]
        L.base_assign_workspace_size.restype = ctypes.c_size_t
        L.base_assign.argtypes = [vp, i32, i64, i64, ctypes.POINTER(AssignOpts), vp, vp, vp, vp,
                                  ctypes.c_size_t, ctypes.POINTER(AssignStats), vp]
        L.base_assign.restype = i32
        L.base_assign_batched_workspace_size.argtypes = [i64, i64, i64]
        L.base_assign_batched_workspace_size.restype = ctypes.c_size_t
        L.base_assign_batched.argtypes = [vp, i32, i64, i64, i64, ctypes.POINTER(AssignOpts), vp,
                                          vp, vp, vp, ctypes.c_size_t,
                                          ctypes.POINTER(AssignStats), vp]
        L.base_assign_batched.restype = i32
        L.base_assign_noalloc.argtypes = [vp, i32, i64, i64, ctypes.POINTER(AssignOpts), vp, vp,
                                          vp, ctypes.POINTER(AssignStats), vp]
        L.base_assign_noalloc.restype = i32
        L.base_assign_status.argtypes = [vp, i64, i64, i64, ctypes.POINTER(AssignStats), vp]
        L.base_assign_status.restype = i32
        L.base_permute.argtypes = [vp, vp, vp, i64, i64, i32, i32, vp]
        L.base_permute.restype = i32
        L.base_permute_batched.argtypes = [vp, vp, vp, vp, i64, i64, i64, i32, i32, vp]
        L.base_permute_batched.restype = i32
        L.base_greedy_workspace_size.argtypes = [i64, i64]
        L.base_greedy_workspace_size.restype = ctypes.c_size_t
        L.base_greedy_assign.argtypes = [vp, i64, i64, vp, vp, vp, vp, ctypes.c_size_t, vp]
        L.base_greedy_assign.restype = i32
        L.base_gate_combine.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, i32, vp]
        L.base_gate_combine.restype = i32
        L.base_gate_combine_batched.argtypes = [vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, i64,
                                                i32, vp]
        L.base_gate_combine_batched.restype = i32
        L.base_gate_backward.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, i64, i64,
                                         i64, i32, vp]
        L.base_gate_backward.restype = i32
        L.base_timing_enable.argtypes = [ctypes.c_int32]
        L.base_timing_enable.restype = i32
        L.base_timing_read.argtypes = [ctypes.POINTER(i64), ctypes.POINTER(ctypes.c_double)]
        L.base_timing_read.restype = i32
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().base_status_string(int(status)).decode()


def _check(status: int, where: str) -> None:
    if status != BASE_OK:
        raise BaseError(status, where)


def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return BASE_BF16
    if t.dtype == torch.float32:
        return BASE_F32
    if t.dtype == torch.int16:
        return BASE_I16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream_ptr(stream) -> int:
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def _need_device(*ts) -> None:
    for t in ts:
        if not t.is_cuda:
            raise ValueError("tensors must be on the GPU")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")


def affinity(H, W, out=None, rows=None, stream=None):
    """S = H . W^T as float32 [T, E] (base_affinity). With `rows` (int32 [N]),
    S[i] = H[rows[i]] . W^T, N rows (base_affinity_gather: the shuffle of
    tokens to workers read through the index)."""
    torch = _torch()
    _need_device(H, W)
    T, d = H.shape
    E, d2 = W.shape
    if d != d2 or H.dtype != W.dtype:
        raise ValueError("H [T, d] and W [E, d] must share d and dtype")
    N = T if rows is None else rows.numel()
    if out is None:
        out = torch.empty((N, E), dtype=torch.float32, device=H.device)
    _need_device(out)
    if rows is None:
        _check(lib().base_affinity(H.data_ptr(), W.data_ptr(), out.data_ptr(), T, E, d,
                                   _dtype_code(H), _stream_ptr(stream)), "base_affinity")
    else:
        _need_device(rows)
        if rows.dtype != torch.int32:
            raise TypeError("rows must be int32")
        _check(lib().base_affinity_gather(H.data_ptr(), T, rows.data_ptr(), W.data_ptr(),
                                          out.data_ptr(), N, E, d, _dtype_code(H),
                                          _stream_ptr(stream)), "base_affinity_gather")
    return out


def assign_workspace_size(T: int, E: int) -> int:
    return int(lib().base_assign_workspace_size(T, E))


@dataclasses.dataclass
class AssignResult:
    assign: object      # int32 [T]
    perm: object        # int32 [T]
    prices: object      # float32 [E] (int64 [E] in integer mode)
    stats: AssignStats | None


def assign(S, *, eps_final: float = 0.0, eps_initial: float = 0.0, eps_factor: float = 0.0,
           max_rounds: int = 0, flags: int = 0, sync_stats: bool = True, workspace=None,
           out_assign=None, out_perm=None, out_prices=None, warm_start: bool = False,
           stream=None) -> AssignResult:
    """Balanced assignment of Eq. 2 (base_assign). Zero-valued options take
    the library defaults. With sync_stats (the default) the call waits for the
    solve and returns its statistics; pass False to keep it asynchronous.
    With warm_start the solve starts from the prices in out_prices (required;
    overwritten with the result)."""
    if warm_start:
        if out_prices is None:
            raise ValueError("warm_start needs out_prices holding the starting prices")
        flags |= BASE_ASSIGN_WARM_PRICES
    torch = _torch()
    _need_device(S)
    T, E = S.shape
    dev = S.device
    integer = S.dtype == torch.int16
    if out_assign is None:
        out_assign = torch.empty(T, dtype=torch.int32, device=dev)
    if out_perm is None:
        out_perm = torch.empty(T, dtype=torch.int32, device=dev)
    if out_prices is None:
        out_prices = torch.empty(E, dtype=torch.int64 if integer else torch.float32, device=dev)
    ws_bytes = assign_workspace_size(T, E)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    opts = AssignOpts(eps_final, eps_initial, eps_factor, max_rounds,
                      flags | (BASE_ASSIGN_SYNC_STATS if sync_stats else 0))
    stats = AssignStats()
    _check(lib().base_assign(S.data_ptr(), _dtype_code(S), T, E, ctypes.byref(opts),
                             out_assign.data_ptr(), out_perm.data_ptr(), out_prices.data_ptr(),
                             workspace.data_ptr(), workspace.numel(), ctypes.byref(stats),
                             _stream_ptr(stream)), "base_assign")
    return AssignResult(out_assign, out_perm, out_prices, stats if sync_stats else None)


def assign_batched_workspace_size(B: int, T: int, E: int) -> int:
    return int(lib().base_assign_batched_workspace_size(B, T, E))


def assign_batched(S, *, eps_final: float = 0.0, eps_initial: float = 0.0,
                   eps_factor: float = 0.0, max_rounds: int = 0, flags: int = 0,
                   sync_stats: bool = True, workspace=None, out_assign=None, out_perm=None,
                   out_prices=None, stream=None) -> AssignResult:
    """B independent balanced assignments of Eq. 2, S [B, T, E]
    (base_assign_batched); outputs [B, T] and prices [B, E]. Statistics are
    aggregated over the problems."""
    torch = _torch()
    _need_device(S)
    B, T, E = S.shape
    dev = S.device
    integer = S.dtype == torch.int16
    if out_assign is None:
        out_assign = torch.empty((B, T), dtype=torch.int32, device=dev)
    if out_perm is None:
        out_perm = torch.empty((B, T), dtype=torch.int32, device=dev)
    if out_prices is None:
        out_prices = torch.empty((B, E), dtype=torch.int64 if integer else torch.float32,
                                 device=dev)
    ws_bytes = assign_batched_workspace_size(B, T, E)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    opts = AssignOpts(eps_final, eps_initial, eps_factor, max_rounds,
                      flags | (BASE_ASSIGN_SYNC_STATS if sync_stats else 0))
    stats = AssignStats()
    _check(lib().base_assign_batched(S.data_ptr(), _dtype_code(S), B, T, E, ctypes.byref(opts),
                                     out_assign.data_ptr(), out_perm.data_ptr(),
                                     out_prices.data_ptr(), workspace.data_ptr(),
                                     workspace.numel(), ctypes.byref(stats), _stream_ptr(stream)),
           "base_assign_batched")
    return AssignResult(out_assign, out_perm, out_prices, stats if sync_stats else None)


NOALLOC_MAX_WORKSPACE = 32 << 20   # BASE_ASSIGN_NOALLOC_MAX_WORKSPACE


def assign_noalloc(S, *, eps_final: float = 0.0, eps_initial: float = 0.0,
                   eps_factor: float = 0.0, max_rounds: int = 0, flags: int = 0,
                   sync_stats: bool = True, out_assign, out_perm, out_prices=None,
                   stream=None) -> AssignResult:
    """base_assign_noalloc: the solve of `assign` on the library's own
    per-device workspace array; allocates nothing (the outputs are the
    caller's, and must be given)."""
    _need_device(S, out_assign, out_perm)
    T, E = S.shape
    opts = AssignOpts(eps_final, eps_initial, eps_factor, max_rounds,
                      flags | (BASE_ASSIGN_SYNC_STATS if sync_stats else 0))
    stats = AssignStats()
    _check(lib().base_assign_noalloc(S.data_ptr(), _dtype_code(S), T, E, ctypes.byref(opts),
                                     out_assign.data_ptr(), out_perm.data_ptr(),
                                     0 if out_prices is None else out_prices.data_ptr(),
                                     ctypes.byref(stats), _stream_ptr(stream)),
           "base_assign_noalloc")
    return AssignResult(out_assign, out_perm, out_prices, stats if sync_stats else None)


def assign_status(workspace, T: int, E: int, B: int = 1, stream=None):
    """How the last solve on `workspace` ended (base_assign_status): waits
    for the stream and returns (status code, AssignStats) without raising.
    dual_gap is NaN (not measured by this read)."""
    _need_device(workspace)
    stats = AssignStats()
    st = lib().base_assign_status(workspace.data_ptr(), B, T, E, ctypes.byref(stats),
                                  _stream_ptr(stream))
    return int(st), stats


def permute(x, perm, inverse: bool = False, out=None, stream=None):
    """Gather rows into expert order (out[k] = x[perm[k]]) or, with inverse,
    scatter them back (out[perm[k]] = x[k]) (base_permute)."""
    torch = _torch()
    _need_device(x, perm)
    T, d = x.shape
    if out is None:
        out = torch.empty_like(x)
    _need_device(out)
    _check(lib().base_permute(x.data_ptr(), perm.data_ptr(), out.data_ptr(), T, d, _dtype_code(x),
                              1 if inverse else 0, _stream_ptr(stream)), "base_permute")
    return out


def permute_batched(x, perm, shuffle=None, inverse: bool = False, out=None, stream=None):
    """Permute of B problems in one pass (base_permute_batched): x [B*T, d],
    perm [B, T]; routed row k = b*T + j has source src = shuffle[b*T +
    perm[b, j]] (or b*T + perm[b, j]); out[k] = x[src], or with inverse
    out[src] = x[k]."""
    torch = _torch()
    _need_device(x, perm)
    B, T = perm.shape
    N, d = x.shape
    if N != B * T:
        raise ValueError("x must have B*T rows")
    if out is None:
        out = torch.empty_like(x)
    _need_device(out)
    sp = 0
    if shuffle is not None:
        _need_device(shuffle)
        if shuffle.numel() != N or shuffle.dtype != torch.int32:
            raise ValueError("shuffle must be int32 [B*T]")
        sp = shuffle.data_ptr()
    _check(lib().base_permute_batched(x.data_ptr(), perm.data_ptr(), sp or None, out.data_ptr(),
                                      B, T, d, _dtype_code(x), 1 if inverse else 0,
                                      _stream_ptr(stream)), "base_permute_batched")
    return out


def greedy_assign(S, workspace=None, stream=None, out_assign=None, out_perm=None,
                  out_offsets=None):
    """Test-time routing (base_greedy_assign): (assign [T], perm [T],
    offsets [E + 1]) with every token at its best expert. The out_* tensors
    (int32, contiguous, on S's device), when given, receive the results, so
    a loop of calls allocates nothing."""
    torch = _torch()
    _need_device(S)
    T, E = S.shape
    dev = S.device

    def out(x, n):
        if x is None:
            return torch.empty(n, dtype=torch.int32, device=dev)
        if x.dtype != torch.int32 or x.numel() != n or not x.is_contiguous() or x.device != dev:
            raise ValueError(f"greedy_assign: an output needs {n} contiguous int32 on {dev}")
        return x

    a = out(out_assign, T)
    perm = out(out_perm, T)
    offsets = out(out_offsets, E + 1)
    n = int(lib().base_greedy_workspace_size(T, E))
    if workspace is None:
        workspace = torch.empty(max(n, 256), dtype=torch.uint8, device=dev)
    _check(lib().base_greedy_assign(S.data_ptr(), T, E, a.data_ptr(), perm.data_ptr(),
                                    offsets.data_ptr(), workspace.data_ptr(), workspace.numel(),
                                    _stream_ptr(stream)), "base_greedy_assign")
    return a, perm, offsets


def gate_combine(F, H, S, assign, perm, out=None, stream=None):
    """Eq. 1 fused into the return to token order (base_gate_combine):
    out[t] = sigmoid(S[t, assign[t]]) * F[k] + H[t] for t = perm[k]."""
    torch = _torch()
    _need_device(F, H, S, assign, perm)
    T, d = H.shape
    E = S.shape[1]
    if out is None:
        out = torch.empty_like(H)
    _check(lib().base_gate_combine(F.data_ptr(), H.data_ptr(), S.data_ptr(), assign.data_ptr(),
                                   perm.data_ptr(), out.data_ptr(), T, E, d, _dtype_code(H),
                                   _stream_ptr(stream)), "base_gate_combine")
    return out


def gate_combine_batched(F, H, S, assign, perm, shuffle=None, out=None, stream=None):
    """Eq. 1 over B problems (base_gate_combine_batched): S [B*T, E], assign
    and perm [B, T] in worker order, F [B*T, d] in routed order, H and the
    result [B*T, d] in the unshuffled token order."""
    torch = _torch()
    _need_device(F, H, S, assign, perm)
    B, T = perm.shape
    N, d = H.shape
    E = S.shape[-1]
    if N != B * T or S.numel() != N * E or F.shape != H.shape:
        raise ValueError("shapes: F, H [B*T, d], S [B*T, E], assign and perm [B, T]")
    if out is None:
        out = torch.empty_like(H)
    sp = 0
    if shuffle is not None:
        _need_device(shuffle)
        if shuffle.numel() != N or shuffle.dtype != torch.int32:
            raise ValueError("shuffle must be int32 [B*T]")
        sp = shuffle.data_ptr()
    _check(lib().base_gate_combine_batched(F.data_ptr(), H.data_ptr(), S.data_ptr(),
                                           assign.data_ptr(), perm.data_ptr(), sp or None,
                                           out.data_ptr(), B, T, E, d, _dtype_code(H),
                                           _stream_ptr(stream)), "base_gate_combine_batched")
    return out


def balanced_offsets(T: int, E: int, device):
    """Routed-order row ranges of a balanced assignment: offsets[e] = e * T/E."""
    torch = _torch()
    return torch.arange(E + 1, dtype=torch.int32).mul_(T // E).to(device)


def gate_backward(dY, F, H, W, S, assign, perm, offsets=None, stream=None):
    """Gradient of Eq. 1's gate and residual (base_gate_backward): returns
    (dH, dF in routed order, dW float32, dS float32)."""
    torch = _torch()
    _need_device(dY, F, H, W, S, assign, perm)
    T, d = H.shape
    E = W.shape[0]
    if offsets is None:
        offsets = balanced_offsets(T, E, H.device)
    dH = torch.empty_like(H)
    dF = torch.empty_like(F)
    dW = torch.empty((E, d), dtype=torch.float32, device=H.device)
    dS = torch.empty(T, dtype=torch.float32, device=H.device)
    _check(lib().base_gate_backward(dY.data_ptr(), F.data_ptr(), H.data_ptr(), W.data_ptr(),
                                    S.data_ptr(), assign.data_ptr(), perm.data_ptr(),
                                    offsets.data_ptr(), dH.data_ptr(), dF.data_ptr(),
                                    dW.data_ptr(), dS.data_ptr(), T, E, d, _dtype_code(H),
                                    _stream_ptr(stream)), "base_gate_backward")
    return dH, dF, dW, dS


def timing_enable(capacity: int) -> None:
    """Start recording event timings of the engine kernel's launches
    (base_timing_enable); capacity <= 0 stops and frees the record."""
    _check(lib().base_timing_enable(int(capacity)), "base_timing_enable")


def timing_read() -> tuple[int, float]:
    """(recorded engine launches, their summed milliseconds); clears the
    record (base_timing_read)."""
    n = ctypes.c_int64()
    ms = ctypes.c_double()
    _check(lib().base_timing_read(ctypes.byref(n), ctypes.byref(ms)), "base_timing_read")
    return int(n.value), float(ms.value)


__all__ = ["affinity", "assign", "assign_batched", "permute", "permute_batched", "greedy_assign",
           "gate_combine", "gate_combine_batched",
           "gate_backward", "balanced_offsets", "assign_workspace_size",
           "assign_batched_workspace_size", "timing_enable",
           "timing_read", "AssignResult", "AssignOpts", "AssignStats", "BaseError", "lib",
           "assign_status", "assign_noalloc", "NOALLOC_MAX_WORKSPACE",
           "status_string", "EXPORTED"]
