"""Python binding of libemb (the C ABI in include/emb.h).

Argument marshalling only: every step of the hot path runs in the HIP kernels
of libemb.so.  PyTorch supplies device memory and the stream
(torch.cuda.current_stream()).  There is no fallback: if the library is not
built, importing this package raises.

torch is imported before the library is loaded so that the process maps a
single HIP runtime (the one torch ships), which the library then shares.
"""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (must be loaded before libemb.so; see module docstring)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libemb.so")

EMB_OK = 0
EMB_ERR_INVALID_ARG = 1
EMB_ERR_WORKSPACE = 2
EMB_ERR_LAUNCH = 3
EMB_ERR_UNSUPPORTED = 4
EMB_F32 = 0
EMB_BF16 = 1
EMB_DEV_ID_OUT_OF_RANGE = 1
EMB_DEV_OWNER_OUT_OF_RANGE = 2
EMB_DEV_STALLED = 4
EMB_COMM_ALLTOALL = 0
EMB_COMM_ALLREDUCE = 1
EMB_COMM_PS = 2
EMB_COMM_ALLGATHER = 3
EMB_ADAM_COEFFS_WORDS = 8

# (name, restype, argtypes) of every symbol include/emb.h declares.
_P, _I32, _I64, _SZ, _D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_double
SIGNATURES = {
    "emb_abi_version": (ctypes.c_int, []),
    "emb_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "emb_gather": (ctypes.c_int, [_P, _I64, _I32, _P, _I32, _P, _P, _P]),
    "emb_grad_coalesce_workspace_bytes": (_SZ, [_I32, _I64, _I32, _I32]),
    "emb_grad_coalesce": (ctypes.c_int, [_P, _I32, _P, _I32, _I32, _I64, _P, _P, _P, _P, _P, _SZ, _P, _P]),
    "emb_grad_coalesce_by_owner": (ctypes.c_int, [_P, _I32, _P, _I32, _I32, _I64, _P, _I32, _P, _P, _P, _P, _P, _P,
                                                  _P, _SZ, _P, _P]),
    "emb_grad_coalesce_by_owner_noalloc": (ctypes.c_int, [_P, _I32, _P, _I32, _I32, _I64, _P, _I32, _P, _P, _P, _P,
                                                          _P, _P, _P, _P]),
    "emb_grad_coalesce_split_workspace_bytes": (_SZ, [_I32, _I32, _I64, _I32, _I32]),
    "emb_grad_coalesce_split": (ctypes.c_int, [_P, _I32, _P, _I32, _P, _I32, _I32, _I64, _P, _I32, _P, _P, _P, _P, _P,
                                               _P, _P, _SZ, _P, _P]),
    "emb_lookup_request_workspace_bytes": (_SZ, [_I32, _I64]),
    "emb_lookup_request": (ctypes.c_int, [_P, _I32, _I64, _P, _I32, _P, _P, _P, _P, _P, _P, _SZ, _P, _P]),
    "emb_exchange_simulated": (ctypes.c_int, [_P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _P, _P]),
    "emb_receive_merge": (ctypes.c_int, [_P, _P, _P, _I32, _I32, _I64, _P, _I32, _P, _P, _P, _P, _P, _P, _P, _SZ,
                                         _P, _P]),
    "emb_pack_by_owner_workspace_bytes": (_SZ, [_I32, _I32]),
    "emb_pack_by_owner": (ctypes.c_int, [_P, _P, _P, _I32, _I32, _P, _I64, _I32, _P, _P, _P, _P, _P, _SZ, _P, _P]),
    "emb_sparse_adam_apply": (ctypes.c_int, [_P, _P, _P, _I64, _I32, _P, _P, _P, _I32, _I32, _I32, _I32,
                                             _D, _D, _D, _D, _I64, _P, _P]),
    "emb_adam_coeffs": (ctypes.c_int, [_D, _D, _D, _D, _I64, _P]),
    "emb_pack_by_column": (ctypes.c_int, [_P, _P, _I32, _I32, _I32, _P, _P, _P]),
    "emb_gather_by_column": (ctypes.c_int, [_P, _I64, _I32, _I32, _P, _I32, _P, _P, _P]),
    "emb_assemble_by_column": (ctypes.c_int, [_P, _I64, _I64, _I32, _I32, _I32, _P, _P]),
    "emb_comm_cost": (ctypes.c_int, [_I32, _I64, _I64, _D, _D, _D, _D, ctypes.POINTER(ctypes.c_double)]),
    "emb_event_create": (ctypes.c_int, [ctypes.POINTER(ctypes.c_void_p), _I32]),
    "emb_event_destroy": (ctypes.c_int, [_P]),
    "emb_event_elapsed_ms": (ctypes.c_int, [_P, _P, ctypes.POINTER(ctypes.c_float)]),
    "emb_step_signals_create": (ctypes.c_int, [ctypes.POINTER(ctypes.c_void_p)]),
    "emb_step_signals_destroy": (ctypes.c_int, [_P]),
    "emb_train_step": (ctypes.c_int, [_P, _P]),
    "emb_step_queue_create": (ctypes.c_int, [ctypes.POINTER(ctypes.c_void_p)]),
    "emb_step_queue_flush": (ctypes.c_int, [_P]),
    "emb_step_queue_destroy": (ctypes.c_int, [_P]),
    "emb_train_step_queued": (ctypes.c_int, [_P, _P, _P]),
}


class StepSchedule(ctypes.Structure):
    """emb_step_schedule of include/emb.h."""
    _fields_ = [("lookup_update", _P), ("coalesce", _P), ("pack", _P), ("delayed", _P), ("sorted", _P),
                ("coalesced", _P), ("packed", _P), ("updated", _P), ("gathered", _P), ("delayed_done", _P),
                ("reuse", _I32), ("by_owner", _I32), ("split", _I32), ("timing", _P * 8), ("signals", _P), ("sets", _I32)]


class StepArgs(ctypes.Structure):
    """emb_step_args of include/emb.h."""
    _fields_ = [("table", _P), ("exp_avg", _P), ("exp_avg_sq", _P), ("V", _I64), ("D", _I32),
                ("row_owner", _P), ("P", _I32), ("ids", _P), ("T", _I32), ("next_ids", _P), ("T_next", _I32),
                ("grad", _P), ("grad_dtype", _I32),
                ("cap_rows", _I32), ("lookup", _P), ("uniq_ids", _P), ("seg_offsets", _P), ("num_unique", _P),
                ("uniq_grad", _P), ("send_ids", _P), ("send_counts", _P), ("send_offsets", _P), ("send_rows", _P),
                ("ws_coalesce", _P), ("ws_coalesce_bytes", _SZ), ("ws_pack", _P), ("ws_pack_bytes", _SZ),
                ("lr", _D), ("beta1", _D), ("beta2", _D), ("eps", _D), ("step", _I64), ("dev_status", _P),
                ("adam_coeffs", _P)]


class EmbError(RuntimeError):
    pass


def _load_library():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2110_09132_amd/build.py (hipcc, gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load_library()


def abi_version() -> int:
    return lib.emb_abi_version()


def status_string(status: int) -> str:
    return lib.emb_status_string(status).decode()


def _check(status: int, what: str):
    if status != EMB_OK:
        raise EmbError(f"{what}: {status_string(status)} ({status})")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t):
    if t.dtype == torch.float32:
        return EMB_F32
    if t.dtype == torch.bfloat16:
        return EMB_BF16
    raise EmbError(f"gradient dtype {t.dtype} is not float32 or bfloat16")


def _need(t, dtype, what):
    if t.dtype != dtype or not t.is_cuda or not t.is_contiguous():
        raise EmbError(f"{what} must be a contiguous {dtype} CUDA tensor (got {t.dtype}, {t.device})")


def _out(t, dtype, n, what):
    """An output (or input) buffer the call reads or writes n elements of."""
    _need(t, dtype, what)
    if t.numel() < n:
        raise EmbError(f"{what} holds {t.numel()} elements; the call uses {n}")


def _rows(t, n, D, what):
    """A row buffer of at least n rows of width D (2-D [>= n, D], or flat with >= n * D elements)."""
    if t.dim() == 2 and t.shape[1] != D:
        raise EmbError(f"{what} has rows of {t.shape[1]} elements; the call uses {D}")
    if t.numel() < n * D:
        raise EmbError(f"{what} holds {t.numel()} elements; the call uses {n} rows of {D}")


def _grad(grad, T, what="grad"):
    """The per-token gradient [T, D] (fp32 or bf16); returns (dtype code, D)."""
    code = _dtype_code(grad)
    if not grad.is_cuda or not grad.is_contiguous() or grad.dim() != 2:
        raise EmbError(f"{what} must be a contiguous 2-D CUDA tensor")
    if grad.shape[0] != T:
        raise EmbError(f"{what} has {grad.shape[0]} rows for {T} tokens")
    return code, grad.shape[1]


class Event:
    """A HIP event made by the library (emb_event_create); destroyed with the object."""

    def __init__(self, timing: bool = False):
        h = ctypes.c_void_p()
        _check(lib.emb_event_create(ctypes.byref(h), 1 if timing else 0), "emb_event_create")
        self.handle = h.value
        self._lib = lib

    def elapsed_ms(self, end: "Event") -> float:
        ms = ctypes.c_float()
        _check(lib.emb_event_elapsed_ms(self.handle, end.handle, ctypes.byref(ms)), "emb_event_elapsed_ms")
        return float(ms.value)

    def __del__(self):
        if getattr(self, "handle", None):
            self._lib.emb_event_destroy(self.handle)
            self.handle = None


class StepSignals:
    """Step signals of one table (emb_step_signals_create); handed back to the library's pool when
    the object goes away (only once the steps enqueued with it have completed)."""

    def __init__(self):
        h = ctypes.c_void_p()
        _check(lib.emb_step_signals_create(ctypes.byref(h)), "emb_step_signals_create")
        self.handle = h.value
        self._lib = lib

    def __del__(self):
        if getattr(self, "handle", None):
            self._lib.emb_step_signals_destroy(self.handle)
            self.handle = None


class StepQueue:
    """Two-thread enqueue of owner-major steps (emb_step_queue_create): emb_train_step_queued
    enqueues a step's sort and reduction on the calling thread and hands its lookup and update to
    the library's worker thread.  flush() returns once the worker has enqueued everything handed
    to it (the steps then run in stream order like any other work); the worker is stopped when
    the object goes away."""

    def __init__(self):
        h = ctypes.c_void_p()
        _check(lib.emb_step_queue_create(ctypes.byref(h)), "emb_step_queue_create")
        self.handle = h.value
        self._lib = lib

    def flush(self):
        _check(self._lib.emb_step_queue_flush(self.handle), "emb_step_queue_flush")

    def __del__(self):
        if getattr(self, "handle", None):
            self._lib.emb_step_queue_destroy(self.handle)
            self.handle = None


def new_status(device=None):
    """A zeroed device status word for the dev_status argument."""
    return torch.zeros(1, dtype=torch.int32, device=device or "cuda")


def gather(table, ids, out=None, dev_status=None, stream=None):
    """out[t] = table[ids[t]] (emb_gather)."""
    _need(table, torch.float32, "table")
    _need(ids, torch.int32, "ids")
    if table.dim() != 2:
        raise EmbError("table must be 2-D [V, D]")
    V, D = table.shape
    T = ids.numel()
    if out is None:
        out = torch.empty((T, D), dtype=torch.float32, device=table.device)
    _out(out, torch.float32, 0, "out")
    _rows(out, T, D, "out")
    _check(lib.emb_gather(_ptr(table), V, D, _ptr(ids), T, _ptr(out), _ptr(dev_status), _stream(stream)),
           "emb_gather")
    return out


def grad_coalesce_workspace_bytes(T, V, D, grad_dtype=EMB_F32) -> int:
    return int(lib.emb_grad_coalesce_workspace_bytes(T, V, D, grad_dtype))


def new_workspace(nbytes, device=None):
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device or "cuda")


def _coalesce_outs(uniq_ids, seg_offsets, uniq_grad, num_unique, T, D):
    _out(uniq_ids, torch.int32, T, "uniq_ids")
    _out(seg_offsets, torch.int32, T + 1, "seg_offsets")
    _out(uniq_grad, torch.float32, 0, "uniq_grad")
    _rows(uniq_grad, T, D, "uniq_grad")
    _out(num_unique, torch.int32, 1, "num_unique")


def _owners(row_owner, V, P):
    _need(row_owner, torch.int32, "row_owner")
    if row_owner.numel() < V:
        raise EmbError(f"row_owner holds {row_owner.numel()} owners for V = {V} rows")
    if not 1 <= P <= 1024:
        raise EmbError(f"P = {P} is outside [1, 1024]")


def grad_coalesce(ids, grad, V, out=None, workspace=None, dev_status=None, stream=None):
    """COALESCE + UNIQUE (emb_grad_coalesce).

    Returns (uniq_ids [T], seg_offsets [T+1], uniq_grad [T, D], num_unique [1]); the
    first num_unique entries are meaningful.  `out` may pass those four tensors in.
    """
    _need(ids, torch.int32, "ids")
    T = ids.numel()
    code, D = _grad(grad, T)
    dev = ids.device
    if out is None:
        out = (torch.empty(T, dtype=torch.int32, device=dev), torch.empty(T + 1, dtype=torch.int32, device=dev),
               torch.empty((T, D), dtype=torch.float32, device=dev), torch.empty(1, dtype=torch.int32, device=dev))
    uniq_ids, seg_offsets, uniq_grad, num_unique = out
    _coalesce_outs(uniq_ids, seg_offsets, uniq_grad, num_unique, T, D)
    nbytes = grad_coalesce_workspace_bytes(T, V, D, code)
    if workspace is None:
        workspace = new_workspace(nbytes, dev)
    _check(lib.emb_grad_coalesce(_ptr(ids), T, _ptr(grad), code, D, V, _ptr(uniq_ids), _ptr(seg_offsets),
                                 _ptr(uniq_grad), _ptr(num_unique), _ptr(workspace), workspace.numel(),
                                 _ptr(dev_status), _stream(stream)), "emb_grad_coalesce")
    return out


def grad_coalesce_by_owner(ids, grad, V, row_owner, P, out=None, workspace=None, dev_status=None, stream=None):
    """Coalesce straight into the owner-major send layout (emb_grad_coalesce_by_owner).

    Returns (send_ids [T], seg_offsets [T+1], send_rows [T, D], send_counts [P], send_offsets [P+1],
    num_unique [1]); `out` may pass those six tensors in.
    """
    _need(ids, torch.int32, "ids")
    _owners(row_owner, V, P)
    T = ids.numel()
    code, D = _grad(grad, T)
    dev = ids.device
    if out is None:
        out = (torch.empty(T, dtype=torch.int32, device=dev), torch.empty(T + 1, dtype=torch.int32, device=dev),
               torch.empty((T, D), dtype=torch.float32, device=dev), torch.empty(P, dtype=torch.int32, device=dev),
               torch.empty(P + 1, dtype=torch.int32, device=dev), torch.empty(1, dtype=torch.int32, device=dev))
    send_ids, seg_offsets, send_rows, send_counts, send_offsets, num_unique = out
    _coalesce_outs(send_ids, seg_offsets, send_rows, num_unique, T, D)
    _out(send_counts, torch.int32, P, "send_counts")
    _out(send_offsets, torch.int32, P + 1, "send_offsets")
    if workspace is None:
        workspace = new_workspace(grad_coalesce_workspace_bytes(T, V, D, code), dev)
    _check(lib.emb_grad_coalesce_by_owner(_ptr(ids), T, _ptr(grad), code, D, V, _ptr(row_owner), P, _ptr(send_ids),
                                          _ptr(seg_offsets), _ptr(send_rows), _ptr(send_counts), _ptr(send_offsets),
                                          _ptr(num_unique), _ptr(workspace), workspace.numel(), _ptr(dev_status),
                                          _stream(stream)), "emb_grad_coalesce_by_owner")
    return out


NOALLOC_SCRATCH_BYTES = 16 << 20  # EMB_NOALLOC_SCRATCH_BYTES


def grad_coalesce_by_owner_noalloc(ids, grad, V, row_owner, P, out, dev_status=None, stream=None):
    """grad_coalesce_by_owner without a workspace (emb_grad_coalesce_by_owner_noalloc: the library's
    static device array serves as the workspace; calls that may overlap on one device race on it).
    `out` passes the six output tensors in (nothing is allocated here either)."""
    _need(ids, torch.int32, "ids")
    _owners(row_owner, V, P)
    T = ids.numel()
    code, D = _grad(grad, T)
    send_ids, seg_offsets, send_rows, send_counts, send_offsets, num_unique = out
    _coalesce_outs(send_ids, seg_offsets, send_rows, num_unique, T, D)
    _out(send_counts, torch.int32, P, "send_counts")
    _out(send_offsets, torch.int32, P + 1, "send_offsets")
    _check(lib.emb_grad_coalesce_by_owner_noalloc(_ptr(ids), T, _ptr(grad), code, D, V, _ptr(row_owner), P,
                                                  _ptr(send_ids), _ptr(seg_offsets), _ptr(send_rows),
                                                  _ptr(send_counts), _ptr(send_offsets), _ptr(num_unique),
                                                  _ptr(dev_status), _stream(stream)),
           "emb_grad_coalesce_by_owner_noalloc")
    return out


def grad_coalesce_split_workspace_bytes(T, T_next, V, D, grad_dtype=EMB_F32) -> int:
    return int(lib.emb_grad_coalesce_split_workspace_bytes(T, T_next, V, D, grad_dtype))


def grad_coalesce_split(ids, next_ids, grad, V, row_owner, P, out=None, workspace=None, dev_status=None,
                        stream=None):
    """Coalesce into the send layout with the prior / delayed split (emb_grad_coalesce_split).

    Returns (send_ids [T], seg_offsets [T+1], send_rows [T, D], send_counts [2P], send_offsets [2P+1],
    num_unique [1]); groups 0 .. P-1 hold the prior rows, P .. 2P-1 the delayed rows.
    """
    _need(ids, torch.int32, "ids")
    _need(next_ids, torch.int32, "next_ids")
    _owners(row_owner, V, P)
    T, T_next = ids.numel(), next_ids.numel()
    code, D = _grad(grad, T)
    dev = ids.device
    if out is None:
        out = (torch.empty(T, dtype=torch.int32, device=dev), torch.empty(T + 1, dtype=torch.int32, device=dev),
               torch.empty((T, D), dtype=torch.float32, device=dev),
               torch.empty(2 * P, dtype=torch.int32, device=dev),
               torch.empty(2 * P + 1, dtype=torch.int32, device=dev), torch.empty(1, dtype=torch.int32, device=dev))
    send_ids, seg_offsets, send_rows, send_counts, send_offsets, num_unique = out
    _coalesce_outs(send_ids, seg_offsets, send_rows, num_unique, T, D)
    _out(send_counts, torch.int32, 2 * P, "send_counts")
    _out(send_offsets, torch.int32, 2 * P + 1, "send_offsets")
    if workspace is None:
        workspace = new_workspace(grad_coalesce_split_workspace_bytes(T, T_next, V, D, code), dev)
    _check(lib.emb_grad_coalesce_split(_ptr(ids), T, _ptr(next_ids), T_next, _ptr(grad), code, D, V,
                                       _ptr(row_owner), P, _ptr(send_ids), _ptr(seg_offsets), _ptr(send_rows),
                                       _ptr(send_counts), _ptr(send_offsets), _ptr(num_unique), _ptr(workspace),
                                       workspace.numel(), _ptr(dev_status), _stream(stream)),
           "emb_grad_coalesce_split")
    return out


def lookup_request_workspace_bytes(T, V) -> int:
    return int(lib.emb_lookup_request_workspace_bytes(T, V))


def lookup_request(ids, V, row_owner, P, out=None, workspace=None, dev_status=None, stream=None):
    """A worker's requests to the row owners (emb_lookup_request).

    Returns (req_ids [T], req_counts [P], req_offsets [P+1], num_unique [1], inverse [T]); `out`
    may pass those five tensors in."""
    _need(ids, torch.int32, "ids")
    _owners(row_owner, V, P)
    T = ids.numel()
    dev = ids.device
    if out is None:
        out = (torch.empty(T, dtype=torch.int32, device=dev), torch.empty(P, dtype=torch.int32, device=dev),
               torch.empty(P + 1, dtype=torch.int32, device=dev), torch.empty(1, dtype=torch.int32, device=dev),
               torch.empty(T, dtype=torch.int32, device=dev))
    req_ids, counts, offsets, nu, inverse = out
    for t, n, what in ((req_ids, T, "req_ids"), (counts, P, "req_counts"), (offsets, P + 1, "req_offsets"),
                       (nu, 1, "num_unique"), (inverse, T, "inverse")):
        _out(t, torch.int32, n, what)
    if workspace is None:
        workspace = new_workspace(lookup_request_workspace_bytes(T, V), dev)
    _check(lib.emb_lookup_request(_ptr(ids), T, V, _ptr(row_owner), P, _ptr(req_ids), _ptr(counts), _ptr(offsets),
                                  _ptr(nu), _ptr(inverse), _ptr(workspace), workspace.numel(), _ptr(dev_status),
                                  _stream(stream)), "emb_lookup_request")
    return out


def exchange_simulated(send_ids, send_rows, send_offsets, out=None, stream=None):
    """Simulated AlltoAll of P workers' send layouts (emb_exchange_simulated).

    send_ids [P, cap], send_rows [P, cap, D] or None (ids only), send_offsets [P, P+1].  Returns
    (recv_ids [P*cap], recv_rows [P*cap, D] or None, recv_offsets [P, P+1], recv_total [1])."""
    _need(send_ids, torch.int32, "send_ids")
    if send_rows is not None:
        _need(send_rows, torch.float32, "send_rows")
    _need(send_offsets, torch.int32, "send_offsets")
    if send_ids.dim() != 2:
        raise EmbError("send_ids must be 2-D [P, cap]")
    P, cap = send_ids.shape
    D = send_rows.shape[-1] if send_rows is not None else 0
    if send_rows is not None:
        _rows(send_rows, P * cap, D, "send_rows")
    _out(send_offsets, torch.int32, P * (P + 1), "send_offsets")
    dev = send_ids.device
    if out is None:
        out = (torch.empty(P * cap, dtype=torch.int32, device=dev),
               torch.empty((P * cap, D), dtype=torch.float32, device=dev) if D else None,
               torch.empty((P, P + 1), dtype=torch.int32, device=dev), torch.empty(1, dtype=torch.int32, device=dev))
    recv_ids, recv_rows, recv_offsets, recv_total = out
    _out(recv_ids, torch.int32, P * cap, "recv_ids")
    if D:
        _out(recv_rows, torch.float32, 0, "recv_rows")
        _rows(recv_rows, P * cap, D, "recv_rows")
    _out(recv_offsets, torch.int32, P * (P + 1), "recv_offsets")
    _out(recv_total, torch.int32, 1, "recv_total")
    _check(lib.emb_exchange_simulated(_ptr(send_ids), _ptr(send_rows), _ptr(send_offsets), P, cap, D, _ptr(recv_ids),
                                      _ptr(recv_rows), _ptr(recv_offsets), _ptr(recv_total), _stream(stream)),
           "emb_exchange_simulated")
    return out


def receive_merge(recv_ids, recv_rows, recv_total, V, row_owner, P, out=None, workspace=None, dev_status=None,
                  stream=None):
    """Owner-major coalesce of the first recv_total received rows (emb_receive_merge).

    Returns (merged_ids, seg_offsets, merged_rows, merged_counts [P], merged_offsets [P+1], num_unique)."""
    _need(recv_ids, torch.int32, "recv_ids")
    _need(recv_rows, torch.float32, "recv_rows")
    _need(recv_total, torch.int32, "recv_total")
    _owners(row_owner, V, P)
    cap = recv_ids.numel()
    if recv_rows.dim() != 2:
        raise EmbError("recv_rows must be 2-D [cap, D]")
    D = recv_rows.shape[1]
    _rows(recv_rows, cap, D, "recv_rows")
    dev = recv_ids.device
    if out is None:
        out = (torch.empty(cap, dtype=torch.int32, device=dev), torch.empty(cap + 1, dtype=torch.int32, device=dev),
               torch.empty((cap, D), dtype=torch.float32, device=dev), torch.empty(P, dtype=torch.int32, device=dev),
               torch.empty(P + 1, dtype=torch.int32, device=dev), torch.empty(1, dtype=torch.int32, device=dev))
    merged_ids, seg, rows, counts, offs, nu = out
    _coalesce_outs(merged_ids, seg, rows, nu, cap, D)
    _out(counts, torch.int32, P, "merged_counts")
    _out(offs, torch.int32, P + 1, "merged_offsets")
    if workspace is None:
        workspace = new_workspace(grad_coalesce_workspace_bytes(cap, V, D, EMB_F32), dev)
    _check(lib.emb_receive_merge(_ptr(recv_ids), _ptr(recv_rows), _ptr(recv_total), cap, D, V, _ptr(row_owner), P,
                                 _ptr(merged_ids), _ptr(seg), _ptr(rows), _ptr(counts), _ptr(offs), _ptr(nu),
                                 _ptr(workspace), workspace.numel(), _ptr(dev_status), _stream(stream)),
           "emb_receive_merge")
    return out


def pack_by_owner_workspace_bytes(cap_rows, P) -> int:
    return int(lib.emb_pack_by_owner_workspace_bytes(cap_rows, P))


def pack_by_owner(uniq_ids, uniq_grad, num_unique, row_owner, P, out=None, workspace=None, dev_status=None,
                  stream=None):
    """Owner-major send buffers (emb_pack_by_owner).

    Returns (send_ids [cap], send_rows [cap, D], send_counts [P], send_offsets [P+1]).
    """
    _need(uniq_ids, torch.int32, "uniq_ids")
    _need(uniq_grad, torch.float32, "uniq_grad")
    _need(num_unique, torch.int32, "num_unique")
    _need(row_owner, torch.int32, "row_owner")
    cap = uniq_ids.numel()
    if uniq_grad.dim() != 2:
        raise EmbError("uniq_grad must be 2-D [cap, D]")
    D = uniq_grad.shape[1]
    _rows(uniq_grad, cap, D, "uniq_grad")
    _out(num_unique, torch.int32, 1, "num_unique")
    V = row_owner.numel()
    dev = uniq_ids.device
    if out is None:
        out = (torch.empty(cap, dtype=torch.int32, device=dev), torch.empty((cap, D), dtype=torch.float32, device=dev),
               torch.empty(P, dtype=torch.int32, device=dev), torch.empty(P + 1, dtype=torch.int32, device=dev))
    send_ids, send_rows, send_counts, send_offsets = out
    _out(send_ids, torch.int32, cap, "send_ids")
    _out(send_rows, torch.float32, 0, "send_rows")
    _rows(send_rows, cap, D, "send_rows")
    _out(send_counts, torch.int32, P, "send_counts")
    _out(send_offsets, torch.int32, P + 1, "send_offsets")
    if workspace is None:
        workspace = new_workspace(pack_by_owner_workspace_bytes(cap, P), dev)
    _check(lib.emb_pack_by_owner(_ptr(uniq_ids), _ptr(uniq_grad), _ptr(num_unique), cap, D, _ptr(row_owner), V, P,
                                 _ptr(send_ids), _ptr(send_rows), _ptr(send_counts), _ptr(send_offsets),
                                 _ptr(workspace), workspace.numel(), _ptr(dev_status), _stream(stream)),
           "emb_pack_by_owner")
    return out


def column_offsets(D, P):
    """First float column of every owner of the column-wise partition, [P + 1]: floor(p * D / P)."""
    return [(p * D) // P for p in range(P + 1)]


def column_block(blocks, C, D, P, p):
    """View of block p ([C, w(p)]) of a flat column-block layout of capacity C."""
    off = column_offsets(D, P)
    return blocks[C * off[p]:C * off[p + 1]].view(C, off[p + 1] - off[p])


def pack_by_column(rows, P, num_rows=None, out=None, stream=None):
    """Column-block layout of the rows (emb_pack_by_column).

    rows [cap, D]; packs the first *num_rows rows (device int32 [1]) or all of them.
    Returns (blocks [cap * D] flat, send_counts [P])."""
    _need(rows, torch.float32, "rows")
    if num_rows is not None:
        _out(num_rows, torch.int32, 1, "num_rows")
    if rows.dim() != 2:
        raise EmbError("rows must be 2-D [cap, D]")
    cap, D = rows.shape
    dev = rows.device
    if out is None:
        out = (torch.empty(cap * D, dtype=torch.float32, device=dev), torch.empty(P, dtype=torch.int32, device=dev))
    blocks, counts = out
    _out(blocks, torch.float32, cap * D, "blocks")
    if counts is not None:
        _out(counts, torch.int32, P, "send_counts")
    _check(lib.emb_pack_by_column(_ptr(rows), _ptr(num_rows), cap, D, P, _ptr(blocks), _ptr(counts), _stream(stream)),
           "emb_pack_by_column")
    return out


def gather_by_column(shards, V, D, P, ids, out=None, dev_status=None, stream=None):
    """Every owner's lookup of ids in its shard (emb_gather_by_column).

    shards: flat column-block layout of capacity V.  Returns blocks [T * D] flat (capacity T)."""
    _need(shards, torch.float32, "shards")
    _need(ids, torch.int32, "ids")
    _out(shards, torch.float32, V * D, "shards")
    T = ids.numel()
    if out is None:
        out = torch.empty(T * D, dtype=torch.float32, device=ids.device)
    _out(out, torch.float32, T * D, "out")
    _check(lib.emb_gather_by_column(_ptr(shards), V, D, P, _ptr(ids), T, _ptr(out), _ptr(dev_status),
                                    _stream(stream)), "emb_gather_by_column")
    return out


def assemble_by_column(blocks, C, D, P, row0=0, R=None, out=None, stream=None):
    """Rows [row0, row0 + R) of a column-block layout of capacity C, joined (emb_assemble_by_column)."""
    _need(blocks, torch.float32, "blocks")
    _out(blocks, torch.float32, C * D, "blocks")
    R = C - row0 if R is None else R
    if out is None:
        out = torch.empty((R, D), dtype=torch.float32, device=blocks.device)
    _out(out, torch.float32, 0, "out")
    _rows(out, max(R, 0), D, "out")
    _check(lib.emb_assemble_by_column(_ptr(blocks), C, row0, R, D, P, _ptr(out), _stream(stream)),
           "emb_assemble_by_column")
    return out


def comm_cost(scheme, N, M, alpha, B, beta, S=1) -> float:
    """Table 2 communication cost of one exchange (emb_comm_cost); host arithmetic."""
    r = ctypes.c_double()
    _check(lib.emb_comm_cost(scheme, N, S, float(M), float(alpha), float(B), float(beta), ctypes.byref(r)),
           "emb_comm_cost")
    return r.value


def adam_coeffs(lr, beta1, beta2, eps, step, out):
    """Write step `step`'s update coefficients (emb_adam_coeffs) into `out`, a float32 CPU tensor of
    EMB_ADAM_COEFFS_WORDS elements (for instance a row of a pinned buffer)."""
    if out.dtype != torch.float32 or out.device.type != "cpu" or not out.is_contiguous() or \
            out.numel() < EMB_ADAM_COEFFS_WORDS:
        raise EmbError(f"out must be a contiguous float32 CPU tensor of {EMB_ADAM_COEFFS_WORDS} elements")
    _check(lib.emb_adam_coeffs(lr, beta1, beta2, eps, step, out.data_ptr()), "emb_adam_coeffs")
    return out


def sparse_adam_apply(table, exp_avg, exp_avg_sq, row_ids, rows, offsets, P, shard_begin, shard_end, lr, beta1,
                      beta2, eps, step, dev_status=None, stream=None):
    """Row-wise Adam on rows [offsets[shard_begin], offsets[shard_end]) (emb_sparse_adam_apply)."""
    for t, n in ((table, "table"), (exp_avg, "exp_avg"), (exp_avg_sq, "exp_avg_sq"), (rows, "rows")):
        _need(t, torch.float32, n)
    _need(row_ids, torch.int32, "row_ids")
    _need(offsets, torch.int32, "offsets")
    if table.dim() != 2:
        raise EmbError("table must be 2-D [V, D]")
    V, D = table.shape
    for t, n in ((exp_avg, "exp_avg"), (exp_avg_sq, "exp_avg_sq")):
        if t.shape != table.shape:
            raise EmbError(f"{n} has shape {tuple(t.shape)}, the table {tuple(table.shape)}")
    _rows(rows, row_ids.numel(), D, "rows")
    _out(offsets, torch.int32, max(P, 0) + 1, "offsets")
    _check(lib.emb_sparse_adam_apply(_ptr(table), _ptr(exp_avg), _ptr(exp_avg_sq), V, D, _ptr(row_ids), _ptr(rows),
                                     _ptr(offsets), P, shard_begin, shard_end, row_ids.numel(), float(lr),
                                     float(beta1), float(beta2), float(eps), int(step), _ptr(dev_status),
                                     _stream(stream)), "emb_sparse_adam_apply")
