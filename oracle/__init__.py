"""ctypes wrapper of the C oracle -- TEST INFRASTRUCTURE ONLY.

Only the tests, `__graft_entry__.smoke()` and the CPU-baseline leg of
`bench.py` may import this package.  The product (the GPU library and its
Python binding) never does.  See oracle.h for the contract of each function
and the passage of the paper it follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "oracle.c")


def build(verbose: bool = False) -> str:
    """Compile oracle.c with gcc (plain C99, -O2, no fast-math)."""
    cmd = ["gcc", "-std=c99", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-o", LIB_PATH + ".tmp", SRC_PATH, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB_PATH + ".tmp", LIB_PATH)
    return LIB_PATH


_lib = None


def build_variant(src_text: str, out_path: str) -> str:
    """Compile an edited copy of oracle.c (used by tests that plant a mistake in
    the oracle to show that the pins catch it)."""
    src = out_path + ".c"
    with open(src, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc", "-std=c99", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fPIC", "-shared",
                    "-I", _HERE, "-o", out_path, src, "-lm"], check=True)
    return out_path


def use_library(path: str | None):
    """Point the wrapper at another build of the oracle (None: the default one)."""
    global _lib
    _lib = None if path is None else _bind(ctypes.CDLL(path))


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(SRC_PATH):
        build()
    _lib = _bind(ctypes.CDLL(LIB_PATH))
    return _lib


def _bind(lib):
    P, I64, I32, D = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double
    lib.orc_gather.argtypes = [P, I64, I64, P, I64, P]
    lib.orc_gather.restype = I64
    lib.orc_coalesce.argtypes = [P, I64, P, I32, I64, I64, P, P, P, P, P, P]
    lib.orc_coalesce.restype = I64
    lib.orc_pack_by_owner.argtypes = [P, P, I64, I64, P, I64, I32, P, P, P, P]
    lib.orc_pack_by_owner.restype = I64
    lib.orc_vertical_split.argtypes = [P, I64, P, I64, P]
    lib.orc_vertical_split.restype = I64
    lib.orc_sparse_adam.argtypes = [P, P, P, I64, I64, P, P, P, I32, I32, D, D, D, D, I64]
    lib.orc_sparse_adam.restype = I64
    lib.orc_lookup_request.argtypes = [P, I64, I64, P, I32, P, P, P, P]
    lib.orc_lookup_request.restype = I64
    lib.orc_pack_by_column.argtypes = [P, I64, I64, I64, I32, P]
    lib.orc_pack_by_column.restype = None
    lib.orc_gather_by_column.argtypes = [P, I64, I64, I32, P, I64, P]
    lib.orc_gather_by_column.restype = I64
    lib.orc_assemble_by_column.argtypes = [P, I64, I64, I64, I64, I32, P]
    lib.orc_assemble_by_column.restype = None
    lib.orc_comm_cost.argtypes = [I32, I64, I64, D, D, D, D]
    lib.orc_comm_cost.restype = D
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def gather(W, ids):
    """out[t] = W[ids[t]] (zero row for an out-of-range id); returns (out, n_invalid)."""
    W = _c(W, np.float32)
    ids = _c(ids, np.int32)
    V, D = W.shape
    out = np.empty((ids.size, D), dtype=np.float32)
    bad = _load().orc_gather(_ptr(W), V, D, _ptr(ids), ids.size, _ptr(out))
    return out, int(bad)


def coalesce(ids, grad, V, grad_is_bf16=False, want_f64=True):
    """COALESCE + UNIQUE.  grad: fp32 [T, D] or uint16 bf16 bits [T, D].

    Returns dict(uniq_ids, seg_offsets, uniq_grad, sum_f64, absum, U, n_invalid).
    """
    ids = _c(ids, np.int32)
    T = ids.size
    grad = _c(grad, np.uint16 if grad_is_bf16 else np.float32)
    D = grad.shape[1] if grad.ndim == 2 else (grad.size // T if T else 0)
    if grad.ndim != 2:
        grad = grad.reshape(T, D)
    uniq_ids = np.empty(max(T, 1), dtype=np.int32)
    seg = np.empty(T + 1, dtype=np.int32)
    ug = np.empty((max(T, 1), D), dtype=np.float32)
    s64 = np.empty((max(T, 1), D), dtype=np.float64) if want_f64 else None
    ab = np.empty((max(T, 1), D), dtype=np.float64) if want_f64 else None
    nbad = ctypes.c_int64(0)
    U = _load().orc_coalesce(_ptr(ids), T, _ptr(grad), 1 if grad_is_bf16 else 0, D, V,
                             _ptr(uniq_ids), _ptr(seg), _ptr(ug), _ptr(s64), _ptr(ab),
                             ctypes.byref(nbad))
    return dict(uniq_ids=uniq_ids[:U].copy(), seg_offsets=seg[:U + 1].copy(), uniq_grad=ug[:U].copy(),
                sum_f64=None if s64 is None else s64[:U].copy(),
                absum=None if ab is None else ab[:U].copy(), U=int(U), n_invalid=int(nbad.value))


def pack_by_owner(uniq_ids, uniq_grad, row_owner, P):
    """Owner-major stable pack.  Returns dict(send_ids, send_rows, send_counts, send_offsets, n_dropped)."""
    uniq_ids = _c(uniq_ids, np.int32)
    U = uniq_ids.size
    uniq_grad = _c(uniq_grad, np.float32).reshape(U, -1) if U else _c(uniq_grad, np.float32)
    D = uniq_grad.shape[1] if uniq_grad.ndim == 2 else 0
    row_owner = _c(row_owner, np.int32)
    send_ids = np.empty(max(U, 1), dtype=np.int32)
    send_rows = np.empty((max(U, 1), max(D, 1)), dtype=np.float32)
    counts = np.empty(P, dtype=np.int32)
    offs = np.empty(P + 1, dtype=np.int32)
    bad = _load().orc_pack_by_owner(_ptr(uniq_ids), _ptr(uniq_grad), U, D, _ptr(row_owner),
                                    row_owner.size, P, _ptr(send_ids), _ptr(send_rows), _ptr(counts),
                                    _ptr(offs))
    n = int(offs[P])
    return dict(send_ids=send_ids[:n].copy(), send_rows=send_rows[:n, :D].copy(), send_counts=counts,
                send_offsets=offs, n_dropped=int(bad))


def vertical_split(uniq_ids, next_ids):
    """Set split of Algorithm 1: is_prior[k] = uniq_ids[k] in next_ids.  Returns (is_prior bool [U], n_prior)."""
    uniq_ids = _c(uniq_ids, np.int32)
    next_ids = _c(next_ids, np.int32)
    is_prior = np.empty(max(uniq_ids.size, 1), dtype=np.int32)
    n = _load().orc_vertical_split(_ptr(uniq_ids), uniq_ids.size, _ptr(next_ids), next_ids.size, _ptr(is_prior))
    return is_prior[:uniq_ids.size].astype(bool), int(n)


def split_pack(uniq_ids, uniq_grad, next_ids, row_owner, P):
    """Algorithm 1's INDEX_SELECT of the prior and delayed rows, each packed by owner (pack_by_owner),
    laid out one after the other: groups g = 0 .. 2P-1, prior owner p is g = p, delayed owner p is
    g = P + p.  Returns dict(send_ids, send_rows, send_counts [2P], send_offsets [2P+1], n_prior,
    is_prior, n_dropped)."""
    uniq_ids = _c(uniq_ids, np.int32)
    uniq_grad = _c(uniq_grad, np.float32).reshape(uniq_ids.size, -1)
    is_prior, n_prior = vertical_split(uniq_ids, next_ids)
    pp = pack_by_owner(uniq_ids[is_prior], uniq_grad[is_prior], row_owner, P)
    pd = pack_by_owner(uniq_ids[~is_prior], uniq_grad[~is_prior], row_owner, P)
    np_ = int(pp["send_offsets"][P])
    return dict(send_ids=np.concatenate([pp["send_ids"], pd["send_ids"]]),
                send_rows=np.concatenate([pp["send_rows"], pd["send_rows"]]),
                send_counts=np.concatenate([pp["send_counts"], pd["send_counts"]]),
                send_offsets=np.concatenate([pp["send_offsets"], pd["send_offsets"][1:] + np_]).astype(np.int32),
                n_prior=n_prior, is_prior=is_prior, n_dropped=pp["n_dropped"] + pd["n_dropped"])


def sparse_adam(W, m, v, row_ids, rows, offsets, shard_begin, shard_end, lr, beta1, beta2, eps, step):
    """In-place row-wise Adam on W, m, v (fp32 [V, D] C-contiguous arrays).  Returns #skipped rows."""
    for a in (W, m, v):
        assert a.dtype == np.float32 and a.flags.c_contiguous and a.ndim == 2
    V, D = W.shape
    row_ids = _c(row_ids, np.int32)
    rows = _c(rows, np.float32)
    offsets = _c(offsets, np.int32)
    return int(_load().orc_sparse_adam(_ptr(W), _ptr(m), _ptr(v), V, D, _ptr(row_ids), _ptr(rows),
                                       _ptr(offsets), int(shard_begin), int(shard_end), float(lr),
                                       float(beta1), float(beta2), float(eps), int(step)))


def pack_by_column(rows, P, C=None):
    """Column-block layout of capacity C (default: the row count) of rows [R, D]; flat float32 [C * D].
    Entries of rows >= R stay NaN."""
    rows = _c(rows, np.float32)
    R, D = rows.shape
    C = R if C is None else C
    blocks = np.full(C * D, np.nan, dtype=np.float32)
    _load().orc_pack_by_column(_ptr(rows), R, C, D, P, _ptr(blocks))
    return blocks


def gather_by_column(shards, V, D, P, ids):
    """Every owner's lookup of ids in its shard; returns (blocks flat [T * D], n_invalid)."""
    shards = _c(shards, np.float32).reshape(-1)
    ids = _c(ids, np.int32)
    blocks = np.empty(ids.size * D, dtype=np.float32)
    bad = _load().orc_gather_by_column(_ptr(shards), V, D, P, _ptr(ids), ids.size, _ptr(blocks))
    return blocks, int(bad)


def assemble_by_column(blocks, C, D, P, row0=0, R=None):
    """Rows [row0, row0 + R) of a column-block layout of capacity C, joined into [R, D]."""
    blocks = _c(blocks, np.float32).reshape(-1)
    R = C - row0 if R is None else R
    rows = np.empty((R, D), dtype=np.float32)
    _load().orc_assemble_by_column(_ptr(blocks), C, row0, R, D, P, _ptr(rows))
    return rows


COMM_SCHEMES = {"alltoall": 0, "allreduce": 1, "ps": 2, "allgather": 3}


def comm_cost(scheme, N, M, alpha, B, beta, S=1):
    """Table 2 cost of one exchange by scheme name (alltoall, allreduce, ps, allgather)."""
    return float(_load().orc_comm_cost(COMM_SCHEMES[scheme], N, S, float(M), float(alpha), float(B), float(beta)))


def lookup_request(ids, V, row_owner, P):
    """Owner-grouped distinct ids of a batch and each token's index in them (-1: takes no part).

    Returns dict(req_ids [U], req_counts [P], req_offsets [P+1], inverse [T], U)."""
    ids = _c(ids, np.int32)
    row_owner = _c(row_owner, np.int32)
    T = ids.size
    req_ids = np.empty(max(T, 1), np.int32)
    counts = np.empty(P, np.int32)
    offs = np.empty(P + 1, np.int32)
    inv = np.empty(max(T, 1), np.int32)
    U = int(_load().orc_lookup_request(_ptr(ids), T, V, _ptr(row_owner), P, _ptr(req_ids), _ptr(counts), _ptr(offs),
                                       _ptr(inv)))
    return dict(req_ids=req_ids[:U], req_counts=counts, req_offsets=offs, inverse=inv[:T], U=U)
