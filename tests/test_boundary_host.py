"""The C ABI library without a GPU: it loads, exports every symbol that
include/emb.h declares, and rejects bad arguments on the host before anything
is enqueued (no device memory is touched by these calls)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2110_09132_amd as emb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "emb.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(emb_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_four_calls():
    names = declared_functions()
    for n in ("emb_gather", "emb_grad_coalesce", "emb_pack_by_owner", "emb_sparse_adam_apply"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(emb.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} declared in emb.h but not exported"
        assert name in emb.SIGNATURES, f"{name} has no binding signature"


def test_status_strings_and_version():
    assert emb.abi_version() == 3
    assert emb.status_string(emb.EMB_OK) == "ok"
    assert "workspace" in emb.status_string(emb.EMB_ERR_WORKSPACE)


FAKE = ctypes.c_void_p(4096)  # never dereferenced: every call below fails validation first
NULL = None


def test_gather_validation():
    L = emb.lib
    assert L.emb_gather(NULL, 10, 4, NULL, 5, NULL, NULL, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_gather(FAKE, 0, 4, FAKE, 5, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG  # V < 1
    assert L.emb_gather(FAKE, 1 << 31, 4, FAKE, 5, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_gather(FAKE, 10, 0, FAKE, 5, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG  # D < 1
    assert L.emb_gather(FAKE, 10, 4, FAKE, -1, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_gather(NULL, 10, 4, NULL, 0, NULL, NULL, NULL) == emb.EMB_OK  # T == 0: no-op


def test_coalesce_validation_and_workspace_query():
    L = emb.lib
    need = L.emb_grad_coalesce_workspace_bytes(1000, 5000, 64, emb.EMB_F32)
    assert need > 0 and need % 256 == 0
    assert L.emb_grad_coalesce_workspace_bytes(1000, 5000, 64, 7) == 0
    assert L.emb_grad_coalesce_workspace_bytes(-1, 5000, 64, 0) == 0
    args = lambda T=1000, dtype=0, D=64, V=5000, ws=FAKE, wsb=need: (
        FAKE, T, FAKE, dtype, D, V, FAKE, FAKE, FAKE, FAKE, ws, wsb, NULL, NULL)
    assert L.emb_grad_coalesce(*args(wsb=need - 1)) == emb.EMB_ERR_WORKSPACE
    assert L.emb_grad_coalesce(*args(dtype=3)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce(*args(D=0)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce(*args(V=0)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce(*args(T=-2)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce(*args(ws=NULL)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce(*args(ws=ctypes.c_void_p(4096 + 64))) == emb.EMB_ERR_INVALID_ARG  # misaligned
    # misaligned fp32 gradient rows
    assert L.emb_grad_coalesce(FAKE, 1000, ctypes.c_void_p(4098), 0, 64, 5000, FAKE, FAKE, FAKE, FAKE, FAKE,
                               need, NULL, NULL) == emb.EMB_ERR_INVALID_ARG


def test_coalesce_by_owner_validation():
    L = emb.lib
    need = L.emb_grad_coalesce_workspace_bytes(1000, 5000, 64, emb.EMB_F32)
    args = lambda T=1000, D=64, V=5000, own=FAKE, P=4, ids=FAKE, counts=FAKE, offs=FAKE, wsb=need: (
        ids, T, FAKE, 0, D, V, own, P, FAKE, FAKE, FAKE, counts, offs, FAKE, FAKE, wsb, NULL, NULL)
    assert L.emb_grad_coalesce_by_owner(*args(wsb=need - 1)) == emb.EMB_ERR_WORKSPACE
    assert L.emb_grad_coalesce_by_owner(*args(P=0)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce_by_owner(*args(P=1025)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce_by_owner(*args(own=NULL)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce_by_owner(*args(counts=NULL)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce_by_owner(*args(offs=NULL)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce_by_owner(*args(ids=NULL)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce_by_owner(*args(D=0)) == emb.EMB_ERR_INVALID_ARG
    # (owner, id) keys must fit 32 bits: bits(V) + bits(P).  The key check comes before the
    # workspace check, so a short workspace tells the two apart without launching anything.
    short = dict(wsb=need - 1)
    assert L.emb_grad_coalesce_by_owner(*args(V=(1 << 31) - 1, P=2, **short)) == emb.EMB_ERR_WORKSPACE
    assert L.emb_grad_coalesce_by_owner(*args(V=(1 << 31) - 1, P=3, **short)) == emb.EMB_ERR_UNSUPPORTED
    assert L.emb_grad_coalesce_by_owner(*args(V=1 << 22, P=1024, **short)) == emb.EMB_ERR_WORKSPACE
    assert L.emb_grad_coalesce_by_owner(*args(V=(1 << 22) + 1, P=1024, **short)) == emb.EMB_ERR_UNSUPPORTED


def test_coalesce_by_owner_noalloc_size_limit():
    # the allocation-free call refuses, on the host, a batch whose workspace exceeds its static array
    L = emb.lib
    assert emb.NOALLOC_SCRATCH_BYTES == 16 << 20
    T, D, V, P = 65536, 4096, 1 << 20, 16
    assert L.emb_grad_coalesce_workspace_bytes(T, V, D, emb.EMB_F32) > emb.NOALLOC_SCRATCH_BYTES
    assert L.emb_grad_coalesce_by_owner_noalloc(FAKE, T, FAKE, 0, D, V, FAKE, P, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                                NULL, NULL) == emb.EMB_ERR_WORKSPACE
    # the largest workload batches fit
    for T, V, D, g in ((65536, 1 << 20, 256, 0), (16384, 262144, 1024, 1), (25000, 32768, 512, 0),
                       (16384, 32000, 1024, 0)):
        assert L.emb_grad_coalesce_workspace_bytes(T, V, D, g) <= emb.NOALLOC_SCRATCH_BYTES


def test_adam_coeffs_host_helper():
    # the coefficients a replayed graph reads: as emb_sparse_adam_apply forms them (fp64, rounded once)
    import torch
    out = torch.zeros(emb.EMB_ADAM_COEFFS_WORDS, dtype=torch.float32)
    for step in (1, 2, 10, 1000):
        emb.adam_coeffs(1e-3, 0.9, 0.999, 1e-8, step, out)
        bc1, bc2 = 1 - 0.9 ** step, 1 - 0.999 ** step
        want = np.array([0.9, 1 - 0.9, 0.999, 1 - 0.999, 1e-3 / bc1, 1 / bc2, 1e-8, 0.0], dtype=np.float32)
        assert np.array_equal(out.numpy(), want)
    L = emb.lib
    buf = (ctypes.c_float * 8)()
    assert L.emb_adam_coeffs(1e-3, 0.9, 0.999, 1e-8, 0, buf) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_adam_coeffs(1e-3, 1.0, 0.999, 1e-8, 1, buf) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_adam_coeffs(1e-3, 0.9, 0.999, 1e-8, 1, NULL) == emb.EMB_ERR_INVALID_ARG


def test_lookup_request_validation_and_workspace_query():
    L = emb.lib
    need = L.emb_lookup_request_workspace_bytes(1000, 5000)
    assert need > 0 and need % 256 == 0
    assert need < L.emb_grad_coalesce_workspace_bytes(1000, 5000, 64, emb.EMB_F32)  # no gradient partials
    assert L.emb_lookup_request_workspace_bytes(-1, 5000) == 0
    assert L.emb_lookup_request_workspace_bytes(1000, 0) == 0
    args = lambda T=1000, V=5000, own=FAKE, P=4, ids=FAKE, req=FAKE, counts=FAKE, offs=FAKE, nu=FAKE, inv=FAKE, \
        ws=FAKE, wsb=need: (ids, T, V, own, P, req, counts, offs, nu, inv, ws, wsb, NULL, NULL)
    assert L.emb_lookup_request(*args(wsb=need - 1)) == emb.EMB_ERR_WORKSPACE
    for bad in (dict(P=0), dict(P=1025), dict(V=0), dict(V=1 << 31), dict(T=-1), dict(T=1 << 30), dict(own=NULL),
                dict(ids=NULL), dict(req=NULL), dict(counts=NULL), dict(offs=NULL), dict(nu=NULL), dict(inv=NULL),
                dict(ws=NULL)):
        assert L.emb_lookup_request(*args(**bad)) == emb.EMB_ERR_INVALID_ARG, bad
    # (owner, id) keys must fit 32 bits, checked before the workspace
    short = dict(wsb=need - 1)
    assert L.emb_lookup_request(*args(V=1 << 22, P=1024, **short)) == emb.EMB_ERR_WORKSPACE
    assert L.emb_lookup_request(*args(V=(1 << 22) + 1, P=1024, **short)) == emb.EMB_ERR_UNSUPPORTED


def test_exchange_validation_ids_only():
    L = emb.lib
    args = lambda D=0, rows=NULL, ids=FAKE, cap=10, P=4: (ids, rows, FAKE, P, cap, D, ids, rows, FAKE, FAKE, NULL)
    assert L.emb_exchange_simulated(*args(D=-1)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_exchange_simulated(*args(D=8)) == emb.EMB_ERR_INVALID_ARG  # rows needed when D > 0
    assert L.emb_exchange_simulated(*args(ids=NULL)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_exchange_simulated(*args(P=0)) == emb.EMB_ERR_INVALID_ARG


def test_coalesce_split_validation_and_workspace_query():
    L = emb.lib
    need = L.emb_grad_coalesce_split_workspace_bytes(1000, 3000, 5000, 64, emb.EMB_F32)
    assert need > L.emb_grad_coalesce_workspace_bytes(1000, 5000, 64, emb.EMB_F32) and need % 256 == 0
    assert L.emb_grad_coalesce_split_workspace_bytes(1000, -1, 5000, 64, emb.EMB_F32) == 0
    args = lambda T=1000, nxt=FAKE, Tn=3000, V=5000, P=4, own=FAKE, wsb=need: (
        FAKE, T, nxt, Tn, FAKE, 0, 64, V, own, P, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, wsb, NULL, NULL)
    assert L.emb_grad_coalesce_split(*args(wsb=need - 1)) == emb.EMB_ERR_WORKSPACE
    assert L.emb_grad_coalesce_split(*args(Tn=-1)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce_split(*args(nxt=NULL)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce_split(*args(own=NULL)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_grad_coalesce_split(*args(P=0)) == emb.EMB_ERR_INVALID_ARG
    # bits(V) + bits(P) + 1 <= 32, checked before the workspace (so nothing launches here)
    short = dict(wsb=need - 1)
    assert L.emb_grad_coalesce_split(*args(V=1 << 21, P=1024, **short)) == emb.EMB_ERR_WORKSPACE
    assert L.emb_grad_coalesce_split(*args(V=(1 << 21) + 1, P=1024, **short)) == emb.EMB_ERR_UNSUPPORTED


def test_pack_validation_and_workspace_query():
    L = emb.lib
    need = L.emb_pack_by_owner_workspace_bytes(1000, 16)
    assert need > 0
    assert L.emb_pack_by_owner_workspace_bytes(1000, 0) == 0
    assert L.emb_pack_by_owner_workspace_bytes(1000, 1025) == 0
    args = lambda cap=1000, P=16, wsb=need, D=8: (FAKE, FAKE, FAKE, cap, D, FAKE, 5000, P, FAKE, FAKE, FAKE, FAKE,
                                                  FAKE, wsb, NULL, NULL)
    assert L.emb_pack_by_owner(*args(wsb=need - 1)) == emb.EMB_ERR_WORKSPACE
    assert L.emb_pack_by_owner(*args(P=0)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_pack_by_owner(*args(P=1025)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_pack_by_owner(*args(cap=-1)) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_pack_by_owner(*args(D=0)) == emb.EMB_ERR_INVALID_ARG


@pytest.mark.parametrize("bad", ["range", "step", "beta1", "beta2", "eps", "lr", "P"])
def test_adam_validation(bad):
    kw = dict(P=4, sb=0, se=4, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, step=1)
    kw.update({"range": dict(sb=3, se=2), "step": dict(step=0), "beta1": dict(b1=1.0), "beta2": dict(b2=-0.1),
               "eps": dict(eps=-1.0), "lr": dict(lr=float("nan")), "P": dict(P=0)}[bad])
    st = emb.lib.emb_sparse_adam_apply(FAKE, FAKE, FAKE, 5000, 8, FAKE, FAKE, FAKE, kw["P"], kw["sb"], kw["se"], 100,
                                       kw["lr"], kw["b1"], kw["b2"], kw["eps"], kw["step"], NULL, NULL)
    assert st == emb.EMB_ERR_INVALID_ARG


def test_adam_empty_range_is_noop():
    assert emb.lib.emb_sparse_adam_apply(FAKE, FAKE, FAKE, 5000, 8, FAKE, FAKE, FAKE, 4, 2, 2, 100, 1e-3, 0.9,
                                         0.999, 1e-8, 1, NULL, NULL) == emb.EMB_OK


def test_column_calls_validation():
    L = emb.lib
    # pack: P must satisfy 1 <= P <= min(D, 1024); sizes >= 0; buffers present when rows > 0
    assert L.emb_pack_by_column(FAKE, NULL, 10, 8, 0, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_pack_by_column(FAKE, NULL, 10, 8, 9, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG  # P > D
    assert L.emb_pack_by_column(FAKE, NULL, 10, 4096, 1025, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_pack_by_column(FAKE, NULL, -1, 8, 2, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_pack_by_column(NULL, NULL, 10, 8, 2, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_pack_by_column(FAKE, NULL, 10, 8, 2, NULL, NULL, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_pack_by_column(FAKE, NULL, 10, 1 << 22, 1024, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_pack_by_column(NULL, NULL, 0, 8, 2, NULL, NULL, NULL) == emb.EMB_OK  # nothing to do
    # lookup
    assert L.emb_gather_by_column(FAKE, 0, 8, 2, FAKE, 5, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_gather_by_column(FAKE, 10, 8, 9, FAKE, 5, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_gather_by_column(FAKE, 10, 8, 2, FAKE, -1, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_gather_by_column(FAKE, 10, 8, 2, NULL, 5, FAKE, NULL, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_gather_by_column(NULL, 10, 8, 2, NULL, 0, NULL, NULL, NULL) == emb.EMB_OK
    # join: row0 + R <= C
    assert L.emb_assemble_by_column(FAKE, 10, 5, 6, 8, 2, FAKE, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_assemble_by_column(FAKE, 10, -1, 2, 8, 2, FAKE, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_assemble_by_column(FAKE, 10, 0, -1, 8, 2, FAKE, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_assemble_by_column(FAKE, 10, 0, 3, 8, 0, FAKE, NULL) == emb.EMB_ERR_INVALID_ARG
    assert L.emb_assemble_by_column(NULL, 10, 10, 0, 8, 2, NULL, NULL) == emb.EMB_OK


def test_comm_cost_validation():
    L = emb.lib
    out = ctypes.c_double()
    ok = (emb.EMB_COMM_ALLTOALL, 8, 1, 1e9, 0.1, 1e10, 1e-5)
    assert L.emb_comm_cost(*ok, ctypes.byref(out)) == emb.EMB_OK
    assert L.emb_comm_cost(*ok, NULL) == emb.EMB_ERR_INVALID_ARG
    for i, bad in ((0, 4), (0, -1), (1, 0), (2, 0), (3, -1.0), (4, 1.5), (4, -0.1), (5, 0.0), (6, -1e-6),
                   (4, float("nan")), (5, float("inf"))):
        args = list(ok)
        args[i] = bad
        assert L.emb_comm_cost(*args, ctypes.byref(out)) == emb.EMB_ERR_INVALID_ARG, (i, bad)


def test_comm_cost_matches_oracle():
    """The library's Table 2 arithmetic (host code) against the oracle's, which is pinned to
    hand-worked values and the section's conclusions."""
    import oracle
    names = {emb.EMB_COMM_ALLTOALL: "alltoall", emb.EMB_COMM_ALLREDUCE: "allreduce", emb.EMB_COMM_PS: "ps",
             emb.EMB_COMM_ALLGATHER: "allgather"}
    for code, name in names.items():
        for N, S in ((1, 1), (2, 1), (8, 1), (8, 2), (64, 8)):
            for M in (0.0, 4e6, 1.2e9):
                for alpha in (0.0, 0.0168, 0.5, 1.0):
                    for B, beta in ((153e9, 0.0), (12.5e9, 5e-6)):
                        got = emb.comm_cost(code, N, M, alpha, B, beta, S=S)
                        want = oracle.comm_cost(name, N, M, alpha, B, beta, S=S)
                        assert got == pytest.approx(want, rel=1e-15, abs=0.0)


def test_bench_refuses_more_than_one_gpu():
    """The benchmark measures one GPU's share; asked for several it says so and exits before touching a GPU."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def _step_structs():
    """A schedule and arguments that pass every host check up to the first HIP call (pointers never
    dereferenced: each case below is refused before that)."""
    a = emb.StepArgs(V=1000, D=8, P=2, T=100, cap_rows=100, grad_dtype=emb.EMB_F32, lr=1e-3, beta1=0.9,
                     beta2=0.999, eps=1e-8, step=1)
    s = emb.StepSchedule(lookup_update=1, coalesce=2, pack=3, delayed=1, sorted=4096, coalesced=4096, packed=4096,
                         updated=4096, by_owner=1, sets=2)
    return a, s


def test_train_step_validation():
    L = emb.lib
    a, s = _step_structs()
    assert L.emb_train_step(None, ctypes.byref(s)) == emb.EMB_ERR_INVALID_ARG
    a.T = 101  # more tokens than the buffers hold
    assert L.emb_train_step(ctypes.byref(a), ctypes.byref(s)) == emb.EMB_ERR_INVALID_ARG
    a, s = _step_structs()
    s.updated = None  # events without the update's end event
    assert L.emb_train_step(ctypes.byref(a), ctypes.byref(s)) == emb.EMB_ERR_INVALID_ARG
    a, s = _step_structs()
    s.by_owner, s.split = 0, 1  # the split is owner-major
    assert L.emb_train_step(ctypes.byref(a), ctypes.byref(s)) == emb.EMB_ERR_INVALID_ARG
    a, s = _step_structs()
    s.sets = 65
    assert L.emb_train_step(ctypes.byref(a), ctypes.byref(s)) == emb.EMB_ERR_INVALID_ARG


def test_train_step_queued_validation():
    # refusals of the two-thread enqueue, all before any HIP call; the queue itself needs no GPU
    L = emb.lib
    q = emb.StepQueue()
    a, s = _step_structs()
    assert L.emb_train_step_queued(None, ctypes.byref(a), ctypes.byref(s)) == emb.EMB_ERR_INVALID_ARG
    for field, value in (("signals", 4096), ("by_owner", 0), ("split", 1)):
        a, s = _step_structs()
        setattr(s, field, value)
        assert L.emb_train_step_queued(q.handle, ctypes.byref(a), ctypes.byref(s)) == emb.EMB_ERR_UNSUPPORTED, field
    a, s = _step_structs()
    s.coalesce = s.lookup_update  # the sort on the stream the worker feeds
    assert L.emb_train_step_queued(q.handle, ctypes.byref(a), ctypes.byref(s)) == emb.EMB_ERR_UNSUPPORTED
    a, s = _step_structs()
    s.pack = s.lookup_update
    assert L.emb_train_step_queued(q.handle, ctypes.byref(a), ctypes.byref(s)) == emb.EMB_ERR_UNSUPPORTED
    a, s = _step_structs()
    a.T = 101
    assert L.emb_train_step_queued(q.handle, ctypes.byref(a), ctypes.byref(s)) == emb.EMB_ERR_INVALID_ARG
    a, s = _step_structs()
    s.sorted = None
    assert L.emb_train_step_queued(q.handle, ctypes.byref(a), ctypes.byref(s)) == emb.EMB_ERR_INVALID_ARG
    a, s = _step_structs()
    s.sets = 65
    assert L.emb_train_step_queued(q.handle, ctypes.byref(a), ctypes.byref(s)) == emb.EMB_ERR_INVALID_ARG
    a, s = _step_structs()  # the owner-major call's own argument checks (no ids)
    assert L.emb_train_step_queued(q.handle, ctypes.byref(a), ctypes.byref(s)) == emb.EMB_ERR_INVALID_ARG
    q.flush()  # nothing was handed to the worker
    assert L.emb_step_queue_flush(None) == emb.EMB_ERR_INVALID_ARG
    del q
