"""The C ABI library without a GPU: it loads, exports every symbol that
include/emb.h declares, and rejects bad arguments on the host before anything
is enqueued (no device memory is touched by these calls)."""
import ctypes
import os
import re

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
    assert emb.abi_version() == 1
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
