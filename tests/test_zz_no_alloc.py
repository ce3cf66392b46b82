"""The allocation-free entry point emb_grad_coalesce_by_owner_noalloc (its workspace is the
library's static device array) against the entry point it mirrors, emb_grad_coalesce_by_owner with
a workspace the caller allocates: both run the same kernels in the same order, so every output is
required bit for bit equal (ids, segment offsets, rows, counts, offsets, the unique count, the
device status).  Three calls in a row on the same array, each smaller than the one before (the
multi-kernel path at the low-duplication stress shape, then a narrower batch, then one small enough
for the one-workgroup path), so that what the first call left in the array cannot leak into the
later ones.  Called through the C ABI."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2110_09132_amd as emb
from workloads import gen

pytestmark = pytest.mark.gpu


def ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def outputs(T, D, P):
    i32 = torch.int32
    return [torch.full((T,), -7, dtype=i32, device="cuda"), torch.full((T + 1,), -7, dtype=i32, device="cuda"),
            torch.full((T, D), float("nan"), dtype=torch.float32, device="cuda"),
            torch.full((P,), -7, dtype=i32, device="cuda"), torch.full((P + 1,), -7, dtype=i32, device="cuda"),
            torch.full((1,), -7, dtype=i32, device="cuda")]


def call(ids, G, V, own, P, noalloc):
    T, D = G.shape
    out = outputs(T, D, P)
    st = emb.new_status()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if noalloc:
        r = emb.lib.emb_grad_coalesce_by_owner_noalloc(ptr(ids), T, ptr(G), emb.EMB_F32, D, V, ptr(own), P,
                                                       *[ptr(o) for o in out], ptr(st), stream)
    else:
        ws = emb.new_workspace(emb.lib.emb_grad_coalesce_workspace_bytes(T, V, D, emb.EMB_F32))
        r = emb.lib.emb_grad_coalesce_by_owner(ptr(ids), T, ptr(G), emb.EMB_F32, D, V, ptr(own), P,
                                               *[ptr(o) for o in out], ptr(ws), ws.numel(), ptr(st), stream)
    assert r == emb.EMB_OK, emb.status_string(r)
    torch.cuda.synchronize()
    U = int(out[5].item())
    res = [out[0][:U], out[1][:U + 1], out[2][:U], out[3], out[4], out[5], st]
    return U, [x.cpu().numpy() for x in res]


SHAPES = [
    ("uniform", 1 << 20, 65536, 256, 16, "mod"),   # the low-duplication stress shape
    ("zipf", 32768, 20000, 64, 4, "range"),        # smaller: fewer tokens, narrower rows
    ("zipf", 5000, 1500, 32, 8, "mod"),            # one-workgroup path
]


def test_noalloc_equals_workspace_call():
    for law, V, T, D, P, rule in SHAPES:  # in a row on the same array, each input smaller than the last
        print(f"noalloc {law} V={V} T={T} D={D} P={P} {rule}", flush=True)
        key = gen.stream_key(V + T, 0, gen.PURPOSE_IDS)
        ids_np = gen.uniform_ids(key, T, V) if law == "uniform" else gen.zipf_ids(key, T, V, 1.1)
        G_np = gen.normal_f32(gen.stream_key(V + D, 0, gen.PURPOSE_GRADS), T * D, 0.01).reshape(T, D)
        own_np = gen.owner_mod(V, P) if rule == "mod" else gen.owner_range(V, P)
        ids = torch.from_numpy(ids_np).cuda()
        G = torch.from_numpy(G_np).cuda()
        own = torch.from_numpy(own_np).cuda()
        U0, want = call(ids, G, V, own, P, noalloc=False)
        for _ in range(2):  # twice on the same input as well
            U1, got = call(ids, G, V, own, P, noalloc=True)
            assert U1 == U0 and U1 > 0
            for a, b in zip(got, want):
                assert np.array_equal(a.view(np.uint32) if a.dtype == np.float32 else a,
                                      b.view(np.uint32) if b.dtype == np.float32 else b)


def largest_batch(V, D):
    """The most tokens whose workspace fits the static array (bisection on the library's query)."""
    lo, hi = 1, 1 << 24
    while lo < hi:
        mid = (lo + hi + 1) // 2
        if emb.lib.emb_grad_coalesce_workspace_bytes(mid, V, D, emb.EMB_F32) <= emb.NOALLOC_SCRATCH_BYTES:
            lo = mid
        else:
            hi = mid - 1
    return lo


def test_noalloc_at_its_largest_batch():
    # the largest batch of 256-float rows the array holds, against the workspace call; one token more
    # is refused on the host
    V, D, P = 1 << 20, 256, 16
    T = largest_batch(V, D)
    print(f"noalloc largest batch T={T} D={D}", flush=True)
    assert T > 65536
    ids = torch.from_numpy(gen.uniform_ids(gen.stream_key(T, 1, gen.PURPOSE_IDS), T, V)).cuda()
    G = torch.from_numpy(gen.normal_f32(gen.stream_key(T, 1, gen.PURPOSE_GRADS), T * D, 0.01).reshape(T, D)).cuda()
    own = torch.from_numpy(gen.owner_mod(V, P)).cuda()
    U0, want = call(ids, G, V, own, P, noalloc=False)
    U1, got = call(ids, G, V, own, P, noalloc=True)
    assert U1 == U0 and U1 > 0
    for a, b in zip(got, want):
        assert np.array_equal(a.view(np.uint32) if a.dtype == np.float32 else a,
                              b.view(np.uint32) if b.dtype == np.float32 else b)
    fake = ctypes.c_void_p(256)
    assert emb.lib.emb_grad_coalesce_by_owner_noalloc(fake, T + 1, fake, emb.EMB_F32, D, V, fake, P, fake, fake,
                                                      fake, fake, fake, fake, None, None) == emb.EMB_ERR_WORKSPACE


def test_noalloc_rejects_sizes_beyond_its_array():
    # 65536 tokens of 4096 floats need more than the 16 MiB array: refused on the host, nothing launched
    T, D, V, P = 65536, 4096, 1 << 20, 16
    need = emb.lib.emb_grad_coalesce_workspace_bytes(T, V, D, emb.EMB_F32)
    assert need > emb.NOALLOC_SCRATCH_BYTES
    fake = ctypes.c_void_p(256)
    assert emb.lib.emb_grad_coalesce_by_owner_noalloc(fake, T, fake, emb.EMB_F32, D, V, fake, P, fake, fake, fake,
                                                      fake, fake, fake, None, None) == emb.EMB_ERR_WORKSPACE
