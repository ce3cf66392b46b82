"""The row-wise forward exchange (Sec. 4.1.1) on the GPU, through the C ABI:
a worker's lookup requests (emb_lookup_request: the distinct ids it needs,
grouped by owner, and each token's index into them) against the oracle, all
integers bit for bit; and end to end for P simulated workers, requests moved
to the owners (emb_exchange_simulated with ids only), answered by the owners'
emb_gather, moved back, and expanded through the inverse map by emb_gather,
which must give exactly the direct lookup table[ids]."""
import numpy as np
import pytest
import torch

import oracle
import paper_2110_09132_amd as emb
from gpu_helpers import host, to_dev
from pins import check_lookup_request
from workloads import gen

pytestmark = pytest.mark.gpu


def batch_ids(law, seed, T, V):
    key = gen.stream_key(seed, 0, gen.PURPOSE_IDS)
    if law == "uniform":
        return gen.uniform_ids(key, T, V)
    return gen.zipf_ids(key, T, V, 1.3 if law == "zipf13" else 1.1)


def owners(rule, V, P):
    if rule == "mod":
        return gen.owner_mod(V, P)
    if rule == "range":
        return gen.owner_range(V, P)
    own = np.random.default_rng(V + P).integers(0, P, V).astype(np.int32)
    own[::13] = P  # rows without an owner take no part
    return own


def gpu_request(ids, V, own, P):
    st = emb.new_status()
    ids_d = to_dev(ids.astype(np.int32))
    T = ids.size
    # sentinels: outputs must be written, not left over
    out = (torch.full((T,), -9, dtype=torch.int32, device="cuda"), torch.full((P,), -9, dtype=torch.int32, device="cuda"),
           torch.full((P + 1,), -9, dtype=torch.int32, device="cuda"), torch.full((1,), -9, dtype=torch.int32, device="cuda"),
           torch.full((T,), -9, dtype=torch.int32, device="cuda"))
    emb.lookup_request(ids_d, V, to_dev(own.astype(np.int32)), P, out=out, dev_status=st)
    torch.cuda.synchronize()
    req, cnt, offs, nu, inv = out
    U = int(nu.item())
    return dict(req_ids=host(req[:U]), req_counts=host(cnt), req_offsets=host(offs), U=U, inverse=host(inv),
                status=int(st.item()), dev=out)


def check_request(ids, V, own, P):
    want = oracle.lookup_request(ids, V, own, P)
    got = gpu_request(ids, V, own, P)
    assert got["U"] == want["U"]
    for k in ("req_ids", "req_counts", "req_offsets", "inverse"):
        assert np.array_equal(got[k], want[k]), k
    check_lookup_request(got, ids, V, own, P)
    bad_id = bool(np.any((ids < 0) | (ids >= V)))
    ok = (ids >= 0) & (ids < V)
    bad_own = bool(np.any((own[ids[ok]] < 0) | (own[ids[ok]] >= P)))
    flags = (emb.EMB_DEV_ID_OUT_OF_RANGE if bad_id else 0) | (emb.EMB_DEV_OWNER_OUT_OF_RANGE if bad_own else 0)
    assert got["status"] == flags
    return got


# (V, T, P, owner rule, id law): one tile and a ragged tail, many tiles, P = 1, P = 1024
# with unowned rows, 17/18-bit keys (two 9-bit passes), a single row, skew
CASES = [(1000, 100, 4, "mod", "uniform"), (5000, 3001, 7, "range", "uniform"), (1 << 16, 20000, 1, "mod", "uniform"),
         (4096, 9000, 1024, "rand", "uniform"), (1 << 14, 12345, 8, "mod", "zipf13"),
         (1 << 15, 40000, 4, "range", "zipf11"), (1, 300, 3, "mod", "uniform"), (1 << 22, 5000, 1024, "range", "uniform"),
         (100003, 65536, 16, "mod", "zipf13"), (1 << 20, 200000, 16, "mod", "uniform"),  # scanned head counts
         (1 << 21, 30000, 16, "mod", "uniform"), (256, 5000, 2, "mod", "zipf11")]  # 25 and 9 key bits


@pytest.mark.parametrize("V,T,P,rule,law", CASES)
def test_lookup_request_matches_oracle(V, T, P, rule, law):
    print(f"lookup_request V={V} T={T} P={P} {rule} {law}", flush=True)
    ids = batch_ids(law, 1000 + P, T, V)
    if T > 10:
        ids[[0, T // 3, T - 1]] = [-3, V, V + 77]  # not rows
    check_request(ids, V, owners(rule, V, P), P)


def test_lookup_request_edge_cases():
    V, P = 50, 3
    own = gen.owner_mod(V, P)
    print("lookup_request edge cases", flush=True)
    # empty batch: the empty result is written
    got = gpu_request(np.zeros(0, np.int32), V, own, P)
    assert got["U"] == 0 and got["req_counts"].tolist() == [0] * P and got["req_offsets"].tolist() == [0] * (P + 1)
    # no token takes part
    got = check_request(np.array([-1, 50, 99, -7], np.int32), V, own, P)
    assert got["U"] == 0 and np.all(got["inverse"] == -1)
    # one id repeated; every id once; an owner with nothing to serve
    check_request(np.full(1000, 7, np.int32), V, own, P)
    check_request(np.random.default_rng(3).permutation(V).astype(np.int32), V, own, P)
    check_request(np.arange(0, V, P, dtype=np.int32), V, own, P)  # owner 0 only


def test_headline_shape_lookup_request():
    """One worker of the uniform low-duplication workload: V = 2^20, T = 65536 tokens, P = 16."""
    V, T, P = 1 << 20, 65536, 16
    print(f"lookup_request headline V={V} T={T} P={P}", flush=True)
    check_request(batch_ids("uniform", 1100, T, V), V, gen.owner_mod(V, P), P)


def rowwise_forward(table, batches, V, own_np, P):
    """P workers: requests -> owners (ids only) -> owners' lookup -> back -> expand."""
    D = table.shape[1]
    own = to_dev(own_np.astype(np.int32))
    cap = max(1, max(ids.size for ids in batches))
    req = torch.full((P, cap), -5, dtype=torch.int32, device="cuda")
    offs = torch.zeros((P, P + 1), dtype=torch.int32, device="cuda")
    invs = []
    for w, ids in enumerate(batches):
        T = ids.size
        cnt = torch.empty(P, dtype=torch.int32, device="cuda")
        nu = torch.empty(1, dtype=torch.int32, device="cuda")
        inv = torch.empty(T, dtype=torch.int32, device="cuda")
        emb.lookup_request(to_dev(ids.astype(np.int32)), V, own, P, out=(req[w, :T], cnt, offs[w], nu, inv))
        invs.append(inv)
    # requests to their owners: owner p gets worker w's ids at [recv_offs[p][w], recv_offs[p][w + 1])
    recv_ids, recv_rows, recv_offs, total = emb.exchange_simulated(req, None, offs)
    assert recv_rows is None
    torch.cuda.synchronize()
    n = int(total.item())
    # each owner looks up what it was asked for in its rows of the table
    answers = emb.gather(table, recv_ids[:n]) if n else torch.zeros((0, D), device="cuda")
    # owner p's answers, block p of a [P, cap2] send layout whose owner blocks are the workers
    ro = host(recv_offs).astype(np.int64)
    cap2 = max(1, int(np.max(ro[:, P] - ro[:, 0])))
    back_ids = torch.full((P, cap2), -5, dtype=torch.int32, device="cuda")
    back_rows = torch.zeros((P, cap2, D), dtype=torch.float32, device="cuda")
    for p in range(P):
        a, b = int(ro[p, 0]), int(ro[p, P])
        back_ids[p, :b - a] = recv_ids[a:b]
        back_rows[p, :b - a] = answers[a:b]
    back_offs = to_dev((ro - ro[:, :1]).astype(np.int32))
    got_ids, got_rows, got_offs, _ = emb.exchange_simulated(back_ids, back_rows, back_offs)
    torch.cuda.synchronize()
    go = host(got_offs).astype(np.int64)
    out = []
    for w, ids in enumerate(batches):
        a, b = int(go[w, 0]), int(go[w, P])
        U = b - a
        # the rows come back in request order, with their ids
        assert np.array_equal(host(got_ids[a:b]), host(req[w, :U]))
        if U:
            out.append(emb.gather(got_rows[a:b], invs[w]))
        else:
            out.append(torch.zeros((ids.size, D), device="cuda"))
    torch.cuda.synchronize()
    return out, [host(i) for i in invs]


@pytest.mark.parametrize("V,D,P,sizes,rule", [(10007, 256, 16, (3000, 0, 2500, 1) + (700,) * 12, "mod"),
                                              (5000, 100, 7, (1200, 800, 1, 0, 64, 3000, 5), "range"),
                                              (300, 13, 3, (77, 500, 1), "mod"), (50, 4, 1, (9,), "mod")])
def test_rowwise_forward_exchange_equals_lookup(V, D, P, sizes, rule):
    sizes = tuple(sizes) + (0,) * (P - len(sizes))
    print(f"row-wise forward V={V} D={D} P={P} sizes={sizes}", flush=True)
    table = gen.normal_f32(gen.stream_key(1200 + D, 0, gen.PURPOSE_WEIGHTS), V * D).reshape(V, D)
    table_d = to_dev(table)
    own = owners(rule, V, P)
    batches = [batch_ids("zipf11" if w % 2 else "uniform", 1300 + w, n, V) for w, n in enumerate(sizes)]
    for ids in batches:
        if ids.size > 5:
            ids[[1, ids.size - 2]] = [-1, V + 3]  # not rows: zero rows
    got, invs = rowwise_forward(table_d, batches, V, own, P)
    for w, ids in enumerate(batches):
        direct = emb.gather(table_d, to_dev(ids.astype(np.int32))) if ids.size else torch.zeros((0, D), device="cuda")
        torch.cuda.synchronize()
        assert torch.equal(got[w], direct), f"worker {w}"
        want = np.where(((ids >= 0) & (ids < V))[:, None], table[np.clip(ids, 0, V - 1)], 0).astype(np.float32)
        assert np.array_equal(host(got[w]).view(np.uint32), want.view(np.uint32))
        assert np.array_equal(invs[w], oracle.lookup_request(ids, V, own, P)["inverse"])
