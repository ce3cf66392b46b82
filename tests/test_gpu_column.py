"""The column-wise partition (Sec. 4.1.1) on the GPU, through the C ABI:
the gradient pack (emb_pack_by_column), every owner's lookup in its shard
(emb_gather_by_column) and the join of a worker's slices
(emb_assemble_by_column) are bit copies and must equal the oracle bit for
bit, with send counts equal to the row count for every owner.  End to end,
the lookup-result exchange must return exactly the row-wise lookup, and the
column-wise update (each owner's Adam on its shard with its column slice)
exactly the row-wise update, since Adam is elementwise."""
import numpy as np
import pytest
import torch

import oracle
import paper_2110_09132_amd as emb
import tolerance
from gpu_helpers import host, to_dev
from workloads import gen

pytestmark = pytest.mark.gpu

ADAM = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8)
SENTINEL = np.float32(-7.25)


def normal(seed, n, purpose=gen.PURPOSE_GRADS):
    return gen.normal_f32(gen.stream_key(seed, 0, purpose), n)


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


# (cap, R, D, P): float4 path (D % 4P == 0) and float path (ragged widths), P = D, P = 1,
# R = 0, R clamped from above, several tiles with a ragged tail
PACK_CASES = [(5000, 4321, 256, 16), (3000, 2999, 100, 7), (777, 777, 13, 13), (1000, 1000, 64, 1),
              (1000, 0, 64, 4), (300, 299, 32, 8), (1, 1, 1, 1), (2049, 2049, 48, 5),
              (64, 50, 4096, 16), (40, 37, 9001, 3), (30, 30, 8192, 8)]  # one-row tiles; rows too wide for a tile


@pytest.mark.parametrize("cap,R,D,P", PACK_CASES)
def test_pack_by_column_matches_oracle(cap, R, D, P):
    print(f"pack_by_column cap={cap} R={R} D={D} P={P}", flush=True)
    rows = normal(100 + D, cap * D).reshape(cap, D)
    rows_d = to_dev(rows)
    blocks = torch.full((cap * D,), float(SENTINEL), dtype=torch.float32, device="cuda")
    counts = torch.full((P,), -1, dtype=torch.int32, device="cuda")
    num = torch.tensor([R], dtype=torch.int32, device="cuda")
    emb.pack_by_column(rows_d, P, num_rows=num, out=(blocks, counts))
    torch.cuda.synchronize()
    got = host(blocks)
    want = oracle.pack_by_column(rows[:R], P, C=cap)
    written = ~np.isnan(want)
    assert np.array_equal(bits(got[written]), bits(want[written]))
    assert np.all(got[~written] == SENTINEL)  # rows >= R untouched
    assert host(counts).tolist() == [R] * P


def test_pack_by_column_clamps_the_row_count():
    cap, D, P = 100, 24, 3
    rows = normal(7, cap * D).reshape(cap, D)
    for R, eff in ((150, 100), (-5, 0)):
        blocks = torch.full((cap * D,), float(SENTINEL), dtype=torch.float32, device="cuda")
        counts = torch.empty(P, dtype=torch.int32, device="cuda")
        emb.pack_by_column(to_dev(rows), P, num_rows=torch.tensor([R], dtype=torch.int32, device="cuda"),
                           out=(blocks, counts))
        torch.cuda.synchronize()
        want = oracle.pack_by_column(rows[:eff], P, C=cap)
        written = ~np.isnan(want)
        assert np.array_equal(bits(host(blocks)[written]), bits(want[written]))
        assert np.all(host(blocks)[~written] == SENTINEL)
        assert host(counts).tolist() == [eff] * P


def test_partition_table_without_count():
    """num_rows NULL packs all cap rows: the partitioned table (capacity V)."""
    V, D, P = 4099, 40, 5
    table = normal(11, V * D, gen.PURPOSE_WEIGHTS).reshape(V, D)
    shards, _ = emb.pack_by_column(to_dev(table), P)
    torch.cuda.synchronize()
    assert np.array_equal(bits(host(shards)), bits(oracle.pack_by_column(table, P)))


# (V, D, P, worker token counts)
FORWARD_CASES = [(10007, 256, 16, (3000, 0, 2500, 1)), (5000, 100, 7, (1200, 800)), (300, 13, 13, (77,)),
                 (1 << 16, 64, 4, (4096, 4096, 4096, 4096)), (50, 3, 1, (9, 9)), (900, 9001, 3, (40, 33)),
                 (700, 4096, 16, (50, 0, 21))]


@pytest.mark.parametrize("V,D,P,sizes", FORWARD_CASES)
def test_lookup_exchange_matches_oracle_and_rowwise_lookup(V, D, P, sizes):
    print(f"gather_by_column V={V} D={D} P={P} sizes={sizes}", flush=True)
    table = normal(200 + D, V * D, gen.PURPOSE_WEIGHTS).reshape(V, D)
    T = sum(sizes)
    ids = gen.uniform_ids(gen.stream_key(300 + D, 0, gen.PURPOSE_IDS), T, V)
    if T > 10:
        ids[[1, T // 2, T - 1]] = [-1, V, 1 << 30]  # not rows: zeros and a flag
    table_d = to_dev(table)
    shards, _ = emb.pack_by_column(table_d, P)
    st = emb.new_status()
    ids_d = to_dev(ids.astype(np.int32))
    blocks = emb.gather_by_column(shards, V, D, P, ids_d, dev_status=st)
    torch.cuda.synchronize()
    want, bad = oracle.gather_by_column(oracle.pack_by_column(table, P), V, D, P, ids)
    assert np.array_equal(bits(host(blocks)), bits(want))
    assert (int(st.item()) == emb.EMB_DEV_ID_OUT_OF_RANGE) == (bad > 0)
    rowwise = emb.gather(table_d, ids_d)
    torch.cuda.synchronize()
    t0 = 0
    for n in sizes:
        got = emb.assemble_by_column(blocks, T, D, P, row0=t0, R=n)
        torch.cuda.synchronize()
        assert np.array_equal(bits(host(got)), bits(oracle.assemble_by_column(want, T, D, P, t0, n)))
        assert np.array_equal(bits(host(got)), bits(host(rowwise[t0:t0 + n])))
        t0 += n


def test_empty_lookup_and_join_are_noops():
    D, P = 8, 2
    out = torch.full((4, D), 3.0, device="cuda")
    emb.gather_by_column(torch.zeros(10 * D, device="cuda"), 10, D, P,
                         torch.zeros(0, dtype=torch.int32, device="cuda"), out=out.view(-1)[:0])
    emb.assemble_by_column(torch.zeros(10 * D, device="cuda"), 10, D, P, row0=10, R=0, out=out[:0])
    torch.cuda.synchronize()
    assert torch.all(out == 3.0)


@pytest.mark.parametrize("V,D,P,T,law", [(20000, 256, 16, 6000, "zipf"), (3000, 100, 7, 2500, "uniform"),
                                         (500, 13, 4, 900, "uniform")])
def test_columnwise_update_equals_rowwise_update(V, D, P, T, law):
    """coalesce -> pack_by_column -> Adam on each shard with its block, three steps, against
    Adam on the whole table with the coalesced rows: bit for bit on the GPU, and within the
    fp32 row tolerance of the oracle's Adam on the same rows."""
    print(f"column-wise update V={V} D={D} P={P} T={T} {law}", flush=True)
    W0 = normal(400 + D, V * D, gen.PURPOSE_WEIGHTS).reshape(V, D)
    row = [to_dev(W0.copy()), torch.zeros((V, D), device="cuda"), torch.zeros((V, D), device="cuda")]
    col = [emb.pack_by_column(x, P)[0] for x in row]
    orc = [W0.copy(), np.zeros((V, D), np.float32), np.zeros((V, D), np.float32)]
    bnd = emb.column_offsets(D, P)
    for t in (1, 2, 3):
        key = gen.stream_key(500 + t, 0, gen.PURPOSE_IDS)
        ids = gen.zipf_ids(key, T, V, 1.1) if law == "zipf" else gen.uniform_ids(key, T, V)
        g = normal(600 + t, T * D).reshape(T, D)
        uid, seg, ug, nu = emb.grad_coalesce(to_dev(ids.astype(np.int32)), to_dev(g), V)
        blocks, counts = emb.pack_by_column(ug, P, num_rows=nu)
        torch.cuda.synchronize()
        U = int(nu.item())
        assert host(counts).tolist() == [U] * P
        offs = torch.tensor([0, U], dtype=torch.int32, device="cuda")
        emb.sparse_adam_apply(*row, uid, ug, offs, 1, 0, 1, step=t, **ADAM)
        for p in range(P):
            shard = [emb.column_block(x, V, D, P, p) for x in col]
            emb.sparse_adam_apply(*shard, uid, emb.column_block(blocks, T, D, P, p), offs, 1, 0, 1, step=t, **ADAM)
        # the oracle's Adam on the same (GPU-coalesced) rows
        oracle.sparse_adam(*orc, host(uid[:U]), host(ug[:U]), np.array([0, U], np.int32), 0, 1,
                           ADAM["lr"], ADAM["beta1"], ADAM["beta2"], ADAM["eps"], t)
    torch.cuda.synchronize()
    assert bnd[-1] == D
    for x_row, x_col, x_orc in zip(row, col, orc):
        joined = host(emb.assemble_by_column(x_col, V, D, P))
        assert np.array_equal(bits(joined), bits(host(x_row)))
    for x_row, x_orc, what in zip(row, orc, ("table", "exp_avg", "exp_avg_sq")):
        tolerance.assert_rows_close(host(x_row), x_orc, what=what)


def test_headline_shape_pack_and_lookup():
    """The shapes of the uniform low-duplication workload (V = 2^20 rows, D = 256, T = 65536 tokens,
    P = 16 owners): the gradient pack of all coalesced rows bit for bit against the oracle, and the
    lookup-result exchange against the row-wise lookup for 16 workers of 4096 tokens, with rows
    sampled against numpy's table[ids]."""
    V, D, T, P = 1 << 20, 256, 65536, 16
    print(f"headline column path V={V} D={D} T={T} P={P}", flush=True)
    ids = gen.uniform_ids(gen.stream_key(700, 0, gen.PURPOSE_IDS), T, V)
    g = normal(701, T * D).reshape(T, D)
    uid, seg, ug, nu = emb.grad_coalesce(to_dev(ids.astype(np.int32)), to_dev(g), V)
    blocks, counts = emb.pack_by_column(ug, P, num_rows=nu)
    torch.cuda.synchronize()
    U = int(nu.item())
    assert host(counts).tolist() == [U] * P
    want = oracle.pack_by_column(host(ug[:U]), P, C=T)
    written = ~np.isnan(want)
    assert np.array_equal(bits(host(blocks)[written]), bits(want[written]))
    del want, written
    table = torch.randn((V, D), device="cuda", generator=torch.Generator("cuda").manual_seed(702))
    shards, _ = emb.pack_by_column(table, P)
    ids_d = to_dev(ids.astype(np.int32))
    lk = emb.gather_by_column(shards, V, D, P, ids_d)
    rowwise = emb.gather(table, ids_d)
    sample = np.random.default_rng(703).choice(T, 512, replace=False)
    torch.cuda.synchronize()
    for q in range(16):
        n = T // 16
        got = emb.assemble_by_column(lk, T, D, P, row0=q * n, R=n)
        torch.cuda.synchronize()
        assert torch.equal(got, rowwise[q * n:(q + 1) * n])
    ref = host(table[to_dev(ids[sample].astype(np.int64))])
    got = host(emb.assemble_by_column(lk, T, D, P))[sample]
    assert np.array_equal(bits(got), bits(ref))
