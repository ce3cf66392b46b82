"""Pins of the oracle against what the paper and the mathematics fix.

Each `pin_*` function raises AssertionError when the oracle disagrees with an
independent reference: a hand-worked fixture (tests/golden), brute force on
tiny inputs (dense fp64 scatter-add over a V-row table, presence bitmaps,
bincounts), invariants, special cases with exactly known results, closed forms
of Adam, and PyTorch's dense Adam where lazy and dense Adam coincide.  The
same functions run against mutated builds of the oracle (see
test_oracle_mutations.py) to show that each planted mistake is caught.
"""
from __future__ import annotations

import numpy as np

import oracle
from golden import load as load_golden
from workloads import gen

ADAM = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8)


def _rng_ids(seed, T, V):
    return gen.uniform_ids(gen.stream_key(seed, 0, gen.PURPOSE_IDS), T, V)


def _rng_normal(seed, n, sigma=1.0, purpose=gen.PURPOSE_GRADS):
    return gen.normal_f32(gen.stream_key(seed, 0, purpose), n, sigma)


# --------------------------------------------------------------------- gather
def pin_gather():
    """out[t] = W[ids[t]] (Sec. 4.1.1), checked against numpy fancy indexing."""
    V, D, T = 37, 5, 200
    W = _rng_normal(7, V * D).reshape(V, D)
    ids = _rng_ids(8, T, V)
    out, bad = oracle.gather(W, ids)
    assert bad == 0
    assert np.array_equal(out.view(np.uint32), W[ids].view(np.uint32))
    ids2 = ids.copy()
    ids2[[3, 50, 199]] = [-1, V, 1 << 30]
    out2, bad2 = oracle.gather(W, ids2)
    assert bad2 == 3
    ok = np.ones(T, bool)
    ok[[3, 50, 199]] = False
    assert np.array_equal(out2[ok], W[ids2[ok]]) and not out2[~ok].any()


# ------------------------------------------------------------------- coalesce
def pin_coalesce_golden():
    """Hand-worked example of COALESCE/UNIQUE (Algorithm 1, Sec. 4.2.2)."""
    g = load_golden("coalesce_pack_worked.txt")
    r = oracle.coalesce(np.array(g["ids"]), np.array(g["grad"], np.float32), g["V"])
    assert r["uniq_ids"].tolist() == g["uniq_ids"]
    assert r["seg_offsets"].tolist() == g["seg_offsets"]
    assert r["uniq_grad"].tolist() == g["uniq_grad"]
    assert r["absum"].tolist() == g["absum"]


def pin_coalesce_bruteforce():
    """Against a dense fp64 V x D scatter-add and a presence bitmap (tiny V)."""
    seed = 100
    for V in (1, 2, 8, 37, 64):
        for T in (0, 1, 5, 100, 333):
            for D in (1, 3, 8):
                seed += 1
                ids = _rng_ids(seed, T, V)
                G = _rng_normal(seed, T * D).reshape(T, D)
                dense = np.zeros((V, D), np.float64)
                np.add.at(dense, ids, G.astype(np.float64))
                dabs = np.zeros((V, D), np.float64)
                np.add.at(dabs, ids, np.abs(G.astype(np.float64)))
                present = np.zeros(V, bool)
                present[ids] = True
                cnt = np.bincount(ids, minlength=V)
                r = oracle.coalesce(ids, G, V)
                u = r["uniq_ids"]
                assert r["U"] == int(present.sum())
                assert np.array_equal(u, np.flatnonzero(present))
                assert np.array_equal(np.diff(r["seg_offsets"]), cnt[u])
                assert r["seg_offsets"][0] == 0 and r["seg_offsets"][-1] == T
                # np.add.at accumulates in token order, as the oracle does: exact.
                assert np.array_equal(r["sum_f64"], dense[u])
                assert np.array_equal(r["absum"], dabs[u])
                assert np.array_equal(r["uniq_grad"], dense[u].astype(np.float32))


def pin_coalesce_invariants():
    """Column sums preserved, multiplicities sum to T, ids strictly ascending (Zipf batch)."""
    V, D, T = 5000, 16, 20000
    ids = gen.zipf_ids(gen.stream_key(3, 0, gen.PURPOSE_IDS), T, V, 1.1)
    G = _rng_normal(3, T * D).reshape(T, D)
    r = oracle.coalesce(ids, G, V)
    assert np.all(np.diff(r["uniq_ids"]) > 0)
    assert set(r["uniq_ids"].tolist()) == set(np.unique(ids).tolist())
    assert int(np.diff(r["seg_offsets"]).sum()) == T and np.all(np.diff(r["seg_offsets"]) > 0)
    col = G.astype(np.float64).sum(axis=0)
    got = r["sum_f64"].sum(axis=0)
    assert np.all(np.abs(got - col) <= 1e-9 * np.abs(G).astype(np.float64).sum(axis=0))


def pin_coalesce_special_cases():
    """Cases whose fp32 result is known exactly."""
    # all ids distinct: a pure permutation of the rows (bit copies)
    V, D, T = 1000, 7, 300
    perm = np.random.default_rng(5).permutation(V)[:T].astype(np.int32)
    G = _rng_normal(11, T * D).reshape(T, D)
    r = oracle.coalesce(perm, G, V)
    order = np.argsort(perm, kind="stable")
    assert np.array_equal(r["uniq_ids"], perm[order])
    assert np.array_equal(r["uniq_grad"].view(np.uint32), G[order].view(np.uint32))
    # every id exactly twice: one fp32 addition, correctly rounded, a + b in token order
    half = perm[:150]
    ids2 = np.concatenate([half, half[::-1]])
    G2 = _rng_normal(12, 300 * D).reshape(300, D)
    r2 = oracle.coalesce(ids2, G2, V)
    first = {int(i): t for t, i in enumerate(ids2[:150])}
    second = {int(i): 150 + t for t, i in enumerate(ids2[150:])}
    exp = np.stack([G2[first[int(i)]] + G2[second[int(i)]] for i in r2["uniq_ids"]])
    assert np.array_equal(r2["uniq_grad"].view(np.uint32), exp.view(np.uint32))
    # bf16 gradients are widened exactly: same as the fp32 path on the widened values
    ids3 = gen.zipf_ids(gen.stream_key(13, 0, gen.PURPOSE_IDS), 500, 300, 1.0)
    h = gen.bf16_round(_rng_normal(13, 500 * D, 0.01)).reshape(500, D)
    rb = oracle.coalesce(ids3, h, 300, grad_is_bf16=True)
    rf = oracle.coalesce(ids3, gen.bf16_bits_to_f32(h).reshape(500, D), 300)
    assert np.array_equal(rb["uniq_grad"], rf["uniq_grad"]) and np.array_equal(rb["uniq_ids"], rf["uniq_ids"])
    # empty batch
    r0 = oracle.coalesce(np.zeros(0, np.int32), np.zeros((0, 4), np.float32), 10)
    assert r0["U"] == 0 and r0["seg_offsets"].tolist() == [0]
    # out-of-range ids are dropped: same as coalescing the valid tokens alone
    ids4 = ids3.copy()
    ids4[[0, 10, 499]] = [-5, 300, 1 << 31 - 1]
    G4 = gen.bf16_bits_to_f32(h).reshape(500, D)
    r4 = oracle.coalesce(ids4, G4, 300)
    keep = (ids4 >= 0) & (ids4 < 300)
    r5 = oracle.coalesce(ids4[keep], G4[keep], 300)
    assert r4["n_invalid"] == 3
    assert np.array_equal(r4["uniq_ids"], r5["uniq_ids"]) and np.array_equal(r4["seg_offsets"], r5["seg_offsets"])
    assert np.array_equal(r4["uniq_grad"], r5["uniq_grad"])


# ----------------------------------------------------------------------- pack
def pin_pack_golden():
    g = load_golden("coalesce_pack_worked.txt")
    V, P = g["V"], g["P"]
    r = oracle.pack_by_owner(np.array(g["uniq_ids"]), np.array(g["uniq_grad"], np.float32),
                             gen.owner_mod(V, P), P)
    assert r["send_ids"].tolist() == g["send_ids"]
    assert r["send_rows"].tolist() == g["send_rows"]
    assert r["send_counts"].tolist() == g["send_counts"]
    assert r["send_offsets"].tolist() == g["send_offsets"]


def check_pack_result(r, uniq_ids, uniq_grad, row_owner, P):
    """Invariants of an owner-major stable pack (shared by oracle pins and GPU tests)."""
    own = row_owner[uniq_ids]
    counts = np.bincount(own, minlength=P)
    assert np.array_equal(r["send_counts"], counts)
    assert np.array_equal(r["send_offsets"], np.concatenate([[0], np.cumsum(counts)]))
    pos = {int(i): k for k, i in enumerate(uniq_ids)}
    for p in range(P):
        a, b = r["send_offsets"][p], r["send_offsets"][p + 1]
        blk = r["send_ids"][a:b]
        assert np.all(row_owner[blk] == p)
        assert np.all(np.diff(blk) > 0)
    assert sorted(r["send_ids"].tolist()) == sorted(uniq_ids.tolist())
    src = np.array([pos[int(i)] for i in r["send_ids"]], dtype=np.int64)
    assert np.array_equal(r["send_rows"].view(np.uint32), uniq_grad[src].view(np.uint32))


def pin_pack_invariants():
    for seed, (V, D, U, P, rule) in enumerate([(1000, 4, 300, 7, "mod"), (1000, 3, 999, 16, "range"),
                                               (50, 2, 50, 1, "mod"), (4096, 5, 1000, 1024, "rand"),
                                               (10, 1, 0, 3, "mod")]):
        uid = np.sort(np.random.default_rng(seed).permutation(V)[:U]).astype(np.int32)
        rows = _rng_normal(200 + seed, U * D).reshape(U, D)
        if rule == "mod":
            own = gen.owner_mod(V, P)
        elif rule == "range":
            own = gen.owner_range(V, P)
        else:
            own = np.random.default_rng(99).integers(0, P, V).astype(np.int32)
        r = oracle.pack_by_owner(uid, rows, own, P)
        assert r["n_dropped"] == 0
        check_pack_result(r, uid, rows, own, P)
        if P == 1 or rule == "range":  # owner-major order is already ascending-id order
            assert np.array_equal(r["send_ids"], uid)
            assert np.array_equal(r["send_rows"].view(np.uint32), rows.view(np.uint32))
    # rows whose owner is out of range are not sent
    V, P = 20, 4
    own = gen.owner_mod(V, P)
    own[[3, 7]] = [4, -1]
    uid = np.arange(0, 20, 2, dtype=np.int32)
    rows = _rng_normal(5, 10 * 2).reshape(10, 2)
    r = oracle.pack_by_owner(uid, rows, own, P)
    assert r["n_dropped"] == 0  # 3 and 7 are odd: not in uid
    uid2 = np.arange(0, 20, 1, dtype=np.int32)
    r2 = oracle.pack_by_owner(uid2, _rng_normal(6, 40).reshape(20, 2), own, P)
    assert r2["n_dropped"] == 2 and r2["send_offsets"][-1] == 18
    assert 3 not in r2["send_ids"].tolist() and 7 not in r2["send_ids"].tolist()


# --------------------------------------------------------- vertical split
def pin_split_golden():
    """Hand-worked set split of Algorithm 1 and the two owner-major packs."""
    g = load_golden("vertical_split_worked.txt")
    c = oracle.coalesce(np.array(g["ids"], np.int32), np.array(g["grad"], np.float32), g["V"])
    assert c["uniq_ids"].tolist() == g["uniq_ids"]
    r = oracle.split_pack(c["uniq_ids"], c["uniq_grad"], np.array(g["next_ids"], np.int32),
                          np.array(g["owner"], np.int32), g["P"])
    assert r["is_prior"].astype(int).tolist() == g["is_prior"] and r["n_prior"] == g["n_prior"]
    assert r["send_ids"].tolist() == g["send_ids"]
    assert r["send_rows"].tolist() == g["send_rows"]
    assert r["send_counts"].tolist() == g["send_counts"]
    assert r["send_offsets"].tolist() == g["send_offsets"]


def check_split_result(r, uniq_ids, uniq_grad, next_ids, row_owner, P):
    """What Algorithm 1 fixes about the split, checked with Python sets (shared by oracle pins and
    GPU tests): prior = D_u & D_next, delayed = D_u - prior, each packed owner-major and stable."""
    nxt = set(int(i) for i in next_ids)
    prior = [int(i) for i in uniq_ids if int(i) in nxt]
    delayed = [int(i) for i in uniq_ids if int(i) not in nxt]
    offs = np.asarray(r["send_offsets"])
    n_prior = int(offs[P])
    assert n_prior == len(prior)
    assert sorted(r["send_ids"][:n_prior].tolist()) == prior
    assert sorted(r["send_ids"][n_prior:].tolist()) == delayed
    assert set(r["send_ids"][:n_prior].tolist()).isdisjoint(r["send_ids"][n_prior:].tolist())
    pos = {int(i): k for k, i in enumerate(uniq_ids)}
    for part, (lo, hi) in enumerate(((0, P), (P, 2 * P))):
        for p in range(P):
            a, b = int(offs[lo + p]), int(offs[lo + p + 1])
            blk = r["send_ids"][a:b]
            assert np.all(row_owner[blk] == p) and np.all(np.diff(blk) > 0)
        assert np.array_equal(np.asarray(r["send_counts"])[lo:hi], np.diff(offs[lo:hi + 1]))
    src = np.array([pos[int(i)] for i in r["send_ids"]], dtype=np.int64)
    assert np.array_equal(np.asarray(r["send_rows"]).view(np.uint32), uniq_grad[src].view(np.uint32))


def pin_split_invariants():
    for seed, (V, D, T, P, law) in enumerate([(1000, 3, 700, 4, "uniform"), (50, 2, 400, 3, "uniform"),
                                             (20000, 4, 3000, 16, "zipf"), (7, 1, 30, 1, "uniform")]):
        key = gen.stream_key(300 + seed, 0, gen.PURPOSE_IDS)
        ids = gen.uniform_ids(key, T, V) if law == "uniform" else gen.zipf_ids(key, T, V, 1.1)
        key2 = gen.stream_key(400 + seed, 0, gen.PURPOSE_IDS)
        nxt = gen.uniform_ids(key2, T, V) if law == "uniform" else gen.zipf_ids(key2, T, V, 1.1)
        c = oracle.coalesce(ids, _rng_normal(500 + seed, T * D).reshape(T, D), V)
        own = gen.owner_mod(V, P)
        r = oracle.split_pack(c["uniq_ids"], c["uniq_grad"], nxt, own, P)
        check_split_result(r, c["uniq_ids"], c["uniq_grad"], nxt, own, P)
    # special cases: the next batch repeats this one (all prior), shares nothing (all delayed),
    # is empty, or holds only ids that are not rows
    V, D, P = 300, 2, 5
    ids = _rng_ids(9, 500, V)
    c = oracle.coalesce(ids, _rng_normal(10, 500 * D).reshape(500, D), V)
    own = gen.owner_mod(V, P)
    for nxt, n_prior in ((ids[::-1].copy(), c["U"]), (ids + V, 0), (np.zeros(0, np.int32), 0),
                         (np.array([-1, V, V + 7], np.int32), 0)):
        is_prior, n = oracle.vertical_split(c["uniq_ids"], nxt)
        assert n == n_prior and int(is_prior.sum()) == n_prior
        r = oracle.split_pack(c["uniq_ids"], c["uniq_grad"], nxt, own, P)
        check_split_result(r, c["uniq_ids"], c["uniq_grad"], nxt, own, P)


def pin_split_two_applies():
    """Applying Adam to the prior rows and then to the delayed rows with the same step t gives
    exactly one apply on their union: the two row sets are disjoint and the update is per
    element (the reading of the step counter rule of Sec. 5.7)."""
    V, D, T, P, t = 400, 3, 600, 4, 3
    ids, nxt = _rng_ids(21, T, V), _rng_ids(22, T, V)
    c = oracle.coalesce(ids, _rng_normal(23, T * D, 0.1).reshape(T, D), V)
    own = gen.owner_mod(V, P)
    r = oracle.split_pack(c["uniq_ids"], c["uniq_grad"], nxt, own, P)
    whole = oracle.pack_by_owner(c["uniq_ids"], c["uniq_grad"], own, P)
    W0, M0, S0 = _adam_tables(V, D, 24)
    M0 += _rng_normal(25, V * D, 0.01).reshape(V, D)
    S0 += np.abs(_rng_normal(26, V * D, 0.01)).reshape(V, D)
    A = [x.copy() for x in (W0, M0, S0)]
    B = [x.copy() for x in (W0, M0, S0)]
    offs = r["send_offsets"]
    oracle.sparse_adam(*A, r["send_ids"], r["send_rows"], offs[:P + 1], 0, P, step=t, **ADAM)
    oracle.sparse_adam(*A, r["send_ids"], r["send_rows"], offs[P:], 0, P, step=t, **ADAM)
    oracle.sparse_adam(*B, whole["send_ids"], whole["send_rows"], whole["send_offsets"], 0, P, step=t, **ADAM)
    for x, y in zip(A, B):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))


# ------------------------------------------------------- lookup requests
def pin_lookup_request_golden():
    """Hand-worked requests of a worker in the row-wise partition (Sec. 4.1.1)."""
    g = load_golden("lookup_request_worked.txt")
    ids = np.array(g["ids"], np.int32)
    for own, sfx in ((gen.owner_mod(g["V"], g["P"]), ""), (np.array(g["row_owner_b"], np.int32), "_b")):
        r = oracle.lookup_request(ids, g["V"], own, g["P"])
        assert r["req_ids"].tolist() == g["req_ids" + sfx]
        assert r["req_counts"].tolist() == g["req_counts" + sfx]
        assert r["req_offsets"].tolist() == g["req_offsets" + sfx]
        assert r["inverse"].tolist() == g["inverse" + sfx]
        assert r["U"] == len(g["req_ids" + sfx])


def check_lookup_request(r, ids, V, row_owner, P):
    """What the requests of a batch must be, checked against Python sets and numpy (shared by
    oracle pins and GPU tests):
      the requested ids are the set of the batch's ids that are rows with an owner in [0, P);
      they come grouped by owner (ascending owners), ascending inside a group, and the counts
      and offsets describe the groups;
      every token that takes part points at its own id, every other token at -1."""
    ids = np.asarray(ids, np.int64)
    take = (ids >= 0) & (ids < V)
    take[take] &= (row_owner[ids[take]] >= 0) & (row_owner[ids[take]] < P)
    want = sorted(set(ids[take].tolist()))
    req = np.asarray(r["req_ids"], np.int64)
    assert r["U"] == len(want) == req.size
    assert sorted(req.tolist()) == want
    own = row_owner[req]
    counts = np.bincount(own, minlength=P)[:P] if req.size else np.zeros(P, np.int64)
    assert np.array_equal(r["req_counts"], counts)
    assert np.array_equal(r["req_offsets"], np.concatenate([[0], np.cumsum(counts)]))
    for p in range(P):
        blk = req[r["req_offsets"][p]:r["req_offsets"][p + 1]]
        assert np.all(row_owner[blk] == p) and np.all(np.diff(blk) > 0)
    inv = np.asarray(r["inverse"], np.int64)
    assert inv.size == ids.size
    assert np.all(inv[~take] == -1)
    assert np.all((inv[take] >= 0) & (inv[take] < req.size))
    assert np.array_equal(req[inv[take]], ids[take])


def pin_lookup_request_invariants():
    for seed, (V, T, P, rule) in enumerate([(1000, 3000, 7, "mod"), (1000, 50, 16, "range"), (50, 500, 1, "mod"),
                                            (4096, 2000, 1024, "rand"), (10, 0, 3, "mod"), (1, 9, 2, "mod")]):
        ids = _rng_ids(400 + seed, T, V + 2)  # a few ids >= V
        if T > 3:
            ids[[0, T // 2]] = [-5, V + 1000]
        if rule == "mod":
            own = gen.owner_mod(V, P)
        elif rule == "range":
            own = gen.owner_range(V, P)
        else:
            own = np.random.default_rng(98).integers(0, P, V).astype(np.int32)
            own[::17] = P  # rows without an owner
        r = oracle.lookup_request(ids, V, own, P)
        check_lookup_request(r, ids, V, own, P)
        if P == 1 and r["U"]:  # a single owner: the request is the sorted distinct ids
            assert np.array_equal(r["req_ids"], np.unique(ids[(ids >= 0) & (ids < V)]))


def pin_lookup_request_serves_the_lookup():
    """Row-wise forward exchange end to end (Sec. 4.1.1): P workers send their requests, each
    owner answers with the rows of its shard (the owner's gather of the ids it received), and a
    worker's gather through its inverse map of the rows it got back equals numpy's table[ids]
    (zero rows for tokens that take part in nothing)."""
    V, D, P = 200, 5, 4
    table = _rng_normal(410, V * D, purpose=gen.PURPOSE_WEIGHTS).reshape(V, D)
    own = gen.owner_range(V, P)
    shard_of = {p: np.nonzero(own == p)[0] for p in range(P)}  # row ids of owner p, ascending
    local = np.zeros(V, np.int32)
    for p, rows in shard_of.items():
        local[rows] = np.arange(rows.size)
    shards = {p: table[rows] for p, rows in shard_of.items()}
    batches = [_rng_ids(420 + q, n, V + 1) for q, n in enumerate((60, 0, 33, 1))]
    for ids in batches:
        r = oracle.lookup_request(ids, V, own, P)
        back = np.zeros((r["U"], D), np.float32)
        for p in range(P):
            a, b = r["req_offsets"][p], r["req_offsets"][p + 1]
            back[a:b] = oracle.gather(shards[p], local[r["req_ids"][a:b]])[0]
        got = oracle.gather(back, r["inverse"])[0]
        want = np.where((ids < V)[:, None], table[np.minimum(ids, V - 1)], 0).astype(np.float32)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


# ------------------------------------------------ receiver side of the exchange
def pin_concat_coalesce_is_sum_of_workers():
    """The exchange delivers every worker's coalesced rows to their owner, who sums the rows of
    one index (Sec. 4.1.1 / 4.1.2).  So the merged result is the coalesce of all workers' tokens
    together: its ids are the union of the workers' ids, and each fp64 sum is the sum of the
    workers' fp64 sums (checked here on the oracle; the GPU merge is compared with it)."""
    V, D, T, P = 300, 3, 500, 4
    ids = [_rng_ids(600 + w, T, V) for w in range(P)]
    grads = [_rng_normal(700 + w, T * D).reshape(T, D) for w in range(P)]
    parts = [oracle.coalesce(i, g, V) for i, g in zip(ids, grads)]
    whole = oracle.coalesce(np.concatenate(ids), np.concatenate(grads), V)
    union = sorted(set().union(*(set(c["uniq_ids"].tolist()) for c in parts)))
    assert whole["uniq_ids"].tolist() == union
    acc = {u: np.zeros(D) for u in union}
    for c in parts:
        for k, u in enumerate(c["uniq_ids"].tolist()):
            acc[u] += c["sum_f64"][k]
    ref = np.array([acc[u] for u in union])
    assert np.allclose(whole["sum_f64"], ref, rtol=1e-12, atol=1e-12)
    counts = np.bincount(np.concatenate(ids), minlength=V)
    assert np.array_equal(np.diff(whole["seg_offsets"]), counts[whole["uniq_ids"]])


# ----------------------------------------------------------------------- adam
def _adam_tables(V, D, seed):
    W = _rng_normal(seed, V * D, purpose=gen.PURPOSE_WEIGHTS).reshape(V, D)
    return W, np.zeros((V, D), np.float32), np.zeros((V, D), np.float32)


def pin_adam_golden():
    """Hand-worked first step from zero moments (Kingma & Ba Algorithm 1, t = 1)."""
    g = load_golden("adam_first_step.txt")
    n = len(g["g"])
    W = np.array(g["w0"], np.float32).reshape(n, 1).copy()
    m = np.zeros((n, 1), np.float32)
    v = np.zeros((n, 1), np.float32)
    rows = np.array(g["g"], np.float32).reshape(n, 1)
    oracle.sparse_adam(W, m, v, np.arange(n, dtype=np.int32), rows, np.array([0, n], np.int32), 0, 1,
                       g["lr"], g["beta1"], g["beta2"], g["eps"], 1)
    np.testing.assert_allclose(W[:, 0], np.array(g["w1"], np.float32), rtol=2e-7, atol=0)
    np.testing.assert_allclose(m[:, 0], np.array(g["m1"], np.float32), rtol=2e-7, atol=0)
    np.testing.assert_allclose(v[:, 0], np.array(g["v1"], np.float32), rtol=2e-7, atol=0)


def pin_adam_closed_forms():
    """Constant gradient: w_t = w_0 - t lr g/(|g|+eps).  Rows touched only at
    steps 1 and 3 (lazy): m_hat_3 = (1+b1) g/(1+b1+b1^2), v_hat_3 =
    (1+b2) g^2/(1+b2+b2^2).  Untouched rows stay bit-identical."""
    lr, b1, b2, eps = ADAM["lr"], ADAM["beta1"], ADAM["beta2"], ADAM["eps"]
    V, D = 12, 6
    W, m, v = _adam_tables(V, D, 21)
    W0 = W.copy()
    rows_const = np.array([1, 4, 5], np.int32)
    g = np.array([[0.3, -2.0, 1e-3, 5e-9, 1.0, -0.7]], np.float32).repeat(3, axis=0)
    g[1] *= -3
    g[2] *= 0.01
    lazy_row = np.array([9], np.int32)
    gl = np.array([[0.2, -0.4, 1e-8, 3.0, -1e-6, 0.05]], np.float32)
    for t in range(1, 6):
        oracle.sparse_adam(W, m, v, rows_const, g, np.array([0, 3], np.int32), 0, 1, lr, b1, b2, eps, t)
        if t in (1, 3):
            oracle.sparse_adam(W, m, v, lazy_row, gl, np.array([0, 1], np.int32), 0, 1, lr, b1, b2, eps, t)
        if t == 3:
            W_lazy3 = W[9].copy()
    g64 = g.astype(np.float64)
    exp = W0[rows_const].astype(np.float64) - 5 * lr * g64 / (np.abs(g64) + eps)
    np.testing.assert_allclose(W[rows_const], exp, rtol=0, atol=4e-7 * np.abs(exp).max())
    # lazy closed form at step 3
    gl64 = gl[0].astype(np.float64)
    w1 = W0[9].astype(np.float64) - lr * gl64 / (np.abs(gl64) + eps)
    mh = (1 + b1) * gl64 / (1 + b1 + b1 * b1)
    vh = (1 + b2) * gl64 * gl64 / (1 + b2 + b2 * b2)
    w3 = w1 - lr * mh / (np.sqrt(vh) + eps)
    np.testing.assert_allclose(W_lazy3, w3, rtol=0, atol=4e-7 * np.abs(w3).max())
    untouched = np.setdiff1d(np.arange(V), np.concatenate([rows_const, lazy_row]))
    assert np.array_equal(W[untouched].view(np.uint32), W0[untouched].view(np.uint32))
    assert not m[untouched].any() and not v[untouched].any()


def pin_adam_vs_torch_dense():
    """When every row is touched at every step, lazy Adam is dense Adam: compare
    with torch.optim.Adam (fp64) over 6 steps, gradients spanning 1e-9 .. 1."""
    import torch
    V, D, steps = 10, 8, 6
    W, m, v = _adam_tables(V, D, 31)
    p = torch.nn.Parameter(torch.tensor(W.astype(np.float64)))
    opt = torch.optim.Adam([p], lr=ADAM["lr"], betas=(ADAM["beta1"], ADAM["beta2"]), eps=ADAM["eps"])
    scale = np.logspace(-9, 0, V * D).reshape(V, D)
    for t in range(1, steps + 1):
        g = (_rng_normal(40 + t, V * D).reshape(V, D) * scale).astype(np.float32)
        oracle.sparse_adam(W, m, v, np.arange(V, dtype=np.int32), g, np.array([0, V], np.int32), 0, 1,
                           ADAM["lr"], ADAM["beta1"], ADAM["beta2"], ADAM["eps"], t)
        p.grad = torch.tensor(g.astype(np.float64))
        opt.step()
    ref = p.detach().numpy()
    st = opt.state[p]
    np.testing.assert_allclose(W, ref, rtol=0, atol=2e-6 * np.abs(ref).max())
    # m can cancel across steps: measure its error against the gradient scale.
    mref = st["exp_avg"].numpy()
    assert np.all(np.abs(m - mref) <= 2e-6 * (np.abs(mref) + 0.1 * scale))
    np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=2e-6, atol=1e-38)


def pin_adam_shard_ranges():
    """Updating shards one by one equals one update over all of them; a prior
    and a delayed part applied with the same step equal one apply on the union
    (the step counter of Sec. 5.7 advances once per iteration)."""
    V, D, P = 40, 3, 4
    Wa, ma, va = _adam_tables(V, D, 51)
    Wb, mb, vb = Wa.copy(), ma.copy(), va.copy()
    ids = np.array([1, 5, 9, 13, 2, 6, 30, 3, 7, 11, 39], np.int32)
    offs = np.array([0, 4, 7, 7, 11], np.int32)  # shard 2 empty
    rows = _rng_normal(52, ids.size * D).reshape(ids.size, D)
    for t in (1, 2):
        oracle.sparse_adam(Wa, ma, va, ids, rows, offs, 0, P, ADAM["lr"], ADAM["beta1"], ADAM["beta2"], ADAM["eps"], t)
        for s in range(P):
            oracle.sparse_adam(Wb, mb, vb, ids, rows, offs, s, s + 1, ADAM["lr"], ADAM["beta1"], ADAM["beta2"],
                               ADAM["eps"], t)
    for a, b in ((Wa, Wb), (ma, mb), (va, vb)):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


# ------------------------------------------------------- column-wise partition
def _col_bounds(D, P):
    return [(p * D) // P for p in range(P + 1)]


def _blocks_equal(got, want_with_none):
    want = np.array([np.nan if x is None else x for x in want_with_none], np.float32)
    written = ~np.isnan(want)
    assert got.shape == want.shape
    assert np.array_equal(got[written], want[written])
    assert np.all(np.isnan(got[~written]))  # the pack leaves rows >= R alone


def pin_column_golden():
    """Hand-worked column split, pack, lookup and join (Sec. 4.1.1)."""
    g = load_golden("column_partition_worked.txt")
    rows = np.array(g["rows"], np.float32)
    _blocks_equal(oracle.pack_by_column(rows, g["P"], C=g["C"]), g["blocks"])
    _blocks_equal(oracle.pack_by_column(rows, g["P3"]), g["blocks3"])
    blocks, bad = oracle.gather_by_column(np.array(g["shards"], np.float32), g["V"], g["D"], g["P"],
                                          np.array(g["ids"], np.int32))
    assert bad == g["n_invalid"]
    assert blocks.tolist() == g["lookup_blocks"]
    out = oracle.assemble_by_column(blocks, len(g["ids"]), g["D"], g["P"], row0=g["row0"], R=g["R"])
    assert out.tolist() == g["assembled"]


def pin_column_layout():
    """Special cases with known layouts, and a column-tagged brute force for ragged splits.
      P = 1: the single block is the rows themselves.
      P = D: block p is column p, so the blocks are the transpose of the rows.
      P | D: the blocks are rows.reshape(R, P, D/P) with the first two axes swapped.
      any P <= D: tag every float with (row, column); each block must hold, row by row, a
      contiguous ascending run of columns, the runs of owners 0 .. P-1 following each other,
      widths within one of each other, every column exactly once."""
    R, C = 7, 9
    for D in (1, 6, 12, 13):
        rows = _rng_normal(60 + D, R * D).reshape(R, D)
        b = oracle.pack_by_column(rows, 1, C=C)
        assert np.array_equal(b[:R * D], rows.reshape(-1)) and np.all(np.isnan(b[R * D:]))
        b = oracle.pack_by_column(rows, D)
        assert np.array_equal(b.reshape(D, R), rows.T)
        for P in (2, 3, 4, 6):
            if D % P == 0:
                b = oracle.pack_by_column(rows, P)
                assert np.array_equal(b.reshape(P, R, D // P), rows.reshape(R, P, D // P).transpose(1, 0, 2))
    for D, P in ((13, 4), (10, 3), (7, 7), (100, 16), (5, 2)):
        tag = (np.arange(R)[:, None] * 1000 + np.arange(D)[None, :]).astype(np.float32)
        b = oracle.pack_by_column(tag, P, C=C)
        seen, start, widths = [], 0, []
        for p in range(P):
            w = None
            for r in range(R):
                blk = b[C * start + r * (w or 0):]
                if w is None:  # width of block p: the run of row 0's columns that are consecutive
                    w = 1
                    while start + w < D and blk[w] == blk[0] + w:
                        w += 1
                    if p == P - 1:
                        w = D - start
                run = b[C * start + r * w: C * start + (r + 1) * w]
                assert np.array_equal(run, r * 1000 + start + np.arange(w, dtype=np.float32))
            seen.extend(range(start, start + w))
            widths.append(w)
            start += w
        assert seen == list(range(D)) and max(widths) - min(widths) <= 1
        assert [0] + np.cumsum(widths).tolist() == _col_bounds(D, P)


def pin_column_roundtrip():
    """Joining the blocks gives back the rows, for every row range (ragged splits included)."""
    for seed, (R, C, D, P) in enumerate(((10, 12, 13, 4), (1, 1, 5, 5), (33, 40, 64, 16), (6, 6, 3, 1))):
        rows = _rng_normal(70 + seed, R * D).reshape(R, D)
        b = oracle.pack_by_column(rows, P, C=C)
        assert np.array_equal(oracle.assemble_by_column(b, C, D, P, 0, R), rows)
        for row0, n in ((1, R - 1), (R // 2, R - R // 2), (R - 1, 1), (R, 0)):
            assert np.array_equal(oracle.assemble_by_column(b, C, D, P, row0, n), rows[row0:row0 + n])


def pin_column_forward():
    """The lookup-result exchange (Sec. 4.1.1): each owner looks up every worker's tokens in its
    shard; joining a worker's rows from all owners gives numpy's table[ids] for that worker's ids
    (zero rows for ids that are not rows), and equals the row-wise lookup."""
    for seed, (V, D, P, sizes) in enumerate(((50, 13, 4, (7, 0, 11, 3)), (300, 64, 16, (40, 25)),
                                             (9, 3, 3, (5,)))):
        table = _rng_normal(80 + seed, V * D, purpose=gen.PURPOSE_WEIGHTS).reshape(V, D)
        shards = oracle.pack_by_column(table, P)
        ids = _rng_ids(90 + seed, sum(sizes), V + 3)  # a few ids >= V
        blocks, bad = oracle.gather_by_column(shards, V, D, P, ids)
        assert bad == int(np.sum(ids >= V))
        t0 = 0
        for n in sizes:
            q = ids[t0:t0 + n]
            want = np.where((q < V)[:, None], table[np.minimum(q, V - 1)], 0).astype(np.float32)
            got = oracle.assemble_by_column(blocks, ids.size, D, P, t0, n)
            assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
            assert np.array_equal(got, oracle.gather(table, q)[0])
            t0 += n


def pin_column_adam():
    """Adam is elementwise, so each owner updating its shard with its column slice of the
    coalesced rows (the column-wise exchange) gives bit for bit the row-wise update."""
    V, D, P = 30, 13, 4
    Wa, ma, va = _adam_tables(V, D, 95)
    ids = np.array([0, 3, 4, 17, 29], np.int32)
    sw, sm, sv = (oracle.pack_by_column(x, P) for x in (Wa, ma, va))
    bnd = _col_bounds(D, P)
    for t in (1, 2, 3):
        rows = _rng_normal(96 + t, ids.size * D).reshape(ids.size, D)
        oracle.sparse_adam(Wa, ma, va, ids, rows, np.array([0, ids.size], np.int32), 0, 1, ADAM["lr"],
                           ADAM["beta1"], ADAM["beta2"], ADAM["eps"], t)
        blocks = oracle.pack_by_column(rows, P)
        for p in range(P):
            a, w = bnd[p], bnd[p + 1] - bnd[p]
            shard = [x[V * a: V * (a + w)].reshape(V, w) for x in (sw, sm, sv)]
            oracle.sparse_adam(*shard, ids, blocks[ids.size * a: ids.size * (a + w)].reshape(ids.size, w),
                               np.array([0, ids.size], np.int32), 0, 1, ADAM["lr"], ADAM["beta1"],
                               ADAM["beta2"], ADAM["eps"], t)
    for full, sh in ((Wa, sw), (ma, sm), (va, sv)):
        assert np.array_equal(oracle.assemble_by_column(sh, V, D, P).view(np.uint32), full.view(np.uint32))


# --------------------------------------------------------- communication cost
_SCHEMES = ("alltoall", "allreduce", "ps", "allgather")


def pin_comm_cost_golden():
    """Table 2 evaluated by hand."""
    g = load_golden("comm_cost_worked.txt")
    for case in ("case_a", "case_b", "case_c"):
        c = g[case]
        got = [oracle.comm_cost(s, c["N"], c["M"], c["alpha"], c["B"], c["beta"], S=c["S"]) for s in _SCHEMES]
        assert np.allclose(got, c["cost"], rtol=1e-15, atol=0), (case, got)


def pin_comm_cost_claims():
    """What Sec. 4.1.2 concludes from Table 2, over a grid of settings:
      for N > 1 and N >= n (S = n servers) and alpha <= 1, AlltoAll is no slower than AllReduce
      (equal at alpha = 1) and faster than PS;
      with N = 2, AllGather undercuts AlltoAll by exactly one start latency;
      without latency, AllGather's time grows linearly in N while AlltoAll's stays below
      2 alpha M / B (AllGather / AlltoAll = N / 2);
      with one worker nothing is exchanged except under PS."""
    M, B = 1e9, 12.5e9
    cost = {s: (lambda N, alpha, beta, S=1, s=s: oracle.comm_cost(s, N, M, alpha, B, beta, S=S)) for s in _SCHEMES}
    for N in (2, 3, 4, 8, 16, 64):
        for n in sorted({1, 2, N // 2 or 1, N}):
            for alpha in (0.0, 0.003, 0.1, 0.4, 1.0):
                for beta in (0.0, 1e-6, 1e-4, 1e-2):
                    a2a = cost["alltoall"](N, alpha, beta)
                    assert a2a <= cost["allreduce"](N, alpha, beta) * (1 + 1e-15)
                    ps = cost["ps"](N, alpha, beta, S=n)
                    assert a2a < ps if alpha > 0 or beta > 0 else a2a == ps == 0.0
                    if alpha == 1.0:
                        assert np.isclose(a2a, cost["allreduce"](N, alpha, beta), rtol=1e-15)
        for alpha in (0.01, 0.5):
            ag, a2a = cost["allgather"](N, alpha, 0.0), cost["alltoall"](N, alpha, 0.0)
            assert np.isclose(ag, (N - 1) * alpha * M / B, rtol=1e-15)
            assert np.isclose(ag / a2a, N / 2, rtol=1e-14) and a2a < 2 * alpha * M / B
    for beta in (1e-6, 1e-3):
        assert np.isclose(cost["alltoall"](2, 0.2, beta) - cost["allgather"](2, 0.2, beta), beta, rtol=1e-9)
    for s in ("alltoall", "allreduce", "allgather"):
        assert cost[s](1, 0.3, 1e-3) == 0.0
    assert np.isclose(cost["ps"](1, 0.3, 1e-3, S=1), 2 * (0.3 * M / B + 1e-3), rtol=1e-15)
