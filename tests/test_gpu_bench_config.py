"""The step exactly as the benchmark runs it, at the full size of every workload and for every table
of it: the step executor (owner-major coalesce, sort and reduction on side streams) under each
schedule the benchmark's tuner may pick (events or step signals; two buffer sets with one sort
stream, four with two, with or without each sort stream running its own reductions, or six with
three sort streams running their own reductions), and the
split schedule of Vertical Sparse Scheduling (Algorithm 1: prior rows updated before the next
lookup, delayed rows beside it), a few steps in a row, checked against the oracle:
  - each step's send layout (ids, counts, offsets; with the split, the 2P groups of the prior and
    delayed rows) bit-exact against the oracle's owner-major pack (or split pack) of its coalesce,
    and the rows within the fp32 summation bound;
  - each step's lookup against the table as the previous steps left it (sampled rows, replayed on
    the CPU: bit-exact at the first step, then to the Adam tolerance);
  - W, m, v after the steps against the oracle's Adam applied to the GPU's own send rows, on a
    sample of touched rows, with the update W_after - W_before judged on its own scale, and
    untouched rows bit-identical."""
import functools

import numpy as np
import pytest
import torch

import oracle
import paper_2110_09132_amd as emb
import tolerance
from gpu_helpers import host, to_dev
from paper_2110_09132_amd.step import EmbeddingTable, StepPipeline
from workloads import configs

pytestmark = pytest.mark.gpu

# (coalesce, cross-stream order, buffer sets, paired)
SCHEDULES = [("by_owner", "events", 2, False), ("by_owner", "events", 4, False),
             ("by_owner", "signals", 2, False), ("by_owner", "signals", 4, False),
             ("by_owner", "events", 4, True), ("by_owner", "signals", 4, True),
             ("by_owner", "events", 6, True), ("by_owner", "signals", 6, True),
             ("split", "events", 2, False), ("split", "signals", 2, False), ("split", "signals", 4, False)]
CASES = [(w,) + s for w in configs.WORKLOADS for s in SCHEDULES]


@functools.lru_cache(maxsize=2)
def weights(name, k):
    return configs.make_weights(configs.WORKLOADS[name].tables[k])


@functools.lru_cache(maxsize=16)
def batch(name, k, step):
    return configs.make_batch(configs.WORKLOADS[name].tables[k], 500 + step)


@pytest.mark.parametrize("name,kind,order,sets,paired", CASES,
                         ids=[f"{w}-{k}-{o}-{s}sets{'-paired' if p else ''}" for w, k, o, s, p in CASES])
def test_bench_schedule_full_size(name, kind, order, sets, paired):
    wl = configs.WORKLOADS[name]
    split = kind == "split"
    steps = sets  # every step's send buffers survive until the end
    print(f"[{name}] {kind}, {order}, {sets} sets{', paired' if paired else ''}, {steps} steps", flush=True)
    nt = len(wl.tables)
    W0s = [weights(name, k) for k in range(nt)]
    owns = [configs.row_owner(sp) for sp in wl.tables]
    tbs = []
    for k, sp in enumerate(wl.tables):
        gdt = torch.bfloat16 if sp.grad_dtype == "bf16" else torch.float32
        tbs.append(EmbeddingTable(to_dev(W0s[k]), to_dev(owns[k]), sp.P, sp.T, gdt, sets=sets))
    st = emb.new_status()
    pipe = StepPipeline(tbs, wl.lr, wl.beta1, wl.beta2, wl.eps, overlap=True, dev_status=st, split=split,
                        signals=order == "signals", sets=sets,
                        sort_streams=(sets // 2 if sets in (4, 6) else 1) if not split else 1, paired=paired)
    # batches of steps 0 .. steps (the last one is only the split's next batch)
    host_batches = [[batch(name, k, s) for k in range(nt)] for s in range(steps + 1)]
    dev_batches = [[(to_dev(ids), to_dev(G)) for ids, G in hb] for hb in host_batches]
    rng = np.random.default_rng(7)
    looked = []
    for s in range(steps):
        pipe.step(dev_batches[s], s + 1, next_ids=[x[0] for x in dev_batches[s + 1]] if split else None)
        # the lookups of step s, sampled, read on the main stream before the next step's lookup overwrites them
        pos = np.sort(rng.choice(wl.tables[0].T, 256, replace=False))
        looked.append([(pos, tb.lookup[torch.from_numpy(pos).to(tb.lookup.device)].clone()) for tb in tbs])
    pipe.finish()
    torch.cuda.synchronize()
    assert int(st.item()) == 0

    for k, (sp, tb, W0, own) in enumerate(zip(wl.tables, tbs, W0s, owns)):
        bf16 = sp.grad_dtype == "bf16"
        G_of = [host_batches[s][k] for s in range(steps + 1)]
        # rows to replay on the CPU: some of every batch, plus untouched ones
        touched = np.unique(np.concatenate([ids for ids, _ in G_of[:steps]]))
        sample = np.unique(np.concatenate([rng.choice(touched, min(384, touched.size), replace=False)] +
                                          [G_of[s][0][looked[s][k][0]] for s in range(steps)]))
        untouched = np.setdiff1d(rng.choice(sp.V, min(sp.V, 2048), replace=False), touched)[:64]
        idx = {int(r): i for i, r in enumerate(sample)}
        Wc = W0[sample].copy()
        Mc = np.zeros_like(Wc)
        Sc = np.zeros_like(Wc)
        for s in range(steps):
            ids, G = G_of[s]
            # the lookup of step s reads the rows as the updates of steps < s left them: bit for bit at
            # the first step, then within the Adam tolerance of the replay (an update is ~lr per element,
            # far above the tolerance, so a lookup that missed an update fails)
            pos, got = looked[s][k]
            want = Wc[[idx[int(i)] for i in ids[pos]]]
            if s == 0:
                assert np.array_equal(host(got).view(np.uint32), want.view(np.uint32)), f"table {k}: lookup of step 1"
            else:
                tolerance.assert_rows_close(host(got), want, what=f"table {k}: lookup of step {s + 1}")
            # the send layout of step s (buffer set s) against the oracle
            sid, srows, cnt, offs = tb.send[s]
            orc = oracle.coalesce(ids, G, sp.V, grad_is_bf16=bf16)
            if split:
                pk = oracle.split_pack(orc["uniq_ids"], orc["uniq_grad"], G_of[s + 1][0], own, sp.P)
                ng = 2 * sp.P
            else:
                pk = oracle.pack_by_owner(orc["uniq_ids"], orc["uniq_grad"], own, sp.P)
                ng = sp.P
            U = orc["U"]
            offs_h = host(offs)[:ng + 1]
            assert np.array_equal(offs_h, pk["send_offsets"]), f"table {k} step {s + 1}: send offsets"
            assert np.array_equal(host(cnt)[:ng], pk["send_counts"]), f"table {k} step {s + 1}: send counts"
            got_ids = host(sid[:U])
            assert np.array_equal(got_ids, pk["send_ids"]), f"table {k} step {s + 1}: send ids"
            rows_h = host(srows[:U])
            order_u = np.searchsorted(orc["uniq_ids"], got_ids)
            tolerance.assert_grad_close(rows_h, orc["sum_f64"][order_u], orc["absum"][order_u],
                                        what=f"table {k} step {s + 1}: send rows")
            # the oracle's Adam on the sampled rows with the GPU's own send rows of this step (with the
            # split the prior and the delayed part, same step, touch disjoint rows: one call covers both)
            sel = np.nonzero(np.isin(got_ids, sample))[0]
            local = np.array([idx[int(i)] for i in got_ids[sel]], dtype=np.int32)
            oracle.sparse_adam(Wc, Mc, Sc, local, rows_h[sel], np.array([0, sel.size], np.int32), 0, 1, wl.lr,
                               wl.beta1, wl.beta2, wl.eps, s + 1)
        sel_dev = torch.from_numpy(sample.astype(np.int64)).to(tb.W.device)
        Wg = host(tb.W[sel_dev])
        for t, ref, what in ((Wg, Wc, "table"), (host(tb.M[sel_dev]), Mc, "exp_avg"),
                             (host(tb.S[sel_dev]), Sc, "exp_avg_sq")):
            tolerance.assert_rows_close(t, ref, what=f"table {k}: {what}")
        tolerance.assert_update_close(Wg, W0[sample], Wc, ulps=steps, what=f"table {k}: update over {steps} steps")
        un_dev = torch.from_numpy(untouched.astype(np.int64)).to(tb.W.device)
        assert np.array_equal(host(tb.W[un_dev]).view(np.uint32), W0[untouched].view(np.uint32))
        assert not host(tb.M[un_dev]).any() and not host(tb.S[un_dev]).any()
