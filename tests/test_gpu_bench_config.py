"""The step exactly as the benchmark runs it, at the full size of the two
largest workloads: the step executor (owner-major coalesce, sort and reduction
on side streams) under each schedule the benchmark may pick (events or step
signals, two buffer sets with one sort stream or four with two), a few steps
in a row, checked against the oracle:
  - each step's send layout (ids, counts, offsets) bit-exact against the
    oracle's owner-major pack of its coalesce, and the rows within the fp32
    summation bound;
  - each step's lookup against the table as the previous steps left it
    (sampled rows, replayed on the CPU: bit-exact at the first step, then to
    the Adam tolerance);
  - W, m, v after the steps against the oracle's Adam applied to the GPU's own
    send rows, on a sample of touched rows, and untouched rows bit-identical."""
import numpy as np
import pytest
import torch

import oracle
import tolerance
from gpu_helpers import host, to_dev
from paper_2110_09132_amd.step import EmbeddingTable, StepPipeline
from workloads import configs

pytestmark = pytest.mark.gpu

SCHEDULES = [("events", 2, 1, False), ("signals", 4, 2, False), ("events", 4, 2, False), ("signals", 4, 2, True)]


@pytest.mark.parametrize("order,sets,sort_streams,paired", SCHEDULES,
                         ids=[f"{o}-{s}sets{'-paired' if p else ''}" for o, s, _, p in SCHEDULES])
@pytest.mark.parametrize("name", ["lowdup_uniform", "lowdup_zipf13"])
def test_bench_schedule_full_size(name, order, sets, sort_streams, paired):
    wl = configs.WORKLOADS[name]
    sp = wl.tables[0]
    steps = sets  # every step's send buffers survive until the end
    print(f"[{name}] {order}, {sets} sets, {steps} steps, V={sp.V} D={sp.D} T={sp.T} P={sp.P}", flush=True)
    W0 = configs.make_weights(sp)
    own = configs.row_owner(sp)
    tb = EmbeddingTable(to_dev(W0), to_dev(own), sp.P, sp.T, sets=sets)
    pipe = StepPipeline([tb], wl.lr, wl.beta1, wl.beta2, wl.eps, overlap=True, signals=order == "signals",
                        sets=sets, sort_streams=sort_streams, paired=paired)
    batches = [configs.make_batch(sp, 500 + k) for k in range(steps)]
    dev_batches = [(to_dev(ids), to_dev(G)) for ids, G in batches]
    rng = np.random.default_rng(7)
    looked = []
    for k in range(steps):
        pipe.step([dev_batches[k]], k + 1)
        # the lookup of step k, sampled, read on the main stream before the next step's lookup overwrites it
        pos = np.sort(rng.choice(sp.T, 256, replace=False))
        looked.append((pos, tb.lookup[torch.from_numpy(pos).to(tb.lookup.device)].clone()))
    pipe.finish()
    torch.cuda.synchronize()

    # rows to replay on the CPU: some of every batch, plus untouched ones
    touched = np.unique(np.concatenate([ids for ids, _ in batches]))
    sample = np.unique(np.concatenate([rng.choice(touched, 384, replace=False)] +
                                      [ids[pos] for (ids, _), (pos, _) in zip(batches, looked)]))
    untouched = np.setdiff1d(rng.choice(sp.V, 2048, replace=False), touched)[:64]
    idx = {int(r): i for i, r in enumerate(sample)}
    Wc = W0[sample].copy()
    Mc = np.zeros_like(Wc)
    Sc = np.zeros_like(Wc)
    for k, (ids, G) in enumerate(batches):
        # the lookup of step k reads the rows as the updates of steps < k left them: bit for bit at
        # the first step, then within the Adam tolerance of the replay (an update is ~lr per element,
        # far above the tolerance, so a lookup that missed an update fails)
        pos, got = looked[k]
        want = Wc[[idx[int(i)] for i in ids[pos]]]
        if k == 0:
            assert np.array_equal(host(got).view(np.uint32), want.view(np.uint32)), "lookup of step 1"
        else:
            tolerance.assert_rows_close(host(got), want, what=f"lookup of step {k + 1}")
        # the send layout of step k (buffer set k) against the oracle
        sid, srows, cnt, offs = tb.send[k]
        orc = oracle.coalesce(ids, G, sp.V)
        pk = oracle.pack_by_owner(orc["uniq_ids"], orc["uniq_grad"], own, sp.P)
        U = orc["U"]
        offs_h = host(offs)[:sp.P + 1]
        assert np.array_equal(offs_h, pk["send_offsets"]) and np.array_equal(host(cnt)[:sp.P], pk["send_counts"])
        got_ids = host(sid[:U])
        assert np.array_equal(got_ids, pk["send_ids"])
        rows_h = host(srows[:U])
        order_u = np.searchsorted(orc["uniq_ids"], got_ids)
        tolerance.assert_grad_close(rows_h, orc["sum_f64"][order_u], orc["absum"][order_u])
        # the oracle's Adam on the sampled rows with the GPU's own send rows of this step
        sel = np.nonzero(np.isin(got_ids, sample))[0]
        local = np.array([idx[int(i)] for i in got_ids[sel]], dtype=np.int32)
        oracle.sparse_adam(Wc, Mc, Sc, local, rows_h[sel], np.array([0, sel.size], np.int32), 0, 1, wl.lr,
                           wl.beta1, wl.beta2, wl.eps, k + 1)
    sel_dev = torch.from_numpy(sample.astype(np.int64)).to(tb.W.device)
    for t, ref, what in ((tb.W, Wc, "table"), (tb.M, Mc, "exp_avg"), (tb.S, Sc, "exp_avg_sq")):
        tolerance.assert_rows_close(host(t[sel_dev]), ref, what=what)
    un_dev = torch.from_numpy(untouched.astype(np.int64)).to(tb.W.device)
    assert np.array_equal(host(tb.W[un_dev]).view(np.uint32), W0[untouched].view(np.uint32))
    assert not host(tb.M[un_dev]).any() and not host(tb.S[un_dev]).any()
