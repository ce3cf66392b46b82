"""Steps captured into a HIP graph (StepGraph: stream capture of the step executor's calls, events for
the cross-stream order, the update's coefficients read from device memory) replayed several times,
with other GPU work and synchronisations between the replays:
  - after the first replay the tables and every step's send layout against the oracle (the steps'
    send buffers, W, m, v on sampled rows with the update on its own scale, untouched rows
    bit-identical);
  - after every replay the tables, the moments and the last step's lookup and send layout bit for bit
    equal to the same steps run without a graph (same kernels in the same order), so that each
    replay applies the step numbers it is given (Sec. 5.7: the step count grows every iteration)."""
import numpy as np
import pytest
import torch

import paper_2110_09132_amd as emb
from gpu_helpers import check_steps_against_oracle, host, to_dev
from paper_2110_09132_amd.step import EmbeddingTable, StepGraph, StepPipeline
from workloads import configs

pytestmark = pytest.mark.gpu


def bits(t):
    return host(t).view(np.uint32) if t.dtype == torch.float32 else host(t)


@pytest.mark.parametrize("name,sets,sort_streams", [("tiny", 4, 2), ("transformer_shared_vocab", 4, 2),
                                                   ("two_table_translation", 6, 3)])
def test_graph_replays(name, sets, sort_streams):
    wl = configs.WORKLOADS[name]
    n = sets  # one step per buffer set: every step's send buffers survive a replay
    print(f"[{name}] graph of {n} steps, {sets} sets, {sort_streams} sort streams", flush=True)
    nt = len(wl.tables)
    W0s = [configs.make_weights(sp) for sp in wl.tables]
    owns = [configs.row_owner(sp) for sp in wl.tables]
    host_batches = [[configs.make_batch(sp, 700 + s) for sp in wl.tables] for s in range(n)]
    dev_batches = [[(to_dev(ids), to_dev(G)) for ids, G in hb] for hb in host_batches]

    def tables():
        out = []
        for k, sp in enumerate(wl.tables):
            gdt = torch.bfloat16 if sp.grad_dtype == "bf16" else torch.float32
            out.append(EmbeddingTable(to_dev(W0s[k]), to_dev(owns[k]), sp.P, sp.T, gdt, sets=sets))
        return out

    eager_tbs, graph_tbs = tables(), tables()
    st_e, st_g = emb.new_status(), emb.new_status()
    eager = StepPipeline(eager_tbs, wl.lr, wl.beta1, wl.beta2, wl.eps, overlap=True, dev_status=st_e, sets=sets,
                         sort_streams=sort_streams, paired=True)
    # eager steps have run in the process before the capture (warm-up of a scratch table)
    scratch = tables()
    warm = StepPipeline(scratch, wl.lr, wl.beta1, wl.beta2, wl.eps, overlap=True, sets=sets,
                        sort_streams=sort_streams, paired=True)
    warm.step(dev_batches[0], 1)
    warm.finish()
    torch.cuda.synchronize()
    del warm, scratch
    graph = StepGraph(graph_tbs, wl.lr, wl.beta1, wl.beta2, wl.eps, dev_batches, sets=sets,
                      sort_streams=sort_streams, paired=True, dev_status=st_g)
    torch.cuda.synchronize()
    # the capture itself ran nothing
    for k in range(nt):
        assert np.array_equal(bits(graph_tbs[k].W), W0s[k].view(np.uint32))
    for r in range(3):
        for s in range(n):
            eager.step(dev_batches[s], r * n + s + 1)
        eager.finish()
        graph.replay(r * n + 1)
        torch.cuda.synchronize()
        x = torch.arange(1 << 16, device="cuda", dtype=torch.float32)  # other work between the replays
        assert float((x * 2).sum().item()) == float((1 << 16) * ((1 << 16) - 1))
        torch.cuda.synchronize()
        assert int(st_e.item()) == 0 and int(st_g.item()) == 0
        if r == 0:
            check_steps_against_oracle(wl, graph_tbs, W0s, owns, host_batches, n, False)
        for k in range(nt):
            e, g = eager_tbs[k], graph_tbs[k]
            for a, b, what in ((e.W, g.W, "table"), (e.M, g.M, "exp_avg"), (e.S, g.S, "exp_avg_sq"),
                               (e.lookup, g.lookup, "lookup")):
                assert np.array_equal(bits(a), bits(b)), f"replay {r + 1}, table {k}: {what}"
            P = wl.tables[k].P
            for i in range(sets):  # ids, rows, counts, offsets (the entries the call defines)
                U = int(e.send[i][3][P].item())
                for a, b, m in zip(e.send[i], g.send[i], (U, U, P, P + 1)):
                    assert np.array_equal(bits(a[:m]), bits(b[:m])), f"replay {r + 1}, set {i}"


def test_capture_refuses_step_signals_and_timing():
    """Under stream capture the executor takes events only and no timing pairs: it refuses before
    anything is enqueued, so the capture stays empty and ends normally.  One stream only (no side
    stream joins the capture)."""
    import ctypes
    wl = configs.WORKLOADS["tiny"]
    sp = wl.tables[0]
    tb = EmbeddingTable(to_dev(configs.make_weights(sp)), to_dev(configs.row_owner(sp)), sp.P, sp.T, sets=2)
    ids, G = configs.make_batch(sp, 1)
    ids_d, G_d = to_dev(ids), to_dev(G)
    s = torch.cuda.Stream()
    sig = emb.StepSignals()
    t0, t1 = emb.Event(timing=True), emb.Event(timing=True)
    with torch.cuda.stream(s):
        pipe = StepPipeline([tb], wl.lr, wl.beta1, wl.beta2, wl.eps, overlap=False, sets=2)
        a, sc = pipe.args[0][0], pipe.sched[0][0]
        a.ids, a.T, a.grad, a.grad_dtype, a.step = ids_d.data_ptr(), sp.T, G_d.data_ptr(), emb.EMB_F32, 1
        for use_signals in (True, False):
            sc.signals = sig.handle if use_signals else None
            sc.timing[6], sc.timing[7] = (None, None) if use_signals else (t0.handle, t1.handle)
            g = torch.cuda.CUDAGraph()
            g.capture_begin()
            r = emb.lib.emb_train_step(ctypes.byref(a), ctypes.byref(sc))
            g.capture_end()
            assert r == emb.EMB_ERR_UNSUPPORTED
            g.replay()  # an empty graph
    torch.cuda.synchronize()
    del sig
