"""The overlapped step schedules give bitwise the same table, moments and
lookups as running their calls one after another on one stream, with the
cross-stream order kept by events or by step signals, and with each step
enqueued from two host threads (emb_train_step_queued); the
owner-major schedule (coalesce straight into the send layout) agrees with
coalesce-then-pack, and the prior / delayed split with one update, to the
fp32 tolerance (their sums add in another grouping)."""
import numpy as np
import pytest
import torch

import tolerance
from paper_2110_09132_amd.step import EmbeddingTable, StepPipeline
from workloads import configs, gen

pytestmark = pytest.mark.gpu


def run(overlap, by_owner, steps=9, split=False, signals=False, sort_streams=1, sets=2, paired=False, queued=False,
        flush_each=True):
    """flush_each (queued): wait for the worker after every step, so that its lookup can be read; else only
    the last step's lookup is read, and the worker's enqueue runs beside the next steps' sorts."""
    torch.cuda.synchronize()
    specs = [configs.TableSpec(20000, 128, 6000, "zipf", 1.05, "f32", 0.01, 8, "mod", 61),
             configs.TableSpec(5000, 64, 3000, "uniform", 0.0, "bf16", 0.01, 3, "range", 62)]
    tables, batches = [], []
    for sp in specs:
        W = torch.from_numpy(configs.make_weights(sp)).cuda()
        gdt = torch.bfloat16 if sp.grad_dtype == "bf16" else torch.float32
        tables.append(EmbeddingTable(W, torch.from_numpy(configs.row_owner(sp)).cuda(), sp.P, sp.T, gdt, sets=sets))
        per = []
        for s in range(3):  # three rotating batches of different sizes
            T = sp.T - 997 * s
            ids, G = configs.make_batch(sp, s, T)
            g = torch.from_numpy(G.view(np.int16)).cuda().view(torch.bfloat16) if G.dtype == np.uint16 \
                else torch.from_numpy(G).cuda()
            per.append((torch.from_numpy(ids).cuda(), g))
        batches.append(per)
    torch.cuda.synchronize()
    pipe = StepPipeline(tables, 1e-3, 0.9, 0.999, 1e-8, overlap=overlap, by_owner=by_owner, split=split,
                        signals=signals, sort_streams=sort_streams, sets=sets, paired=paired, queued=queued)
    lookups = []
    empty = torch.zeros(0, dtype=torch.int32, device="cuda")
    for t in range(1, steps + 1):
        nxt = [batches[k][(t + 1) % 3][0] if t < steps else empty for k in range(len(specs))]
        pipe.step([batches[k][t % 3] for k in range(len(specs))], t, next_ids=nxt if split else None)
        if queued:
            if not flush_each and t < steps:
                continue
            pipe.queue.flush()  # the worker has enqueued this step's lookup
        # the lookup of step t is read on the main stream before step t+1's lookup overwrites it
        lookups.append([tb.lookup[: batches[k][t % 3][0].numel()].clone() for k, tb in enumerate(tables)])
    pipe.finish()
    torch.cuda.synchronize()
    return [(tb.W.cpu().numpy(), tb.M.cpu().numpy(), tb.S.cpu().numpy()) for tb in tables], \
           [[x.cpu().numpy() for x in l] for l in lookups]


@pytest.mark.parametrize("signals", [True, False], ids=["signals", "events"])
@pytest.mark.parametrize("by_owner,split", [(False, False), (True, False), (True, True)])
def test_overlapped_schedule_equals_sequential(by_owner, split, signals):
    print(f"overlapped vs sequential by_owner={by_owner} split={split} signals={signals}", flush=True)
    a, la = run(True, by_owner, split=split, signals=signals)
    b, lb = run(False, by_owner, split=split)
    for x, y in zip(a, b):
        for u, v in zip(x, y):
            assert np.array_equal(u.view(np.uint32), v.view(np.uint32))
    for x, y in zip(la, lb):
        for u, v in zip(x, y):
            assert np.array_equal(u.view(np.uint32), v.view(np.uint32))


@pytest.mark.parametrize("sets,paired", [(2, False), (4, False), (4, True)])
@pytest.mark.parametrize("signals", [False, True], ids=["events", "signals"])
def test_two_sort_streams_equal_sequential(signals, sets, paired):
    print(f"two sort streams, signals={signals}, sets={sets}, paired={paired}", flush=True)
    a, la = run(True, True, signals=signals, sort_streams=2, sets=sets, paired=paired)
    b, lb = run(False, True)
    for x, y in zip(a, b):
        for u, v in zip(x, y):
            assert np.array_equal(u.view(np.uint32), v.view(np.uint32))
    for x, y in zip(la, lb):
        for u, v in zip(x, y):
            assert np.array_equal(u.view(np.uint32), v.view(np.uint32))


@pytest.mark.parametrize("sets,sort_streams,paired", [(2, 1, False), (4, 2, False), (4, 2, True), (6, 3, True)])
@pytest.mark.parametrize("flush_each", [True, False], ids=["flush-each", "flush-last"])
def test_queued_enqueue_equals_sequential(sets, sort_streams, paired, flush_each):
    print(f"queued, sets={sets}, sort streams={sort_streams}, paired={paired}, flush_each={flush_each}", flush=True)
    a, la = run(True, True, steps=12, sort_streams=sort_streams, sets=sets, paired=paired, queued=True,
                flush_each=flush_each)
    b, lb = run(False, True, steps=12)
    for x, y in zip(a, b):
        for u, v in zip(x, y):
            assert np.array_equal(u.view(np.uint32), v.view(np.uint32))
    lb = lb if flush_each else lb[-1:]
    assert len(la) == len(lb)
    for x, y in zip(la, lb):
        for u, v in zip(x, y):
            assert np.array_equal(u.view(np.uint32), v.view(np.uint32))


def test_owner_major_schedule_matches_coalesce_then_pack():
    a, la = run(True, True)
    b, lb = run(False, False)
    for x, y in zip(a, b):
        for u, v, name in zip(x, y, ("table", "exp_avg", "exp_avg_sq")):
            tolerance.assert_rows_close(u, v, tolerance.RTOL_F32, name)
    for x, y in zip(la, lb):
        for u, v in zip(x, y):
            tolerance.assert_rows_close(u, v, tolerance.RTOL_F32, "lookup")


def test_split_schedule_matches_one_update():
    """The prior and delayed updates of the split (same step t) give the table of one update on all
    rows, to the fp32 tolerance: each row gets the same Adam arithmetic, and only the grouping of
    the fp32 additions of a row's gradient sum follows the (split) sorted positions."""
    a, la = run(True, True, split=True)
    b, lb = run(False, True, split=False)
    for x, y in zip(a, b):
        for u, v, name in zip(x, y, ("table", "exp_avg", "exp_avg_sq")):
            tolerance.assert_rows_close(u, v, tolerance.RTOL_F32, name)
    for x, y in zip(la, lb):
        for u, v in zip(x, y):
            tolerance.assert_rows_close(u, v, tolerance.RTOL_F32, "lookup")


def test_failed_step_leaves_no_wait_blocked():
    """A step that fails on the host part-way (here: the pack workspace of one call is declared
    too small, after the coalesce was enqueued) marks its stages done, so the later steps of the
    same step-signal handle run to the end and give the table of the sequential schedule when
    the failed step is left out of both."""
    import paper_2110_09132_amd as emb

    def go(overlap):
        torch.cuda.synchronize()
        sp = configs.TableSpec(3000, 64, 2000, "zipf", 1.1, "f32", 0.01, 4, "mod", 63)
        tb = EmbeddingTable(torch.from_numpy(configs.make_weights(sp)).cuda(),
                            torch.from_numpy(configs.row_owner(sp)).cuda(), sp.P, sp.T)
        pipe = StepPipeline([tb], 1e-3, 0.9, 0.999, 1e-8, overlap=overlap, by_owner=False, signals=True)
        bs = []
        for s in range(3):
            ids, G = configs.make_batch(sp, s)
            bs.append([(torch.from_numpy(ids).cuda(), torch.from_numpy(G).cuda())])
        t = 0
        for k in range(6):
            if k == 2 and overlap:
                i = pipe.count % pipe.sets
                good = pipe.args[0][i].ws_pack_bytes
                pipe.args[0][i].ws_pack_bytes = 1
                with pytest.raises(emb.EmbError):
                    pipe.step(bs[k % 3], t + 1)
                pipe.args[0][i].ws_pack_bytes = good
                pipe.count += 1  # the failed call's buffer set is skipped as if used
                continue
            if k == 2:
                continue
            t += 1
            pipe.step(bs[k % 3], t)
        pipe.finish()
        torch.cuda.synchronize()
        return tb.W.cpu().numpy()
    print("failed step, then four more steps", flush=True)
    a = go(True)
    b = go(False)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("by_owner,split", [(False, False), (True, True)])
def test_three_sets_with_signals_equal_sequential(by_owner, split):
    """An odd number of buffer sets (one sort stream), including the split, whose lookup waits for
    the delayed update two steps back whatever the number of sets."""
    print(f"three sets by_owner={by_owner} split={split}", flush=True)
    a, la = run(True, by_owner, split=split, signals=True, sets=3)
    b, lb = run(False, by_owner, split=split)
    for x, y in zip(a, b):
        for u, v in zip(x, y):
            assert np.array_equal(u.view(np.uint32), v.view(np.uint32))
    for x, y in zip(la, lb):
        for u, v in zip(x, y):
            assert np.array_equal(u.view(np.uint32), v.view(np.uint32))
