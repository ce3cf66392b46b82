"""The step exactly as the benchmark runs it, at the full size of every workload and for every table
of it: the step executor (owner-major coalesce, sort and reduction on side streams) under each
schedule the benchmark's tuner may pick (events or step signals; two buffer sets with one sort
stream, four with two, with or without each sort stream running its own reductions, or six with
three sort streams running their own reductions; four or six with each step enqueued from two host
threads), and the
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

import paper_2110_09132_amd as emb
from gpu_helpers import check_steps_against_oracle, to_dev
from paper_2110_09132_amd.step import EmbeddingTable, StepPipeline
from workloads import configs

pytestmark = pytest.mark.gpu

# (coalesce, cross-stream order, buffer sets, paired)
SCHEDULES = [("by_owner", "events", 2, False), ("by_owner", "events", 4, False),
             ("by_owner", "signals", 2, False), ("by_owner", "signals", 4, False),
             ("by_owner", "events", 4, True), ("by_owner", "signals", 4, True),
             ("by_owner", "events", 6, True), ("by_owner", "signals", 6, True),
             ("by_owner", "queued", 4, True), ("by_owner", "queued", 6, True),
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
                        signals=order == "signals", queued=order == "queued", sets=sets,
                        sort_streams=(sets // 2 if sets in (4, 6) else 1) if not split else 1, paired=paired)
    # batches of steps 0 .. steps (the last one is only the split's next batch)
    host_batches = [[batch(name, k, s) for k in range(nt)] for s in range(steps + 1)]
    dev_batches = [[(to_dev(ids), to_dev(G)) for ids, G in hb] for hb in host_batches]
    rng = np.random.default_rng(7)
    looked = []
    for s in range(steps):
        pipe.step(dev_batches[s], s + 1, next_ids=[x[0] for x in dev_batches[s + 1]] if split else None)
        if pipe.queue is not None:
            pipe.queue.flush()  # the worker has enqueued this step's lookup, read below
        # the lookups of step s, sampled, read on the main stream before the next step's lookup overwrites them
        pos = np.sort(rng.choice(wl.tables[0].T, 256, replace=False))
        looked.append([(pos, tb.lookup[torch.from_numpy(pos).to(tb.lookup.device)].clone()) for tb in tbs])
    pipe.finish()
    torch.cuda.synchronize()
    assert int(st.item()) == 0

    check_steps_against_oracle(wl, tbs, W0s, owns, host_batches, steps, split, looked)
