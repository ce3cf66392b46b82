"""The two-stream step schedule gives bitwise the same table, moments and
lookups as running the four calls one after another."""
import numpy as np
import pytest
import torch

from paper_2110_09132_amd.step import EmbeddingTable, StepPipeline
from workloads import configs, gen

pytestmark = pytest.mark.gpu


def run(overlap, steps=7):
    torch.cuda.synchronize()
    specs = [configs.TableSpec(20000, 128, 6000, "zipf", 1.05, "f32", 0.01, 8, "mod", 61),
             configs.TableSpec(5000, 64, 3000, "uniform", 0.0, "bf16", 0.01, 3, "range", 62)]
    tables, batches = [], []
    for sp in specs:
        W = torch.from_numpy(configs.make_weights(sp)).cuda()
        gdt = torch.bfloat16 if sp.grad_dtype == "bf16" else torch.float32
        tables.append(EmbeddingTable(W, torch.from_numpy(configs.row_owner(sp)).cuda(), sp.P, sp.T, gdt))
        per = []
        for s in range(3):  # three rotating batches of different sizes
            T = sp.T - 997 * s
            ids, G = configs.make_batch(sp, s, T)
            g = torch.from_numpy(G.view(np.int16)).cuda().view(torch.bfloat16) if G.dtype == np.uint16 \
                else torch.from_numpy(G).cuda()
            per.append((torch.from_numpy(ids).cuda(), g))
        batches.append(per)
    torch.cuda.synchronize()
    pipe = StepPipeline(tables, 1e-3, 0.9, 0.999, 1e-8, overlap=overlap)
    lookups = []
    for t in range(1, steps + 1):
        pipe.step([batches[k][t % 3] for k in range(len(specs))], t)
        # the lookup of step t is read on the main stream before step t+1's lookup overwrites it
        lookups.append([tb.lookup[: batches[k][t % 3][0].numel()].clone() for k, tb in enumerate(tables)])
    pipe.finish()
    torch.cuda.synchronize()
    return [(tb.W.cpu().numpy(), tb.M.cpu().numpy(), tb.S.cpu().numpy()) for tb in tables], \
           [[x.cpu().numpy() for x in l] for l in lookups]


def test_overlapped_schedule_equals_sequential():
    a, la = run(True)
    b, lb = run(False)
    for x, y in zip(a, b):
        for u, v in zip(x, y):
            assert np.array_equal(u.view(np.uint32), v.view(np.uint32))
    for x, y in zip(la, lb):
        for u, v in zip(x, y):
            assert np.array_equal(u.view(np.uint32), v.view(np.uint32))
