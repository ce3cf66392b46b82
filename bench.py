#!/usr/bin/env python3
"""Benchmark of the sparse-embedding hot path on one MI355X.

One step = the whole path over one batch of every table of the workload:
forward gather, coalesce of the per-token gradients, pack by owner shard,
and the row-wise Adam update of all owners' rows (the P shards are simulated
on this GPU).  Inputs (ids, gradients, table, moments) are resident in HBM
before the timed region; batches rotate over a few pre-generated ones.

value = unique gradient rows processed per second over the K timed steps.
The JSON line also carries the step's effective HBM bandwidth under the
algorithmic byte model, the roofline of the dominant kernel (the Adam
update, timed with HIP events on the stream it runs on), and the CPU oracle
timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def byte_model(T, U, D, g, P):
    """Algorithmic bytes of each call: inputs read once, outputs written once,
    repeated table rows counted once; sort scratch is not counted."""
    gather = 4 * T + 4 * D * U + 4 * D * T
    coalesce = 4 * T + g * D * T + 4 * U + 4 * D * U + 4 * (U + 1)
    pack = 12 * U + 8 * D * U + 8 * P
    adam = 4 * U + 4 * D * U + 24 * D * U
    return dict(gather=gather, coalesce=coalesce, pack=pack, adam=adam)


class Table:
    """Device state, pre-generated batches and pre-allocated outputs of one table."""

    def __init__(self, spec, nbatches, torch, emb, configs):
        self.spec = spec
        dev = "cuda"
        V, D, T, P = spec.V, spec.D, spec.T, spec.P
        self.W = torch.from_numpy(configs.make_weights(spec)).to(dev)
        self.M = torch.zeros_like(self.W)
        self.S = torch.zeros_like(self.W)
        self.owner = torch.from_numpy(configs.row_owner(spec)).to(dev)
        self.ids, self.grads = [], []
        for b in range(nbatches):
            ids, G = configs.make_batch(spec, 1000 + b)
            self.ids.append(torch.from_numpy(ids).to(dev))
            if spec.grad_dtype == "bf16":
                self.grads.append(torch.from_numpy(G.view(np.int16)).to(dev).view(torch.bfloat16))
            else:
                self.grads.append(torch.from_numpy(G).to(dev))
        i32, f32 = torch.int32, torch.float32
        self.out = torch.empty((T, D), dtype=f32, device=dev)
        self.coal = (torch.empty(T, dtype=i32, device=dev), torch.empty(T + 1, dtype=i32, device=dev),
                     torch.empty((T, D), dtype=f32, device=dev), torch.empty(1, dtype=i32, device=dev))
        self.pack = (torch.empty(T, dtype=i32, device=dev), torch.empty((T, D), dtype=f32, device=dev),
                     torch.empty(P, dtype=i32, device=dev), torch.empty(P + 1, dtype=i32, device=dev))
        code = emb.EMB_BF16 if spec.grad_dtype == "bf16" else emb.EMB_F32
        self.ws_c = emb.new_workspace(emb.grad_coalesce_workspace_bytes(T, V, D, code), dev)
        self.ws_p = emb.new_workspace(emb.pack_by_owner_workspace_bytes(T, P), dev)
        self.U = [0] * nbatches


def run_step(tables, b, step, wl, emb, ev=None):
    for tb in tables:
        sp = tb.spec
        if ev is not None:
            ev["gather"][0].record()
        emb.gather(tb.W, tb.ids[b], out=tb.out)
        if ev is not None:
            ev["gather"][1].record()
            ev["coalesce"][0].record()
        emb.grad_coalesce(tb.ids[b], tb.grads[b], sp.V, out=tb.coal, workspace=tb.ws_c)
        if ev is not None:
            ev["coalesce"][1].record()
            ev["pack"][0].record()
        uid, _, ug, nu = tb.coal
        emb.pack_by_owner(uid, ug, nu, tb.owner, sp.P, out=tb.pack, workspace=tb.ws_p)
        if ev is not None:
            ev["pack"][1].record()
            ev["adam"][0].record()
        send_ids, send_rows, _, offs = tb.pack
        emb.sparse_adam_apply(tb.W, tb.M, tb.S, send_ids, send_rows, offs, sp.P, 0, sp.P, wl.lr, wl.beta1, wl.beta2,
                              wl.eps, step)
        if ev is not None:
            ev["adam"][1].record()


def cpu_baseline(wl, seconds):
    """The C oracle, single-threaded, on full steps of the same workload (same
    shapes, same generators) until about `seconds` of CPU time have passed."""
    import oracle
    from workloads import configs
    t_total, rows, steps = 0.0, 0, 0
    states = []
    for spec in wl.tables:
        W = configs.make_weights(spec)
        states.append((spec, W, np.zeros_like(W), np.zeros_like(W), configs.row_owner(spec)))
    while True:
        steps += 1
        for spec, W, M, S, own in states:
            ids, G = configs.make_batch(spec, 1000 + steps)
            t0 = time.perf_counter()
            oracle.gather(W, ids)
            c = oracle.coalesce(ids, G, spec.V, grad_is_bf16=spec.grad_dtype == "bf16", want_f64=False)
            pk = oracle.pack_by_owner(c["uniq_ids"], c["uniq_grad"], own, spec.P)
            oracle.sparse_adam(W, M, S, pk["send_ids"], pk["send_rows"], pk["send_offsets"], 0, spec.P, wl.lr,
                               wl.beta1, wl.beta2, wl.eps, steps)
            t_total += time.perf_counter() - t0
            rows += c["U"]
        if t_total >= seconds:
            break
    return dict(value=rows / t_total, unit="unique grad rows/s", cores=1, kind="oracle",
                sample=f"{steps} full steps (gather+coalesce+pack+adam) of workload {wl.name}, "
                       f"single-threaded C oracle, {t_total:.1f} s of timed CPU work")


def host_info():
    model = platform.processor() or ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return dict(cpu=model, nproc=os.cpu_count())


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="lowdup_uniform")
    ap.add_argument("--batches", type=int, default=8)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU's share of the path; runs on more than one GPU are not "
              "supported by this build (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2110_09132_amd as emb
    from workloads import configs

    wl = configs.WORKLOADS[args.workload]
    log(f"workload {wl.name}: {wl.description}")
    tables = [Table(sp, args.batches, torch, emb, configs) for sp in wl.tables]
    torch.cuda.synchronize()

    # unique counts of each batch (outside any timed region)
    for b in range(args.batches):
        for tb in tables:
            emb.grad_coalesce(tb.ids[b], tb.grads[b], tb.spec.V, out=tb.coal, workspace=tb.ws_c)
            torch.cuda.synchronize()
            tb.U[b] = int(tb.coal[3].item())

    step = 0
    for _ in range(args.warmup):
        step += 1
        run_step(tables, step % args.batches, step, wl, emb)
    torch.cuda.synchronize()

    # timed region: exactly K steps
    stream = torch.cuda.current_stream()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    rows = 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        step += 1
        b = step % args.batches
        run_step(tables, b, step, wl, emb)
        rows += sum(tb.U[b] for tb in tables)
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = start.elapsed_time(end)
    ms_step = ms_total / args.steps

    # per-stage timing in a second pass with events between the calls
    stage_ms = {k: 0.0 for k in ("gather", "coalesce", "pack", "adam")}
    for _ in range(args.steps):
        step += 1
        b = step % args.batches
        ev = {k: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for k in stage_ms}
        run_step(tables, b, step, wl, emb, ev)
        torch.cuda.synchronize()
        for k in stage_ms:
            stage_ms[k] += ev[k][0].elapsed_time(ev[k][1]) / args.steps

    # byte model over the timed steps
    bytes_step = {k: 0.0 for k in stage_ms}
    for s in range(args.steps):
        b = (step - 2 * args.steps + 1 + s) % args.batches
        for tb in tables:
            g = 2 if tb.spec.grad_dtype == "bf16" else 4
            bm = byte_model(tb.spec.T, tb.U[b], tb.spec.D, g, tb.spec.P)
            for k in bytes_step:
                bytes_step[k] += bm[k] / args.steps
    total_bytes = sum(bytes_step.values())
    step_gbps = total_bytes / (ms_step * 1e-3) / 1e9
    adam_launches = len(tables)
    adam_gbps = bytes_step["adam"] / (stage_ms["adam"] * 1e-3) / 1e9

    result = {
        "metric": "unique grad rows/sec for coalesce+pack+update; achieved HBM GB/s vs peak",
        "value": rows / (ms_total * 1e-3),
        "unit": "unique grad rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16-in/f32" if any(tb.spec.grad_dtype == "bf16" for tb in tables) else "f32",
        "data": "synthetic (seeded ids and N(0,sigma) gradients, random-init table)",
        "config": {"workload": wl.name, "tables": [dict(V=t.spec.V, D=t.spec.D, T=t.spec.T, P=t.spec.P,
                                                        ids=t.spec.id_law, owner=t.spec.owner_rule)
                                                   for t in tables],
                   "mean_unique_rows_per_step": rows / args.steps, "batches_rotated": args.batches},
        "step_bytes_model": total_bytes,
        "step_hbm_GBps": step_gbps,
        "step_hbm_frac": step_gbps / HBM_PEAK_GBPS,
        "stage_ms": stage_ms,
        "wall_s_timed": wall,
        "roofline": {"bound": "hbm", "kernel": "adam_kernel (emb_sparse_adam_apply)",
                     "achieved": adam_gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": adam_gbps / HBM_PEAK_GBPS, "traffic": None,
                     "bytes_per_launch": bytes_step["adam"] / adam_launches,
                     "avg_launch_us": stage_ms["adam"] * 1e3 / adam_launches},
        "host": host_info(),
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle ...")
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
