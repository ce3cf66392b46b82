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


def byte_model(T, U, D, g, P, by_owner=False, T_next=0):
    """Algorithmic bytes of each call: inputs read once, outputs written once,
    repeated table rows counted once; sort scratch is not counted.  by_owner:
    coalesce writes the send layout itself (emb_grad_coalesce_by_owner), so the
    pack's read and write of the U rows (8 D U) and of the unique ids are gone:
    it reads the ids, the owners of the U distinct ids and the gradient rows,
    and writes the send ids and rows, the segment offsets and the owner counts
    and offsets.  The split (T_next > 0) also reads the next batch's ids."""
    gather = 4 * T + 4 * D * U + 4 * D * T
    adam = 4 * U + 4 * D * U + 24 * D * U
    if by_owner:
        coalesce = 4 * T + 4 * T_next + g * D * T + 8 * U + 4 * D * U + 4 * (U + 1) + 8 * P
        return dict(gather=gather, coalesce=coalesce, pack=0, adam=adam)
    coalesce = 4 * T + g * D * T + 4 * U + 4 * D * U + 4 * (U + 1)
    pack = 12 * U + 8 * D * U + 8 * P
    return dict(gather=gather, coalesce=coalesce, pack=pack, adam=adam)


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


ADAM_KERNEL = "adam_kernel"
COPY_KERNEL = "bitwise_not"  # the reference stream: read N bytes, write N bytes
COPY_MIB = 256
PROFILES = os.path.join(ROOT, "profiles")
TRAFFIC_FILE = os.path.join(PROFILES, "adam_kernel_traffic_lowdup_uniform.json")


def source_hash(path):
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


ADAM_SOURCE = os.path.join(ROOT, "paper_2110_09132_amd", "csrc", "adam.hip")


def copy_reference(torch, mib=COPY_MIB, reps=20):
    """A plain device stream of known size (read mib MiB, write mib MiB), timed with events:
    the bandwidth a streaming kernel reaches here, and the calibration dispatch for the
    HBM byte counters."""
    n = mib * (1 << 20) // 4
    a = torch.randint(0, 1 << 30, (n,), dtype=torch.int32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        torch.bitwise_not(a, out=b)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        torch.bitwise_not(a, out=b)
    e1.record()
    torch.cuda.synchronize()
    return 2 * n * 4 * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9


def measured_traffic():
    """HBM bytes per launch of the update kernel from the committed counter summary, or
    None when there is none or the kernel source changed since the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("adam_source_sha256_16") != source_hash(ADAM_SOURCE):
        return None
    return t.get("traffic_bytes_per_launch")


def _read_csv(path):
    import csv
    with open(path) as f:
        return list(csv.DictReader(f))


def _find(directory, suffix):
    for root, _, files in os.walk(directory):
        for fn in files:
            if fn.endswith(suffix):
                return os.path.join(root, fn)
    raise FileNotFoundError(f"no *{suffix} under {directory}")


def summarize_trace(directory, command, skip=20, steps=200, every=20):
    """Text summary of a rocprofv3 --kernel-trace --stats run (kernel_stats.csv), plus the
    average duration of the update kernel over the timed steps of the bench run (its
    dispatches skip+1 .. skip+steps in launch order, from kernel_trace.csv; skip counts the
    untimed steps before them: the order tuning and the warm-up)."""
    trace = [r for r in _read_csv(_find(directory, "kernel_trace.csv")) if ADAM_KERNEL in r["Kernel_Name"]]
    trace.sort(key=lambda r: int(r["Start_Timestamp"]))
    durs = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in trace[skip:skip + steps]]
    sampled = durs[::every]  # the launches the bench times with events (every `every`-th timed step)
    rows = _read_csv(_find(directory, "kernel_stats.csv"))
    out = [f"command: {command}", "", f"{'kernel':64s} {'calls':>6s} {'avg_us':>9s} {'min_us':>9s} "
           f"{'max_us':>9s} {'share':>6s}"]
    for r in rows:
        name = r["Name"].replace("(anonymous namespace)::", "").split("(")[0][:64]
        out.append(f"{name:64s} {int(r['Calls']):6d} {float(r['AverageNs']) / 1e3:9.2f} "
                   f"{float(r['MinNs']) / 1e3:9.2f} {float(r['MaxNs']) / 1e3:9.2f} {float(r['Percentage']):5.1f}%")
    if durs:
        out += ["", f"{ADAM_KERNEL} over the {len(sampled)} launches the bench times with events (every "
                    f"{every}th timed step): avg {sum(sampled) / len(sampled):.2f} us",
                f"{ADAM_KERNEL} over the {len(durs)} timed steps (dispatches {skip + 1}..{skip + len(durs)}): "
                    f"avg {sum(durs) / len(durs):.2f} us, min {min(durs):.2f} us, max {max(durs):.2f} us"]
    return "\n".join(out) + "\n"


def summarize_pmc(fetch_dir, write_dir, command_fetch, command_write):
    """Scale FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the update kernel by what the same
    counters read for the reference stream of known size."""
    def per_kernel(directory, counter):
        rows = _read_csv(_find(directory, "counter_collection.csv"))
        vals = {}
        for r in rows:
            if r.get("Counter_Name") != counter:
                continue
            name = r["Kernel_Name"]
            key = ADAM_KERNEL if ADAM_KERNEL in name else (COPY_KERNEL if COPY_KERNEL in name else None)
            if key:
                vals.setdefault(key, []).append(float(r["Counter_Value"]))
        return {k: sum(v) / len(v) for k, v in vals.items()}
    f = per_kernel(fetch_dir, "FETCH_SIZE")
    w = per_kernel(write_dir, "WRITE_SIZE")
    copy_bytes = COPY_MIB * (1 << 20)
    f_scale = copy_bytes / (f[COPY_KERNEL] * 1024.0)
    w_scale = copy_bytes / (w[COPY_KERNEL] * 1024.0)
    fetch_b = f[ADAM_KERNEL] * 1024.0 * f_scale
    write_b = w[ADAM_KERNEL] * 1024.0 * w_scale
    return {"kernel": ADAM_KERNEL, "workload": "lowdup_uniform",
            "fetch_kib_per_dispatch": f[ADAM_KERNEL], "write_kib_per_dispatch": w[ADAM_KERNEL],
            "copy_fetch_kib": f[COPY_KERNEL], "copy_write_kib": w[COPY_KERNEL], "copy_bytes_each_way": copy_bytes,
            "fetch_scale": f_scale, "write_scale": w_scale,
            "fetch_bytes_per_launch": fetch_b, "write_bytes_per_launch": write_b,
            "traffic_bytes_per_launch": fetch_b + write_b,
            "adam_source_sha256_16": source_hash(ADAM_SOURCE),
            "command_fetch": command_fetch, "command_write": command_write}


XGMI_LINK_GBPS = 153.0  # one MI355X xGMI link, per direction (one link per peer in an 8-GPU node)


def column_partition_report(torch, emb, sp, tb, batches, U, owner_rows, reps=20):
    """The column-wise partition (Sec. 4.1.1) beside the row-wise one for the first table:
    per-owner bytes of the gradient AlltoAll payload in each partition (ids as int32, rows fp32),
    and the column kernels timed at the table's shape, each over `reps` back-to-back launches
    (outside the timed steps).  Byte models: pack reads and writes U rows; the lookup reads each
    distinct row once, the ids, and writes T rows; the join reads and writes T rows."""
    V, D, P, T = sp.V, sp.D, sp.P, sp.T
    off = emb.column_offsets(D, P)
    widths = np.diff(off)
    row_b, col_b = [], []
    for b, (ids, g) in enumerate(batches):
        rows_p = np.asarray(owner_rows[b], dtype=np.float64)
        row_b.append(rows_p * (4 * D + 4))
        col_b.append(U[b] * (4.0 * widths + 4))

    def balance(per_owner):
        a = np.array(per_owner)
        return {"max_MB": float(a.max(axis=1).mean() / 1e6), "mean_MB": float(a.mean(axis=1).mean() / 1e6),
                "max_over_mean": float((a.max(axis=1) / np.maximum(a.mean(axis=1), 1e-30)).mean())}

    shards = emb.pack_by_column(tb.W, P)[0]
    coalesced = []
    for ids, g in batches:  # coalesced rows of each batch (any order serves the pack)
        uid, seg, ug, nu = emb.grad_coalesce(ids, g, V)
        coalesced.append((ug, nu))
    blocks = torch.empty(T * D, dtype=torch.float32, device="cuda")
    counts = torch.empty(P, dtype=torch.int32, device="cuda")
    look = torch.empty(T * D, dtype=torch.float32, device="cuda")
    joined = torch.empty((T, D), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn):
        for i in range(3):
            fn(i)
        torch.cuda.synchronize()
        e0.record()
        for i in range(reps):
            fn(i)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / reps

    nb = len(batches)
    Um = float(np.mean(U))
    us_pack = timed(lambda i: emb.pack_by_column(coalesced[i % nb][0], P, num_rows=coalesced[i % nb][1],
                                                 out=(blocks, counts)))
    us_look = timed(lambda i: emb.gather_by_column(shards, V, D, P, batches[i % nb][0], out=look))
    us_join = timed(lambda i: emb.assemble_by_column(look, T, D, P, out=joined))
    kern = {}
    for name, us, nbytes in (("pack_by_column", us_pack, 2 * Um * D * 4 + 4),
                             ("gather_by_column", us_look, Um * D * 4 + T * 4 + T * D * 4),
                             ("assemble_by_column", us_join, 2 * T * D * 4)):
        kern[name] = {"avg_launch_us": us, "bytes_model": nbytes, "GBps": nbytes / (us * 1e-6) / 1e9,
                      "frac": nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS}
    del shards
    return {"table": 0, "owner_rule_rowwise": sp.owner_rule, "column_widths": [int(widths.min()), int(widths.max())],
            "payload_rowwise": balance(row_b), "payload_columnwise": balance(col_b), "kernels": kern}


def forward_exchange_report(torch, emb, sp, tb, batches, U, reps=20):
    """The forward pass of the two partitions (Sec. 4.1.1) for the first table, one worker's batch of
    T tokens: row-wise, the worker asks each owner for its U distinct rows (ids out, rows back) and
    expands them to T rows; column-wise, every owner gets the worker's T ids and returns its w(p)
    columns of all T rows.  Bytes the worker sends plus receives (ids int32, rows fp32, its own
    owner's share included), and the row-wise kernels timed at the table's shape over `reps`
    back-to-back launches (outside the timed steps): the request (emb_lookup_request), the answer
    (emb_gather of the U requested rows) and the expansion (emb_gather through the inverse map).
    Byte models count what the call must touch: the request reads the ids and their owners and
    writes the requests and the inverse map (the sort passes are not counted); the answer reads
    and writes U rows; the expansion reads the inverse map and U rows and writes T rows."""
    V, D, P, T = sp.V, sp.D, sp.P, sp.T
    nb = len(batches)
    req = [emb.lookup_request(ids, V, tb.row_owner, P) for ids, _ in batches]
    torch.cuda.synchronize()
    Us = [int(r[3].item()) for r in req]
    assert Us == [int(u) for u in U], "the requests ask for the coalesce's distinct rows"
    ws = emb.new_workspace(emb.lookup_request_workspace_bytes(T, V))
    out = tuple(torch.empty_like(x) for x in req[0])
    ans = torch.empty((T, D), dtype=torch.float32, device="cuda")
    look = torch.empty((T, D), dtype=torch.float32, device="cuda")
    answers = [emb.gather(tb.W, r[0][:u]) for r, u in zip(req, Us)]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn):
        for i in range(3):
            fn(i)
        torch.cuda.synchronize()
        e0.record()
        for i in range(reps):
            fn(i)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / reps

    us_req = timed(lambda i: emb.lookup_request(batches[i % nb][0], V, tb.row_owner, P, out=out, workspace=ws))
    us_ans = timed(lambda i: emb.gather(tb.W, req[i % nb][0][:Us[i % nb]], out=ans[:Us[i % nb]]))
    us_exp = timed(lambda i: emb.gather(answers[i % nb], req[i % nb][4], out=look))
    Um = float(np.mean(Us))
    kern = {}
    for name, us, nbytes in (("lookup_request", us_req, T * 4 * 3 + Um * 4),
                             ("answer_gather", us_ans, 2 * Um * D * 4 + Um * 4),
                             ("expand_gather", us_exp, T * 4 + Um * D * 4 + T * D * 4)):
        kern[name] = {"avg_launch_us": us, "bytes_model": nbytes, "GBps": nbytes / (us * 1e-6) / 1e9,
                      "frac": nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS}
    return {"table": 0, "T": T, "distinct_rows": Um,
            "rowwise_MB": {"requests": Um * 4 / 1e6, "answers": Um * D * 4 / 1e6},
            "columnwise_MB": {"ids_to_owners": P * T * 4 / 1e6, "lookup_results": T * D * 4 / 1e6},
            "kernels": kern}


def exchange_report(torch, emb, sp, tb, batches, reps=10):
    """The receiver side of the gradient exchange (Sec. 4.1.1 / 4.1.2) for P simulated workers of the
    first table's shape: every worker's owner-major coalesce into its own send layout (worker w takes
    batch w mod 8 of the rotation; not timed), then the simulated AlltoAll (emb_exchange_simulated: a
    P x P block transpose of ids and rows) and every owner's merge of what it received
    (emb_receive_merge), each timed over `reps` back-to-back launches.  Byte models: the exchange reads
    and writes every sent row and id; the merge reads the received rows and ids and writes the merged
    rows and ids (its sort passes are not counted)."""
    V, D, P, T = sp.V, sp.D, sp.P, sp.T
    i32, f32 = torch.int32, torch.float32
    send_ids = torch.empty((P, T), dtype=i32, device="cuda")
    send_rows = torch.empty((P, T, D), dtype=f32, device="cuda")
    send_offs = torch.empty((P, P + 1), dtype=i32, device="cuda")
    seg = torch.empty(T + 1, dtype=i32, device="cuda")
    cnt = torch.empty(P, dtype=i32, device="cuda")
    nu = torch.empty(1, dtype=i32, device="cuda")
    ws = emb.new_workspace(emb.grad_coalesce_workspace_bytes(T, V, D))
    for w in range(P):
        ids, g = batches[w % len(batches)]
        emb.grad_coalesce_by_owner(ids, g, V, tb.row_owner, P, out=(send_ids[w], seg, send_rows[w], cnt, send_offs[w], nu),
                                   workspace=ws)
    recv = emb.exchange_simulated(send_ids, send_rows, send_offs)
    merged = emb.receive_merge(recv[0], recv[1], recv[3], V, tb.row_owner, P)
    torch.cuda.synchronize()
    R, Um = int(recv[3].item()), int(merged[5].item())
    mws = emb.new_workspace(emb.grad_coalesce_workspace_bytes(P * T, V, D))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / reps

    us_x = timed(lambda: emb.exchange_simulated(send_ids, send_rows, send_offs, out=recv))
    us_m = timed(lambda: emb.receive_merge(recv[0], recv[1], recv[3], V, tb.row_owner, P, out=merged, workspace=mws))
    kern = {}
    for name, us, nbytes in (("exchange_simulated", us_x, 2 * R * (4 * D + 4)),
                             ("receive_merge", us_m, R * (4 * D + 4) + Um * (4 * D + 4))):
        kern[name] = {"avg_call_us": us, "bytes_model": nbytes, "GBps": nbytes / (us * 1e-6) / 1e9,
                      "frac": nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS}
    del send_rows, recv, merged, mws
    return {"table": 0, "workers": P, "rows_sent": R, "rows_merged": Um,
            "merge_per_owner_mean_rows": Um / P, "calls": kern}


def cost_model_report(emb, sp, U, N=8):
    """Table 2 (Sec. 4.1.2) fed with the measured density alpha = U / V of the first table's batches,
    for N workers of one node with B = one xGMI link; the bandwidth terms (beta = 0) in microseconds
    and, separately, how many start latencies each scheme pays."""
    alpha = float(np.mean(U)) / sp.V
    M = float(sp.V) * sp.D * 4
    B = XGMI_LINK_GBPS * 1e9
    names = (("alltoall", emb.EMB_COMM_ALLTOALL, 2 * (N - 1)), ("allreduce", emb.EMB_COMM_ALLREDUCE, 2 * (N - 1)),
             ("ps_one_server_per_node", emb.EMB_COMM_PS, 2 * N), ("allgather", emb.EMB_COMM_ALLGATHER, N - 1))
    return {"N": N, "alpha": alpha, "M_bytes": M, "B_GBps": XGMI_LINK_GBPS,
            "bandwidth_term_us": {n: emb.comm_cost(c, N, M, alpha, B, 0.0, S=1) * 1e6 for n, c, _ in names},
            "start_latencies": {n: k for n, _, k in names}}


def schedule_candidates(args):
    """(cross-stream order, buffer sets) pairs the bench chooses among: those the options leave open."""
    if args.sequential:
        return [("events", 2, False)]
    orders = ("events", "signals") if args.order == "auto" else (args.order,)
    sets = (2, 4) if args.sets == 0 else (args.sets,)
    # with events the split needs two sets (its lookup waits for the delayed update two steps back)
    cands = [(o, n, False) for o in orders for n in sets
             if not (args.schedule == "split" and o == "events" and n != 2)]
    # owner-major with four sets: also with each sort stream running its steps' reductions
    if args.schedule == "by_owner":
        cands += [(o, 4, True) for o in orders if 4 in sets]
    return cands


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
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="lowdup_uniform")
    ap.add_argument("--batches", type=int, default=8)
    ap.add_argument("--time-every", type=int, default=20, help="time the update kernel on every n-th timed step")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sequential", action="store_true", help="one stream, calls one after another")
    ap.add_argument("--schedule", choices=("by_owner", "split", "unfused"), default="by_owner",
                    help="by_owner: emb_grad_coalesce_by_owner, one update; split: owner-major coalesce with "
                         "the prior/delayed split of Vertical Sparse Scheduling (emb_grad_coalesce_split; the "
                         "delayed update beside the next lookup); unfused: emb_grad_coalesce then "
                         "emb_pack_by_owner")
    ap.add_argument("--sets", type=int, choices=(0, 2, 4), default=0,
                    help="buffer sets rotated between steps, with the sorts of odd and even sets on two side "
                         "streams when 4 and not split (0: tuned; the split with events uses 2)")
    ap.add_argument("--order", choices=("auto", "signals", "events"), default="auto",
                    help="cross-stream order of the overlapped schedule: step signals (stream memory operations), "
                         "events, or auto (tuned)")
    ap.add_argument("--tune-steps", type=int, default=30)
    ap.add_argument("--summarize-trace", metavar="DIR", help="print a summary of a rocprofv3 kernel-stats run")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print the scaled HBM traffic of the update kernel from two rocprofv3 --pmc runs")
    ap.add_argument("--command", default="", help="the command recorded in a summary")
    ap.add_argument("--command2", default="", help="the second command recorded in a summary")
    args = ap.parse_args()
    if args.summarize_trace:
        tuned = len(schedule_candidates(args)) * (5 + args.tune_steps) if not args.sequential else 0
        tuned = tuned if tuned > 5 + args.tune_steps else 0
        print(summarize_trace(args.summarize_trace, args.command, tuned + args.warmup, args.steps, args.time_every),
              end="")
        return
    if args.summarize_pmc:
        print(json.dumps(summarize_pmc(*args.summarize_pmc, args.command, args.command2), indent=1))
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU's share of the path; runs on more than one GPU are not "
              "supported (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2110_09132_amd as emb
    from paper_2110_09132_amd.step import EmbeddingTable, StepPipeline
    from workloads import configs

    wl = configs.WORKLOADS[args.workload]
    log(f"workload {wl.name}: {wl.description}")
    dev = "cuda"
    tables, batches = [], []
    for sp in wl.tables:
        gdt = torch.bfloat16 if sp.grad_dtype == "bf16" else torch.float32
        W = torch.from_numpy(configs.make_weights(sp)).to(dev)
        tables.append(EmbeddingTable(W, torch.from_numpy(configs.row_owner(sp)).to(dev), sp.P, sp.T, gdt,
                                     sets=4))
        tb_batches = []
        for b in range(args.batches):
            ids, G = configs.make_batch(sp, 1000 + b)
            g = torch.from_numpy(G.view(np.int16)).to(dev).view(torch.bfloat16) if sp.grad_dtype == "bf16" \
                else torch.from_numpy(G).to(dev)
            tb_batches.append((torch.from_numpy(ids).to(dev), g))
        batches.append(tb_batches)
    step_batches = [[batches[k][b] for k in range(len(tables))] for b in range(args.batches)]

    # unique and prior row counts of each batch (the next batch is the next one in rotation),
    # outside any timed region
    U = [[0] * len(tables) for _ in range(args.batches)]
    U_prior = [[0] * len(tables) for _ in range(args.batches)]
    owner_rows = [None] * args.batches  # rows per owner of the first table (prior + delayed)
    for b in range(args.batches):
        for k, tb in enumerate(tables):
            ids, g = step_batches[b][k]
            nxt = step_batches[(b + 1) % args.batches][k][0]
            out = emb.grad_coalesce_split(ids, nxt, g, tb.V, tb.row_owner, tb.P, workspace=tb.ws_coalesce)
            torch.cuda.synchronize()
            U[b][k] = int(out[5].item())
            U_prior[b][k] = int(out[4][tb.P].item())
            if k == 0:
                owner_rows[b] = out[3].view(2, tb.P).sum(0).cpu().numpy()

    split = args.schedule == "split"
    by_owner = args.schedule != "unfused"
    def make_pipe(cand):
        order, sets, paired = cand
        return StepPipeline(tables, wl.lr, wl.beta1, wl.beta2, wl.eps, overlap=not args.sequential,
                            by_owner=by_owner, split=split, signals=order == "signals",
                            sort_streams=2 if (sets == 4 and by_owner and not split) else 1, sets=sets,
                            paired=paired)

    def next_ids(t):
        return [x[0] for x in step_batches[(t + 1) % args.batches]] if split else None

    t = 0
    # the schedule: time a few untimed steps of each candidate (cross-stream order x buffer sets)
    # and keep the fastest.  Events cost the GPU nothing but the host ~85 us per overlapped step;
    # step signals halve the host's cost but add small runtime kernels to the streams.  Four sets
    # (sorts on two streams) free the sorts of latency-bound steps; two interfere less with the
    # bandwidth-bound ones.
    tune_ms = {}
    cands = schedule_candidates(args)
    cand = cands[0]
    if len(cands) > 1:
        for c in cands:
            trial = make_pipe(c)
            for k in range(5 + args.tune_steps):
                if k == 5:
                    trial.finish()
                    torch.cuda.synchronize()
                    t_start = time.perf_counter()
                t += 1
                trial.step(step_batches[t % args.batches], t, next_ids=next_ids(t))
            trial.finish()
            torch.cuda.synchronize()
            tune_ms[f"{c[0]}/{c[1]} sets{'/paired' if c[2] else ''}"] = \
                (time.perf_counter() - t_start) * 1e3 / args.tune_steps
            del trial
        cand = cands[min(range(len(cands)), key=lambda i: list(tune_ms.values())[i])]
    order, nsets, paired = cand
    log(f"schedule: {order}, {nsets} buffer sets{', paired' if paired else ''} {tune_ms or ''}")
    pipe = make_pipe(cand)
    for _ in range(args.warmup):
        t += 1
        pipe.step(step_batches[t % args.batches], t, next_ids=next_ids(t))
    pipe.finish()
    torch.cuda.synchronize()

    # timed region: exactly K steps; the update's duration is recorded on its own stream
    main = torch.cuda.current_stream()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # the update's own duration, on its stream, on every time_every-th step (an event pair
    # costs the stream a few microseconds of idle time)
    timed = [s for s in range(args.steps) if s % args.time_every == 0]
    adam_ev = {s: (emb.Event(timing=True), emb.Event(timing=True)) for s in timed}
    rows, used = 0, []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(main)
    for s in range(args.steps):
        t += 1
        b = t % args.batches
        pipe.step(step_batches[b], t, timing={"adam": adam_ev[s]} if s in adam_ev else None, next_ids=next_ids(t))
        rows += sum(U[b])
        used.append(b)
    pipe.finish()
    end.record(main)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = start.elapsed_time(end)
    log(f"timed {args.steps} steps: {ms_total / args.steps:.4f} ms/step")
    ms_step = ms_total / args.steps
    adam_us = 1e3 * sum(a.elapsed_ms(z) for a, z in adam_ev.values()) / len(adam_ev)

    # per-stage breakdown: the same steps run one call after another on one stream (with the
    # split, the "pack" pair of timing events times the prior update, "adam" the delayed one)
    seq = StepPipeline(tables, wl.lr, wl.beta1, wl.beta2, wl.eps, overlap=False, by_owner=by_owner, split=split)
    stage_ms = {k: 0.0 for k in (("gather", "coalesce", "pack", "adam") if split or not by_owner
                                 else ("gather", "coalesce", "adam"))}
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    seq_total = 0.0
    for s in range(args.steps):
        t += 1
        ev = {k: (emb.Event(timing=True), emb.Event(timing=True)) for k in stage_ms}
        s0.record(main)
        seq.step(step_batches[t % args.batches], t, timing=ev, next_ids=next_ids(t))
        s1.record(main)
        torch.cuda.synchronize()
        seq_total += s0.elapsed_time(s1) / args.steps
        for k in stage_ms:
            stage_ms[k] += ev[k][0].elapsed_ms(ev[k][1]) / args.steps

    if split:  # name the timing pairs for what they time under the split
        stage_ms = {"gather": stage_ms["gather"], "coalesce": stage_ms["coalesce"],
                    "update_prior": stage_ms["pack"], "update_delayed": stage_ms["adam"]}

    log("per-stage breakdown done; copy reference, column partition, cost model ...")
    copy_gbps = copy_reference(torch)
    column = column_partition_report(torch, emb, wl.tables[0], tables[0], [x[0] for x in step_batches],
                                     [U[b][0] for b in range(args.batches)], owner_rows)
    cost = cost_model_report(emb, wl.tables[0], [U[b][0] for b in range(args.batches)])
    forward = forward_exchange_report(torch, emb, wl.tables[0], tables[0], [x[0] for x in step_batches],
                                      [U[b][0] for b in range(args.batches)])
    exchange = exchange_report(torch, emb, wl.tables[0], tables[0], [x[0] for x in step_batches])

    # algorithmic bytes of the timed steps
    bytes_step = {k: 0.0 for k in ("gather", "coalesce", "pack", "adam")}
    for b in used:
        for k, tb in enumerate(tables):
            sp = wl.tables[k]
            bm = byte_model(sp.T, U[b][k], sp.D, 2 if sp.grad_dtype == "bf16" else 4, sp.P, by_owner,
                            sp.T if split else 0)
            for name in bytes_step:
                bytes_step[name] += bm[name] / args.steps
    total_bytes = sum(bytes_step.values())
    step_gbps = total_bytes / (ms_step * 1e-3) / 1e9
    # the roofline kernel: the update launch of the first table (with the split, its delayed part,
    # the larger one), every time_every-th step
    sp0 = wl.tables[0]
    upd_rows = [U[used[s]][0] - (U_prior[used[s]][0] if split else 0) for s in timed]
    adam_bytes = sum(byte_model(sp0.T, r, sp0.D, 4, sp0.P)["adam"] for r in upd_rows) / len(timed)
    adam_gbps = adam_bytes / (adam_us * 1e-6) / 1e9
    # sizes of the sparse gradient as Table 3 reports them (per step, all tables): the per-token
    # COO gradient (original), after COALESCE (coalesced), and the prior part of the vertical split
    # (prioritized: rows whose id is in the next batch, the part that must arrive before the next
    # forward pass); ids int32, rows in the gradient's element type
    def mb(rows, sp):
        return rows * (4 + sp.D * (2 if sp.grad_dtype == "bf16" else 4)) / 1e6
    orig = sum(mb(sp.T, sp) for sp in wl.tables)
    coal = sum(mb(U[b][k], wl.tables[k]) for b in range(args.batches) for k in range(len(tables))) / args.batches
    prio = sum(mb(U_prior[b][k], wl.tables[k]) for b in range(args.batches) for k in range(len(tables))) / args.batches
    table3 = {"original_MB": orig, "coalesced_MB": coal, "prioritized_MB": prio,
              "reduction_by_coalescing": 1 - coal / orig, "further_reduction_by_prioritizing": 1 - prio / coal,
              "next_batch": "the next batch of the rotation"}
    prior_frac = sum(U_prior[b][k] for b in used for k in range(len(tables))) / max(1, sum(
        U[b][k] for b in used for k in range(len(tables))))

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
        "dtype": "bf16-in/f32" if any(sp.grad_dtype == "bf16" for sp in wl.tables) else "f32",
        "data": "synthetic (seeded ids and N(0,sigma) gradients, random-init table)",
        "config": {"workload": wl.name,
                   "tables": [dict(V=sp.V, D=sp.D, T=sp.T, P=sp.P, ids=sp.id_law, owner=sp.owner_rule)
                              for sp in wl.tables],
                   "mean_unique_rows_per_step": rows / args.steps, "batches_rotated": args.batches,
                   "coalesce": {"split": "emb_grad_coalesce_split (owner-major, prior/delayed split)",
                                "by_owner": "emb_grad_coalesce_by_owner (coalesce straight into the send layout)",
                                "unfused": "emb_grad_coalesce + emb_pack_by_owner"}[args.schedule],
                   "schedule": "one stream" if args.sequential else
                   {"split": "sort, reduction and delayed update on three side streams; lookup and prior "
                             "update on the main stream",
                    "by_owner": "sort and reduction on two side streams; lookup and update on the main stream",
                    "unfused": "coalesce and pack on two side streams; lookup and update on the main stream"}[
                       args.schedule],
                   "sort_streams": None if (args.sequential or split or not by_owner) else (2 if nsets == 4 else 1),
                   "buffer_sets": nsets,
                   "sort_and_reduce_paired": paired,
                   "cross_stream_order": None if args.sequential else
                   {"signals": "step signals (hipStreamWriteValue32 / hipStreamWaitValue32)",
                    "events": "events (hipEventRecord / hipStreamWaitEvent)"}[order],
                   "schedule_tuning_ms_per_step": tune_ms or None,
                   "prior_rows_frac": prior_frac if split else None},
        "step_bytes_model": total_bytes,
        "step_bytes_model_kind": "fused minimum (pack folded into coalesce)" if by_owner else "four calls",
        "stage_bytes_model": bytes_step,
        "step_hbm_GBps": step_gbps,
        "step_hbm_frac": step_gbps / HBM_PEAK_GBPS,
        "sequential_ms_per_step": seq_total,
        "stage_ms_sequential": stage_ms,
        "wall_s_timed": wall,
        "roofline": {"bound": "hbm",
                     "kernel": "adam_kernel (emb_sparse_adam_apply)" + (", delayed rows" if split else ""),
                     "achieved": adam_gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": adam_gbps / HBM_PEAK_GBPS,
                     "traffic": measured_traffic() if args.workload == "lowdup_uniform" else None,
                     "bytes_per_launch": adam_bytes, "avg_launch_us": adam_us,
                     "launches_timed": len(adam_ev)},
        "copy_GBps": copy_gbps,
        "gradient_sizes_table3": table3,
        "column_partition": column,
        "forward_exchange": forward,
        "gradient_exchange": exchange,
        "comm_cost_model": cost,
        "step_frac_of_copy": step_gbps / copy_gbps,
        "host": host_info(),
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle ...")
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
