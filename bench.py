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
import math
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E
TUNE_FINALISTS = 3  # schedule candidates timed a second time
TUNE_TRIAL_MS = 15.0  # the shortest trial of a schedule candidate


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


def summarize_trace(directory, command, skip=20, steps=200, every=20, tables=1):
    """Text summary of a rocprofv3 --kernel-trace --stats run (kernel_stats.csv), plus the
    average duration of the first table's update kernel over the steps of the bench run's roofline
    window (steps skip+1 .. skip+steps in launch order, one update dispatch per table each, from
    kernel_trace.csv; skip counts the steps before them: the order tuning, the warm-up and the
    timed steps), every `every`-th of which the bench times with events."""
    trace = [r for r in _read_csv(_find(directory, "kernel_trace.csv")) if ADAM_KERNEL in r["Kernel_Name"]]
    trace.sort(key=lambda r: int(r["Start_Timestamp"]))
    durs = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            for r in trace[skip * tables:(skip + steps) * tables:tables]]
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
                    f"{every}th step of the roofline window): avg {sum(sampled) / len(sampled):.2f} us",
                f"{ADAM_KERNEL} over the {len(durs)} steps of the roofline window (dispatches {skip + 1}.."
                    f"{skip + len(durs)}): avg {sum(durs) / len(durs):.2f} us, min {min(durs):.2f} us, "
                    f"max {max(durs):.2f} us"]
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


def summarize_traffic(fetch_dir, write_dir, bench_json, command_fetch, command_write):
    """HBM traffic per kernel from two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE in KiB per dispatch,
    averaged over each kernel's dispatches), each scaled by what the counter reads for the reference
    stream of the same run (torch.bitwise_not over COPY_MIB MiB: reads and writes that many bytes);
    beside the algorithmic bytes of the lookup, the reduction and the update for the run's mean
    distinct-row count (from its bench line, `bench_json`)."""
    def per_kernel(directory, counter):
        vals = {}
        for r in _read_csv(_find(directory, "counter_collection.csv")):
            if r.get("Counter_Name") != counter:
                continue
            name = r["Kernel_Name"].replace("(anonymous namespace)::", "").split("(")[0]
            name = name.replace("void ", "").replace("emb::", "")
            vals.setdefault(name, []).append(float(r["Counter_Value"]))
        return {k: sum(v) / len(v) for k, v in vals.items()}, {k: len(v) for k, v in vals.items()}
    f, nf = per_kernel(fetch_dir, "FETCH_SIZE")
    w, _ = per_kernel(write_dir, "WRITE_SIZE")
    copy = next(k for k in f if COPY_KERNEL in k)
    copy_bytes = COPY_MIB * (1 << 20)
    fs, ws = copy_bytes / (f[copy] * 1024.0), copy_bytes / (w[copy] * 1024.0)
    with open(bench_json) as fh:
        b = json.loads(fh.read().strip().splitlines()[-1])
    t = b["config"]["tables"][0]
    T, D, U = t["T"], t["D"], b["config"]["mean_unique_rows_per_step"]
    model = {"adam_kernel": (4 * U + 16 * D * U, 12 * D * U), "gather_kernel": (4 * T + 4 * D * U, 4 * D * T),
             "seg_reduce_kernel": (8 * T + 4 * D * T, 8 * U + 4 * D * U + 4)}  # sorted keys and positions in
    out = [f"command_fetch: {command_fetch}", f"command_write: {command_write}",
           f"scales (reference stream of {COPY_MIB} MiB each way): FETCH x{fs:.4f}, WRITE x{ws:.4f}; "
           f"mean distinct rows U = {U:.0f} of T = {T}, D = {D}", "",
           f"{'kernel':56s} {'disp':>5s} {'read MB':>9s} {'write MB':>9s} {'model r/w MB':>15s} {'ratio':>6s}"]
    for k in sorted(f, key=lambda k: -f[k] * nf[k]):
        if k == copy or k not in w:
            continue
        rd, wr = f[k] * 1024.0 * fs / 1e6, w[k] * 1024.0 * ws / 1e6
        m = next((v for key, v in model.items() if key in k), None)
        ms = f"{m[0] / 1e6:7.1f}/{m[1] / 1e6:7.1f}" if m else ""
        ratio = f"{(rd + wr) * 1e6 / (m[0] + m[1]):6.3f}" if m else ""
        out.append(f"{k[:56]:56s} {nf[k]:5d} {rd:9.1f} {wr:9.1f} {ms:>15s} {ratio:>6s}")
    return "\n".join(out) + "\n"

CU_NUM = 256  # MI355X compute units


def summarize_counters(dirs, command):
    """Per-kernel figures from rocprofv3 --pmc runs (counter_collection.csv of each directory; a kernel's
    counters averaged over its dispatches, which the profiler runs one at a time).  The derived figures
    follow the profiler's own definitions for gfx950 (CU_NUM = 256):
      occupancy  mean resident waves per CU: 4 SQ_WAVE_CYCLES / (GRBM_GUI_ACTIVE CU_NUM), of 32
      VALU busy  100 SQ_ACTIVE_INST_VALU / (CU_NUM GRBM_GUI_ACTIVE)
      LDS util   100 SQ_LDS_IDX_ACTIVE / (GRBM_GUI_ACTIVE CU_NUM)
      LDS bank conflict  100 SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE (conflict cycles per LDS-active cycle)
      L2 hit     100 TCC_HIT / (TCC_HIT + TCC_MISS)
    plus VALU and LDS instructions per wave and the mean duration of a dispatch under the profiler."""
    per = {}  # kernel -> counter -> [values]
    durs = {}
    for d in dirs:
        for r in _read_csv(_find(d, "counter_collection.csv")):
            name = r["Kernel_Name"].replace("(anonymous namespace)::", "").split("(")[0]
            name = name.replace("void ", "").replace("emb::", "")[:60]
            per.setdefault(name, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
            durs.setdefault(name, {})[(d, r["Dispatch_Id"])] = \
                (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3

    def mean(k, c):
        v = per[k].get(c)
        return sum(v) / len(v) if v else None

    def ratio(a, b, scale=1.0):
        return None if a is None or not b else scale * a / b

    def fmt(x, w=8, p=1):
        return f"{'-':>{w}s}" if x is None else f"{x:{w}.{p}f}"

    rows = []
    for k in per:
        gui = mean(k, "GRBM_GUI_ACTIVE")
        waves = mean(k, "SQ_WAVES")
        hit, miss = mean(k, "TCC_HIT_sum"), mean(k, "TCC_MISS_sum")
        per_dir = max(sum(1 for key in durs[k] if key[0] == d) for d in dirs)  # dispatches of one run
        rows.append((k, per_dir, sum(durs[k].values()) / len(durs[k]), waves,
                     ratio(mean(k, "SQ_WAVE_CYCLES"), None if gui is None else gui * CU_NUM, 4.0),
                     ratio(mean(k, "SQ_ACTIVE_INST_VALU"), None if gui is None else gui * CU_NUM, 100.0),
                     ratio(mean(k, "SQ_LDS_IDX_ACTIVE"), None if gui is None else gui * CU_NUM, 100.0),
                     ratio(mean(k, "SQ_LDS_BANK_CONFLICT"), mean(k, "SQ_LDS_IDX_ACTIVE"), 100.0),
                     ratio(hit, None if hit is None or miss is None else hit + miss, 100.0),
                     ratio(mean(k, "SQ_INSTS_VALU"), waves), ratio(mean(k, "SQ_INSTS_LDS"), waves)))
    rows.sort(key=lambda r: -r[1] * r[2])
    out = [f"command: {command}", "",
           f"{'kernel':60s} {'disp':>5s} {'us':>8s} {'waves':>8s} {'occ/CU':>7s} {'VALU%':>6s} {'LDS%':>6s} "
           f"{'bankc%':>6s} {'L2hit%':>6s} {'VALUi/w':>8s} {'LDSi/w':>7s}"]
    for k, n, us, waves, occ, valu, lds, bank, l2, vi, li in rows:
        out.append(f"{k:60s} {n:5d} {us:8.2f} {fmt(waves, 8, 0)} {fmt(occ, 7, 2)} {fmt(valu, 6)} {fmt(lds, 6)} "
                   f"{fmt(bank, 6)} {fmt(l2, 6)} {fmt(vi, 8)} {fmt(li, 7)}")
    return "\n".join(out) + "\n"


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
    """(cross-stream order, buffer sets, paired) triples the bench chooses among: those the options leave
    open (--candidate names one)."""
    if args.sequential:
        return [("events", 2, False)]
    if args.candidate:
        parts = args.candidate.split("/")
        if parts[0] not in ("events", "signals", "queued") or len(parts) not in (2, 3):
            raise SystemExit(f"--candidate {args.candidate!r}: expected ORDER/SETS[/paired], ORDER events, signals "
                             f"or queued")
        return [(parts[0], int(parts[1]), len(parts) > 2 and parts[2] == "paired")]
    orders = ("events", "signals") if args.order == "auto" else (args.order,)
    if args.order == "queued" and args.schedule != "by_owner":
        raise SystemExit("--order queued takes the owner-major schedule")
    sets = (2, 4, 6) if args.sets == 0 else (args.sets,)
    # with events the split needs two sets (its lookup waits for the delayed update two steps back)
    cands = [(o, n, False) for o in orders for n in sets
             if n != 6 and not (args.schedule == "split" and o == "events" and n != 2)]
    # owner-major with four sets: also with each sort stream running its steps' reductions; with six,
    # three such streams; and, tuned, those two with the two-thread enqueue
    if args.schedule == "by_owner":
        cands += [(o, 4, True) for o in orders if 4 in sets]
        cands += [(o, 6, True) for o in orders if 6 in sets]
        if args.order == "auto":
            cands += [("queued", n, True) for n in (4, 6) if n in sets]
    return cands


def cand_name(c):
    return f"{c[0]}/{c[1]} sets{'/paired' if c[2] else ''}"


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


def spread(xs):
    """Median, 10th and 90th percentile of a list of times."""
    a = np.asarray(xs, dtype=np.float64)
    return {"median": float(np.median(a)), "p10": float(np.percentile(a, 10)),
            "p90": float(np.percentile(a, 90)), "n": int(a.size)}


FLUSH_BYTES = 1 << 30  # written between the steps of the cold runs: four times the 256 MB last-level cache


class WorkloadRun:
    """One workload resident on the GPU: its tables (W, Adam moments, four buffer sets), `nbatches`
    pre-generated batches of every table, and each batch's distinct and prior row counts (taken with
    the library before any timing; the next batch of the split is the next one in the rotation)."""

    def __init__(self, torch, emb, wl, nbatches, schedule):
        from paper_2110_09132_amd.step import EmbeddingTable
        from workloads import configs
        self.torch, self.emb, self.wl = torch, emb, wl
        self.nb = nbatches
        self.split = schedule == "split"
        self.by_owner = schedule != "unfused"
        self.schedule = schedule
        self.t = 0  # Adam step counter, advanced by every step enqueued on the tables
        dev = "cuda"
        self.tables, batches = [], []
        for sp in wl.tables:
            gdt = torch.bfloat16 if sp.grad_dtype == "bf16" else torch.float32
            W = torch.from_numpy(configs.make_weights(sp)).to(dev)
            self.tables.append(EmbeddingTable(W, torch.from_numpy(configs.row_owner(sp)).to(dev), sp.P, sp.T, gdt,
                                              sets=6))
            tb_batches = []
            for b in range(nbatches):
                ids, G = configs.make_batch(sp, 1000 + b)
                g = torch.from_numpy(G.view(np.int16)).to(dev).view(torch.bfloat16) if sp.grad_dtype == "bf16" \
                    else torch.from_numpy(G).to(dev)
                tb_batches.append((torch.from_numpy(ids).to(dev), g))
            batches.append(tb_batches)
        self.step_batches = [[batches[k][b] for k in range(len(self.tables))] for b in range(nbatches)]
        nt = len(self.tables)
        self.U = [[0] * nt for _ in range(nbatches)]
        self.U_prior = [[0] * nt for _ in range(nbatches)]
        self.owner_rows = [None] * nbatches  # rows per owner of the first table (prior + delayed)
        for b in range(nbatches):
            for k, tb in enumerate(self.tables):
                ids, g = self.step_batches[b][k]
                nxt = self.step_batches[(b + 1) % nbatches][k][0]
                out = emb.grad_coalesce_split(ids, nxt, g, tb.V, tb.row_owner, tb.P, workspace=tb.ws_coalesce)
                torch.cuda.synchronize()
                self.U[b][k] = int(out[5].item())
                self.U_prior[b][k] = int(out[4][tb.P].item())
                if k == 0:
                    self.owner_rows[b] = out[3].view(2, tb.P).sum(0).cpu().numpy()

    def make_pipe(self, cand, sequential=False):
        from paper_2110_09132_amd.step import StepPipeline
        wl = self.wl
        if sequential:
            return StepPipeline(self.tables, wl.lr, wl.beta1, wl.beta2, wl.eps, overlap=False,
                                by_owner=self.by_owner, split=self.split)
        order, sets, paired = cand
        return StepPipeline(self.tables, wl.lr, wl.beta1, wl.beta2, wl.eps, overlap=True, by_owner=self.by_owner,
                            split=self.split, signals=order == "signals", queued=order == "queued",
                            sort_streams=(sets // 2 if sets in (4, 6) else 1) if (self.by_owner and not self.split)
                            else 1, sets=sets, paired=paired)

    def next_ids(self, t):
        return [x[0] for x in self.step_batches[(t + 1) % self.nb]] if self.split else None

    def step(self, pipe, timing=None):
        """Enqueue the next step; returns the index of the batch it used."""
        self.t += 1
        b = self.t % self.nb
        pipe.step(self.step_batches[b], self.t, timing=timing, next_ids=self.next_ids(self.t))
        return b

    def settle(self, pipe):
        pipe.finish()
        self.torch.cuda.synchronize()

    def tune(self, cands, tune_steps):
        """Time `tune_steps` untimed steps of each candidate schedule (after 5 more), then the
        TUNE_FINALISTS fastest once more in reverse order, and keep the candidate with the smallest of
        its times (a single trial of a few milliseconds is at the mercy of host jitter).  Events cost
        the GPU nothing but the host tens of microseconds per overlapped step; step signals halve the
        host's cost but add small runtime kernels to the streams.  Four sets (sorts on two streams)
        free the sorts of latency-bound steps; two interfere less with the bandwidth-bound ones."""
        tune_ms = {}
        if len(cands) == 1:
            return cands[0], tune_ms

        def trial_ms(c, n):
            trial = self.make_pipe(c)
            for k in range(5 + n):
                if k == 5:
                    self.settle(trial)
                    t_start = time.perf_counter()
                self.step(trial)
            self.settle(trial)
            ms = (time.perf_counter() - t_start) * 1e3 / n
            del trial
            return ms

        # each trial runs for at least TUNE_TRIAL_MS, so that host jitter does not pick the schedule
        # of a short-stepped workload (a 30-step trial of 50 us steps lasts 1.5 ms)
        tune_steps = max(tune_steps, math.ceil(TUNE_TRIAL_MS / trial_ms(cands[0], tune_steps)))
        for c in cands:
            tune_ms[cand_name(c)] = trial_ms(c, tune_steps)
        order = sorted(range(len(cands)), key=lambda i: tune_ms[cand_name(cands[i])])
        for i in reversed(order[:TUNE_FINALISTS]):
            name = cand_name(cands[i])
            tune_ms[name] = min(tune_ms[name], trial_ms(cands[i], tune_steps))
        best = min(range(len(cands)), key=lambda i: tune_ms[cand_name(cands[i])])
        return cands[best], tune_ms

    def timed(self, pipe, K, time_every):
        """Exactly K steps between two synchronisations, timed with events on the main stream; the update
        kernel of the first table is timed on its own stream (a pair of events attached to its dispatch)
        on every time_every-th step (0: on none; each pair costs the step about 9 us)."""
        torch, emb = self.torch, self.emb
        main = torch.cuda.current_stream()
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        timed_steps = [s for s in range(K) if time_every > 0 and s % time_every == 0]
        adam_ev = {s: (emb.Event(timing=True), emb.Event(timing=True)) for s in timed_steps}
        used = []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        start.record(main)
        for s in range(K):
            used.append(self.step(pipe, timing={"adam": adam_ev[s]} if s in adam_ev else None))
        host_enqueue = time.perf_counter() - t0
        pipe.finish()
        end.record(main)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms_total = start.elapsed_time(end)
        adam_us = [1e3 * adam_ev[s][0].elapsed_ms(adam_ev[s][1]) for s in timed_steps]
        rows = sum(sum(self.U[b]) for b in used)
        return dict(ms_total=ms_total, wall=wall, used=used, rows=rows, adam_us=adam_us,
                    adam_steps=timed_steps, host_enqueue_ms=host_enqueue * 1e3)

    def sequential(self, n, cold, per_call):
        """n steps one after another on one stream, an event pair around each step, and with per_call
        around each call as well (their records sit between the calls and lengthen the step, so the
        step's own spread comes from a run without them).  cold: a 1 GiB buffer is written between the
        steps, outside the events, so that each step starts with the caches (L2 and the last-level
        cache) holding none of its data."""
        torch, emb = self.torch, self.emb
        main = torch.cuda.current_stream()
        stages = ("gather", "coalesce", "pack", "adam") if (self.split or not self.by_owner) else \
            ("gather", "coalesce", "adam")
        seq = self.make_pipe(None, sequential=True)
        flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.int32, device="cuda") if cold else None
        evs = []
        for s in range(n):
            if flush is not None:
                flush.fill_(s)
            ev = {k: (emb.Event(timing=True), emb.Event(timing=True)) for k in stages} if per_call else None
            s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s0.record(main)
            b = self.step(seq, timing=ev)
            s1.record(main)
            evs.append((b, s0, s1, ev))
            if s % 25 == 24:  # bounded numbers of live events
                torch.cuda.synchronize()
        torch.cuda.synchronize()
        step_ms = [s0.elapsed_time(s1) for _, s0, s1, _ in evs]
        stage_ms = {k: [ev[k][0].elapsed_ms(ev[k][1]) for _, _, _, ev in evs] for k in stages} if per_call else {}
        if self.split and per_call:  # the timing pairs' names under the split
            stage_ms = {"gather": stage_ms["gather"], "coalesce": stage_ms["coalesce"],
                        "update_prior": stage_ms["pack"], "update_delayed": stage_ms["adam"]}
        used = [b for b, _, _, _ in evs]
        del flush
        return dict(step_ms=step_ms, stage_ms=stage_ms, used=used)

    def step_bytes(self, used):
        """Mean algorithmic bytes per step (per stage) over the batches `used`."""
        out = {k: 0.0 for k in ("gather", "coalesce", "pack", "adam")}
        for b in used:
            for k, tb in enumerate(self.tables):
                sp = self.wl.tables[k]
                bm = byte_model(sp.T, self.U[b][k], sp.D, 2 if sp.grad_dtype == "bf16" else 4, sp.P, self.by_owner,
                                sp.T if self.split else 0)
                for name in out:
                    out[name] += bm[name] / len(used)
        return out

    def update_bytes(self, b):
        """Algorithmic bytes of the first table's update launch of batch b (with the split: the delayed part)."""
        sp0 = self.wl.tables[0]
        rows = self.U[b][0] - (self.U_prior[b][0] if self.split else 0)
        return byte_model(sp0.T, rows, sp0.D, 4, sp0.P)["adam"]

    def release(self):
        del self.tables, self.step_batches
        self.torch.cuda.synchronize()
        self.torch.cuda.empty_cache()


def sequential_report(run, n):
    """Warm and cold figures of the step run call after call on one stream (median, p10, p90 over n
    steps): the step (event pairs around the steps only), each call (a second run with event pairs
    around the calls too), and the step's effective bandwidth at the median."""
    out = {}
    for kind, cold in (("warm", False), ("cold", True)):
        r = run.sequential(n, cold, per_call=False)
        c = run.sequential(n, cold, per_call=True)
        nbytes = sum(run.step_bytes(r["used"]).values())
        st = spread(r["step_ms"])
        out[kind] = {"step_ms": st, "stage_ms": {k: spread(v) for k, v in c["stage_ms"].items()},
                     "step_ms_with_call_events": spread(c["step_ms"]),
                     "step_hbm_frac_at_median": nbytes / (st["median"] * 1e-3) / 1e9 / HBM_PEAK_GBPS}
    out["flush_bytes_cold"] = FLUSH_BYTES
    return out


def pipelined_report(run, args, K):
    """Tune the schedule, warm up, then exactly K timed steps (no event pairs among them); then the
    roofline window: --roofline-steps more steps of the same schedule, the update kernel timed with
    events attached to its dispatch on every --roofline-every-th of them.  The step figures and the
    update kernel's live duration.  With --sequential: one stream, calls one after another."""
    cands = schedule_candidates(args)
    cand, tune_ms = run.tune(cands, args.tune_steps)
    pipe = run.make_pipe(cand, sequential=args.sequential)
    for _ in range(args.warmup):
        run.step(pipe)
    run.settle(pipe)
    r = run.timed(pipe, K, 0)
    steps_before_window = run.t  # every step enqueued so far on this workload: tuning, warm-up, timed
    w = run.timed(pipe, args.roofline_steps, args.roofline_every)
    ms_step = r["ms_total"] / K
    bytes_step = run.step_bytes(r["used"])
    total = sum(bytes_step.values())
    adam_us = float(np.mean(w["adam_us"]))
    adam_bytes = float(np.mean([run.update_bytes(w["used"][s]) for s in w["adam_steps"]]))
    del pipe
    return dict(cand=cand, tune_ms=tune_ms, ms_step=ms_step, ms_total=r["ms_total"], wall=r["wall"],
                rows=r["rows"], used=r["used"], bytes_step=bytes_step, total_bytes=total,
                step_gbps=total / (ms_step * 1e-3) / 1e9, adam_us=adam_us, adam_us_all=w["adam_us"],
                adam_bytes=adam_bytes, adam_gbps=adam_bytes / (adam_us * 1e-6) / 1e9,
                window_ms_step=w["ms_total"] / args.roofline_steps, host_enqueue_ms=r["host_enqueue_ms"],
                steps_before_window=steps_before_window)


def config_report(torch, emb, name, args, K, run=None, pl=None):
    """One workload's entry of the `configs` object: pipelined steps (tuned schedule), the update
    kernel's live duration, and the sequential warm and cold spreads."""
    from workloads import configs
    wl = configs.WORKLOADS[name]
    own = run is None
    if own:
        log(f"config {name}: {wl.description}")
        run = WorkloadRun(torch, emb, wl, args.batches, args.schedule)
        pl = pipelined_report(run, args, K)
    seqr = sequential_report(run, args.seq_steps)
    entry = {
        "tables": [dict(V=sp.V, D=sp.D, T=sp.T, P=sp.P, ids=sp.id_law + (f" s={sp.zipf_s}" if sp.id_law == "zipf"
                                                                          else ""), owner=sp.owner_rule,
                        grad=sp.grad_dtype) for sp in wl.tables],
        "schedule": cand_name(pl["cand"]), "timed_steps": K,
        "ms_per_step": pl["ms_step"], "unique_rows_per_s": pl["rows"] / (pl["ms_total"] * 1e-3),
        "mean_unique_rows_per_step": pl["rows"] / K,
        "step_bytes_model": pl["total_bytes"], "step_hbm_GBps": pl["step_gbps"],
        "step_hbm_frac": pl["step_gbps"] / HBM_PEAK_GBPS,
        "update_kernel": {"avg_launch_us": pl["adam_us"], "launches_timed": len(pl["adam_us_all"]),
                          "bytes_per_launch": pl["adam_bytes"], "GBps": pl["adam_gbps"],
                          "frac": pl["adam_gbps"] / HBM_PEAK_GBPS},
        "sequential": seqr,
    }
    if own:
        run.release()
    return entry


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="lowdup_uniform")
    ap.add_argument("--batches", type=int, default=8)
    ap.add_argument("--roofline-steps", type=int, default=200,
                    help="steps of the roofline window that follows the timed steps")
    ap.add_argument("--roofline-every", type=int, default=10,
                    help="time the update kernel on every n-th step of the roofline window")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sequential", action="store_true", help="one stream, calls one after another")
    ap.add_argument("--schedule", choices=("by_owner", "split", "unfused"), default="by_owner",
                    help="by_owner: emb_grad_coalesce_by_owner, one update; split: owner-major coalesce with "
                         "the prior/delayed split of Vertical Sparse Scheduling (emb_grad_coalesce_split; the "
                         "delayed update beside the next lookup); unfused: emb_grad_coalesce then "
                         "emb_pack_by_owner")
    ap.add_argument("--sets", type=int, choices=(0, 2, 4, 6), default=0,
                    help="buffer sets rotated between steps, with the sorts of odd and even sets on two side "
                         "streams when 4 and not split (0: tuned; the split with events uses 2)")
    ap.add_argument("--order", choices=("auto", "signals", "events", "queued"), default="auto",
                    help="cross-stream order of the overlapped schedule: step signals (stream memory operations), "
                         "events, events with the two-thread enqueue (queued; owner-major), or auto (tuned)")
    ap.add_argument("--candidate", default="",
                    help="one schedule, ORDER/SETS[/paired] (e.g. events/4/paired): no tuning")
    ap.add_argument("--tune-steps", type=int, default=30)
    ap.add_argument("--seq-steps", type=int, default=100,
                    help="steps of each sequential (warm, cold) run of the timing protocol")
    ap.add_argument("--config-steps", type=int, default=100,
                    help="timed steps of each workload of the `configs` object (at least --steps)")
    ap.add_argument("--only-steps", action="store_true",
                    help="tuning, warm-up and the timed steps only (for profiler runs)")
    ap.add_argument("--no-configs", action="store_true", help="leave out the `configs` object")
    ap.add_argument("--summarize-trace", metavar="DIR", help="print a summary of a rocprofv3 kernel-stats run")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print the scaled HBM traffic of the update kernel from two rocprofv3 --pmc runs")
    ap.add_argument("--summarize-traffic", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "BENCH_JSON"),
                    help="print the scaled HBM traffic of every kernel from two rocprofv3 --pmc runs")
    ap.add_argument("--summarize-counters", nargs="+", metavar="DIR",
                    help="print per-kernel occupancy, VALU, LDS and L2 figures from rocprofv3 --pmc runs")
    ap.add_argument("--bench-line", metavar="JSON", default="",
                    help="with --summarize-trace: the traced run's bench line, for the number of steps before "
                         "its roofline window (else counted from the options, with trials of --tune-steps)")
    ap.add_argument("--command", default="", help="the command recorded in a summary")
    ap.add_argument("--command2", default="", help="the second command recorded in a summary")
    args = ap.parse_args()
    if args.summarize_trace:
        from workloads import configs
        tables = len(configs.WORKLOADS[args.workload].tables)
        if args.bench_line:  # the traced run's own count of the steps before its roofline window
            with open(args.bench_line) as f:
                skip = json.loads(f.read().strip().splitlines()[-1])["roofline"]["steps_before_window"]
        else:
            n = len(schedule_candidates(args))
            tuned = (n + 1 + min(n, TUNE_FINALISTS)) * (5 + args.tune_steps) if n > 1 else 0
            skip = tuned + args.warmup + args.steps
        print(summarize_trace(args.summarize_trace, args.command, skip, args.roofline_steps, args.roofline_every,
                              tables), end="")
        return
    if args.summarize_pmc:
        print(json.dumps(summarize_pmc(*args.summarize_pmc, args.command, args.command2), indent=1))
        return
    if args.summarize_traffic:
        print(summarize_traffic(*args.summarize_traffic, args.command, args.command2), end="")
        return
    if args.summarize_counters:
        print(summarize_counters(args.summarize_counters, args.command), end="")
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU's share of the path; runs on more than one GPU are not "
              "supported (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2110_09132_amd as emb
    from workloads import configs

    wl = configs.WORKLOADS[args.workload]
    log(f"workload {wl.name}: {wl.description}")
    run = WorkloadRun(torch, emb, wl, args.batches, args.schedule)
    pl = pipelined_report(run, args, args.steps)
    order, nsets, paired = pl["cand"]
    log(f"schedule: {cand_name(pl['cand'])} {pl['tune_ms'] or ''}")
    log(f"timed {args.steps} steps: {pl['ms_step']:.4f} ms/step")
    split, by_owner = run.split, run.by_owner
    used = pl["used"]
    U, U_prior = run.U, run.U_prior
    ms_step = pl["ms_step"]

    # sizes of the sparse gradient as Table 3 reports them (per step, all tables): the per-token
    # COO gradient (original), after COALESCE (coalesced), and the prior part of the vertical split
    # (prioritized: rows whose id is in the next batch, the part that must arrive before the next
    # forward pass); ids int32, rows in the gradient's element type
    def mb(rows, sp):
        return rows * (4 + sp.D * (2 if sp.grad_dtype == "bf16" else 4)) / 1e6
    nt, nb = len(run.tables), args.batches
    orig = sum(mb(sp.T, sp) for sp in wl.tables)
    coal = sum(mb(U[b][k], wl.tables[k]) for b in range(nb) for k in range(nt)) / nb
    prio = sum(mb(U_prior[b][k], wl.tables[k]) for b in range(nb) for k in range(nt)) / nb
    table3 = {"original_MB": orig, "coalesced_MB": coal, "prioritized_MB": prio,
              "reduction_by_coalescing": 1 - coal / orig, "further_reduction_by_prioritizing": 1 - prio / coal,
              "next_batch": "the next batch of the rotation"}
    prior_frac = sum(U_prior[b][k] for b in used for k in range(nt)) / max(1, sum(
        U[b][k] for b in used for k in range(nt)))

    result = {
        "metric": "unique grad rows/sec for coalesce+pack+update; achieved HBM GB/s vs peak",
        "value": pl["rows"] / (pl["ms_total"] * 1e-3),
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
                   "mean_unique_rows_per_step": pl["rows"] / args.steps, "batches_rotated": args.batches,
                   "coalesce": {"split": "emb_grad_coalesce_split (owner-major, prior/delayed split)",
                                "by_owner": "emb_grad_coalesce_by_owner (coalesce straight into the send layout)",
                                "unfused": "emb_grad_coalesce + emb_pack_by_owner"}[args.schedule],
                   "schedule": "one stream" if args.sequential else
                   {"split": "sort, reduction and delayed update on three side streams; lookup and prior "
                             "update on the main stream",
                    "by_owner": "sort and reduction on two side streams; lookup and update on the main stream",
                    "unfused": "coalesce and pack on two side streams; lookup and update on the main stream"}[
                       args.schedule],
                   "sort_streams": None if (args.sequential or split or not by_owner) else
                   (nsets // 2 if nsets in (4, 6) else 1),
                   "buffer_sets": nsets,
                   "sort_and_reduce_paired": paired,
                   "cross_stream_order": None if args.sequential else
                   {"signals": "step signals (hipStreamWriteValue32 / hipStreamWaitValue32)",
                    "events": "events (hipEventRecord / hipStreamWaitEvent)",
                    "queued": "events, each step enqueued from two host threads (emb_train_step_queued)"}[order],
                   "schedule_tuning_ms_per_step": pl["tune_ms"] or None,
                   "prior_rows_frac": prior_frac if split else None},
        "step_bytes_model": pl["total_bytes"],
        "step_bytes_model_kind": "fused minimum (pack folded into coalesce)" if by_owner else "four calls",
        "stage_bytes_model": pl["bytes_step"],
        "step_hbm_GBps": pl["step_gbps"],
        "step_hbm_frac": pl["step_gbps"] / HBM_PEAK_GBPS,
        "wall_s_timed": pl["wall"],
        "host_enqueue_ms_timed": pl["host_enqueue_ms"],
        "roofline": {"bound": "hbm",
                     "kernel": "adam_kernel (emb_sparse_adam_apply)" + (", delayed rows" if split else ""),
                     "achieved": pl["adam_gbps"], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": pl["adam_gbps"] / HBM_PEAK_GBPS,
                     "traffic": measured_traffic() if args.workload == "lowdup_uniform" else None,
                     "bytes_per_launch": pl["adam_bytes"], "avg_launch_us": pl["adam_us"],
                     "launches_timed": len(pl["adam_us_all"]),
                     "launch_us_spread": spread(pl["adam_us_all"]),
                     "window": f"{args.roofline_steps} steps after the timed ones, same schedule, the update "
                               f"timed on every {args.roofline_every}th",
                     "window_ms_per_step": pl["window_ms_step"],
                     "steps_before_window": pl["steps_before_window"]},
        "gradient_sizes_table3": table3,
        "host": host_info(),
    }
    copy_gbps = copy_reference(torch)  # also the calibration dispatch of the byte counters
    result["copy_GBps"] = copy_gbps
    result["step_frac_of_copy"] = pl["step_gbps"] / copy_gbps
    if not args.only_steps:
        log("sequential warm and cold runs ...")
        seqr = sequential_report(run, args.seq_steps)
        result["timing_protocol"] = seqr
        result["stage_ms_sequential"] = {k: v["median"] for k, v in seqr["warm"]["stage_ms"].items()}
        result["sequential_ms_per_step"] = seqr["warm"]["step_ms"]["median"]
        log("column partition, cost model, exchanges ...")
        sp0, tb0 = wl.tables[0], run.tables[0]
        batches0 = [x[0] for x in run.step_batches]
        U0 = [U[b][0] for b in range(nb)]
        result["column_partition"] = column_partition_report(torch, emb, sp0, tb0, batches0, U0, run.owner_rows)
        result["forward_exchange"] = forward_exchange_report(torch, emb, sp0, tb0, batches0, U0)
        result["gradient_exchange"] = exchange_report(torch, emb, sp0, tb0, batches0)
        result["comm_cost_model"] = cost_model_report(emb, sp0, U0)
        if not args.no_configs and not args.sequential:
            # every workload, at least config_steps timed steps each (the headline workload again,
            # in a fresh run, unless its timed steps were that many)
            K = max(args.steps, args.config_steps)
            reuse = K == args.steps
            if not reuse:
                run.release()
                run = None
            cfgs = {}
            for name in configs.WORKLOADS:
                if reuse and name == wl.name:
                    cfgs[name] = config_report(torch, emb, name, args, K, run=run, pl=pl)
                else:
                    cfgs[name] = config_report(torch, emb, name, args, K)
            result["configs"] = cfgs
    if run is not None:
        run.release()
    if not args.no_cpu_baseline and not args.only_steps:
        log("timing the CPU oracle ...")
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
