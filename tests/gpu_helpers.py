"""Drivers that run the HIP library (through the C ABI binding) on numpy inputs
and compare each call with the oracle on identical inputs."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2110_09132_amd as emb
import tolerance
from pins import check_pack_result

DEV = "cuda"


def to_dev(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:  # bf16 bit patterns
        return torch.from_numpy(a.view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(a).to(DEV)


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


def gpu_gather(W_dev, ids_np):
    st = emb.new_status()
    out = emb.gather(W_dev, to_dev(ids_np.astype(np.int32)), dev_status=st)
    torch.cuda.synchronize()
    return host(out), int(st.item())


def gpu_coalesce(ids_np, grad_np, V, grad_dev=None):
    ids = to_dev(ids_np.astype(np.int32))
    g = to_dev(grad_np) if grad_dev is None else grad_dev
    st = emb.new_status()
    dev_out = emb.grad_coalesce(ids, g, V, dev_status=st)
    torch.cuda.synchronize()
    uid, seg, ug, nu = dev_out
    U = int(nu.item())
    return dict(U=U, uniq_ids=host(uid[:U]), seg_offsets=host(seg[:U + 1]), uniq_grad=host(ug[:U]),
                status=int(st.item()), dev=dev_out)


def check_coalesce(ids_np, grad_np, V, bf16=False, rtol=None, grad_dev=None):
    """GPU coalesce vs the oracle: integers bit-exact, sums within the summation bound,
    segments of one or two tokens bit-exact (a copy, or one correctly rounded add)."""
    orc = oracle.coalesce(ids_np, grad_np, V, grad_is_bf16=bf16)
    gpu = gpu_coalesce(ids_np, grad_np, V, grad_dev=grad_dev)
    assert gpu["U"] == orc["U"], (gpu["U"], orc["U"])
    assert np.array_equal(gpu["uniq_ids"], orc["uniq_ids"])
    assert np.array_equal(gpu["seg_offsets"], orc["seg_offsets"])
    r = tolerance.assert_grad_close(gpu["uniq_grad"], orc["sum_f64"], orc["absum"],
                                    rtol if rtol is not None else tolerance.RTOL_F32)
    short = np.diff(orc["seg_offsets"]) <= 2
    assert np.array_equal(gpu["uniq_grad"][short].view(np.uint32), orc["uniq_grad"][short].view(np.uint32))
    expect_flag = emb.EMB_DEV_ID_OUT_OF_RANGE if orc["n_invalid"] else 0
    assert gpu["status"] == expect_flag
    return gpu, orc, r


def gpu_pack(coal_dev, row_owner_np, P):
    uid, _, ug, nu = coal_dev
    st = emb.new_status()
    out = emb.pack_by_owner(uid, ug, nu, to_dev(row_owner_np.astype(np.int32)), P, dev_status=st)
    torch.cuda.synchronize()
    send_ids, send_rows, counts, offs = out
    n = int(offs[P].item())
    return dict(send_ids=host(send_ids[:n]), send_rows=host(send_rows[:n]), send_counts=host(counts),
                send_offsets=host(offs), status=int(st.item()), dev=out)


def check_pack(coal_dev, U, row_owner_np, P):
    """GPU pack vs the oracle on the GPU's own coalesce output: all bit-exact."""
    uid, _, ug, _ = coal_dev
    uid_h, ug_h = host(uid[:U]), host(ug[:U])
    orc = oracle.pack_by_owner(uid_h, ug_h, row_owner_np, P)
    gpu = gpu_pack(coal_dev, row_owner_np, P)
    for k in ("send_ids", "send_counts", "send_offsets"):
        assert np.array_equal(gpu[k], orc[k]), k
    assert np.array_equal(gpu["send_rows"].view(np.uint32), orc["send_rows"].view(np.uint32))
    check_pack_result(gpu, uid_h, ug_h, row_owner_np, P)
    assert gpu["status"] == 0
    return gpu


def check_adam(state_dev, pack_dev, P, shard_begin, shard_end, hp, step, rtol=tolerance.RTOL_F32):
    """GPU Adam vs the oracle on identical inputs (the GPU's pre-call state of the
    touched rows and the GPU pack output): W, m, v rows, and the update W_after - W_before on
    its own scale.  Rows not listed must stay bit-identical."""
    W, M, S = state_dev
    send_ids, send_rows, _, offs = pack_dev
    offs_h = host(offs)
    lo, hi = int(offs_h[shard_begin]), int(offs_h[shard_end])
    rid = host(send_ids[lo:hi]).astype(np.int64)
    rows_h = host(send_rows[lo:hi])
    before = [host(t[torch.from_numpy(rid).to(DEV)]) for t in (W, M, S)]
    snap = [t.clone() for t in (W, M, S)]
    st = emb.new_status()
    emb.sparse_adam_apply(W, M, S, send_ids, send_rows, offs, P, shard_begin, shard_end, hp["lr"], hp["beta1"],
                          hp["beta2"], hp["eps"], step, dev_status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    # oracle on a compact table holding just the touched rows
    n = rid.size
    Wc, Mc, Sc = (np.array(b.reshape(n, -1), copy=True) for b in before)  # `before` stays as it was
    oracle.sparse_adam(Wc, Mc, Sc, np.arange(n, dtype=np.int32), rows_h, np.array([0, n], np.int32), 0, 1,
                       hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], step)
    idx = torch.from_numpy(rid).to(DEV)
    ratios = []
    for t, ref, name in ((W, Wc, "table"), (M, Mc, "exp_avg"), (S, Sc, "exp_avg_sq")):
        ratios.append(tolerance.assert_rows_close(host(t[idx]), ref, rtol, name))
    # the update itself, on its own scale (Sec. 5.7; Kingma & Ba, Algorithm 1)
    ratios.append(tolerance.assert_update_close(host(W[idx]), before[0], Wc, rtol, what="table update"))
    mask = torch.ones(W.shape[0], dtype=torch.bool, device=DEV)
    mask[idx] = False
    for t, s in zip((W, M, S), snap):
        assert torch.equal(t[mask], s[mask]), "an untouched row changed"
    return max(ratios)


def check_steps_against_oracle(wl, tbs, W0s, owns, host_batches, steps, split, looked=None, seed=7):
    """The state the step executor left after `steps` steps of workload `wl` (one buffer set per step,
    so every step's send buffers survive) against the oracle, for every table:
      - each step's send layout (ids, counts, offsets; with the split, the 2P groups of the prior and
        delayed rows) bit-exact against the oracle's owner-major pack (or split pack) of its coalesce,
        and the rows within the fp32 summation bound;
      - each step's sampled lookup (looked[s][k] = (positions, rows), if given) against the table as
        the previous steps left it, replayed on the CPU: bit-exact at the first step, then to the Adam
        tolerance;
      - W, m, v after the steps against the oracle's Adam applied to the GPU's own send rows, on a
        sample of touched rows, with the update W_after - W_before judged on its own scale, and
        untouched rows bit-identical.
    host_batches[s][k] = (ids, grads) of step s (steps + 1 of them with the split: the last is only
    the next batch)."""
    rng = np.random.default_rng(seed)
    for k, (sp, tb, W0, own) in enumerate(zip(wl.tables, tbs, W0s, owns)):
        bf16 = sp.grad_dtype == "bf16"
        G_of = [host_batches[s][k] for s in range(len(host_batches))]
        # rows to replay on the CPU: some of every batch, plus untouched ones
        touched = np.unique(np.concatenate([ids for ids, _ in G_of[:steps]]))
        extra = [G_of[s][0][looked[s][k][0]] for s in range(steps)] if looked is not None else []
        sample = np.unique(np.concatenate([rng.choice(touched, min(384, touched.size), replace=False)] + extra))
        untouched = np.setdiff1d(rng.choice(sp.V, min(sp.V, 2048), replace=False), touched)[:64]
        idx = {int(r): i for i, r in enumerate(sample)}
        Wc = W0[sample].copy()
        Mc = np.zeros_like(Wc)
        Sc = np.zeros_like(Wc)
        for s in range(steps):
            ids, G = G_of[s]
            if looked is not None:
                pos, got = looked[s][k]
                want = Wc[[idx[int(i)] for i in ids[pos]]]
                if s == 0:
                    assert np.array_equal(host(got).view(np.uint32), want.view(np.uint32)), \
                        f"table {k}: lookup of step 1"
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


# run lengths around the reduction's 32-token chunks and 128-token workgroups
RUN_LENGTHS = [1, 2, 3, 30, 31, 32, 33, 34, 62, 63, 64, 65, 66, 95, 96, 97, 126, 127, 128, 129, 130, 160, 255, 256,
               257, 300, 511, 512, 513]


def runs_ids(seed, n_runs, V, bad_frac=0.0):
    """Ids in runs of the lengths above (each run one id, ids ascending with gaps), tokens shuffled:
    the sorted sequence is the runs in order, so their ends fall at every offset from the chunk and
    workgroup boundaries.  bad_frac of the tokens get an id past V (left out of the sort)."""
    rng = np.random.default_rng(seed)
    lengths = rng.choice(RUN_LENGTHS, n_runs)
    vals = np.cumsum(rng.integers(1, 40, n_runs))
    assert vals[-1] < V
    ids = np.repeat(vals, lengths).astype(np.int32)
    bad = rng.random(ids.size) < bad_frac
    ids[bad] = V + rng.integers(0, 1000, int(bad.sum()))
    rng.shuffle(ids)
    return ids
