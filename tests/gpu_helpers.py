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
