"""Parity of emb_grad_coalesce_by_owner (coalesce straight into the per-owner
send layout) with the oracle's pack_by_owner applied to its coalesce: ids,
counts and offsets bit-exact, rows within the summation bound, rows of one or
two tokens bit-exact, token counts per row equal to the oracle's segment
lengths.  Sizes span several sort tiles and reduction chunks with ragged
tails; owner maps by id mod P, by range and at random; bad ids and owners;
empty and degenerate batches; the key-width limit."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2110_09132_amd as emb
import tolerance
from gpu_helpers import host, runs_ids, to_dev
from workloads import configs, gen

pytestmark = pytest.mark.gpu


def ids_for(law, seed, T, V, s=1.1):
    key = gen.stream_key(seed, 0, gen.PURPOSE_IDS)
    return gen.uniform_ids(key, T, V) if law == "uniform" else gen.zipf_ids(key, T, V, s)


def grads_for(seed, T, D, sigma=1.0, bf16=False):
    g = gen.normal_f32(gen.stream_key(seed, 0, gen.PURPOSE_GRADS), T * D, sigma).reshape(T, D)
    return gen.bf16_round(g).reshape(T, D) if bf16 else g


def owners(rule, V, P, seed=0):
    if rule == "mod":
        return gen.owner_mod(V, P)
    if rule == "range":
        return gen.owner_range(V, P)
    return np.random.default_rng(seed).integers(0, P, V).astype(np.int32)


def gpu_by_owner(ids_np, grad_np, V, own_np, P, grad_dev=None):
    st = emb.new_status()
    g = to_dev(grad_np) if grad_dev is None else grad_dev
    out = emb.grad_coalesce_by_owner(to_dev(ids_np.astype(np.int32)), g, V, to_dev(own_np.astype(np.int32)), P,
                                     dev_status=st)
    torch.cuda.synchronize()
    send_ids, seg, rows, counts, offs, nu = out
    U = int(nu.item())
    return dict(U=U, send_ids=host(send_ids[:U]), seg_offsets=host(seg[:U + 1]), send_rows=host(rows[:U]),
                send_counts=host(counts), send_offsets=host(offs), status=int(st.item()), dev=out)


def check_by_owner(ids_np, grad_np, V, own_np, P, bf16=False, grad_dev=None):
    orc = oracle.coalesce(ids_np, grad_np, V, grad_is_bf16=bf16)
    pk = oracle.pack_by_owner(orc["uniq_ids"], orc["uniq_grad"], own_np, P)
    gpu = gpu_by_owner(ids_np, grad_np, V, own_np, P, grad_dev=grad_dev)
    n = int(pk["send_offsets"][P])
    assert gpu["U"] == n, (gpu["U"], n)
    for k in ("send_ids", "send_counts", "send_offsets"):
        assert np.array_equal(gpu[k], pk[k]), k
    # each sent row against the oracle's exact sum of its id
    idx = np.searchsorted(orc["uniq_ids"], pk["send_ids"])
    assert np.array_equal(orc["uniq_ids"][idx], pk["send_ids"])
    r = tolerance.assert_grad_close(gpu["send_rows"], orc["sum_f64"][idx], orc["absum"][idx], tolerance.RTOL_F32)
    seglen = np.diff(orc["seg_offsets"])[idx]
    assert gpu["seg_offsets"][0] == 0 and np.array_equal(np.diff(gpu["seg_offsets"]), seglen)
    short = seglen <= 2
    assert np.array_equal(gpu["send_rows"][short].view(np.uint32), orc["uniq_grad"][idx][short].view(np.uint32))
    bad_owner = np.any((own_np[orc["uniq_ids"]] < 0) | (own_np[orc["uniq_ids"]] >= P)) if orc["U"] else False
    expect = (emb.EMB_DEV_ID_OUT_OF_RANGE if orc["n_invalid"] else 0) | \
             (emb.EMB_DEV_OWNER_OUT_OF_RANGE if bad_owner else 0)
    assert gpu["status"] == expect, (gpu["status"], expect)
    return gpu, r


@pytest.mark.parametrize("law,V,T,D,P,rule", [
    ("zipf", 1000, 512, 64, 2, "mod"),              # the tiny workload's shape
    ("zipf", 32768, 25000, 64, 4, "range"),         # shared-vocab shape, narrower rows
    ("zipf", 32000, 16384, 32, 8, "mod"),           # translation shape, narrower rows
    ("uniform", 1 << 20, 20000, 16, 16, "mod"),     # 20 + 4 key bits: three 8-bit passes
    ("zipf", 5000, 2049, 3, 7, "rand"),             # ragged tile, scalar width path
    ("zipf", 300, 4001, 256, 5, "rand"),            # heavy duplication
    ("uniform", 50, 33, 1, 3, "mod"),               # one chunk + 1, D = 1
    ("zipf", 1, 777, 4, 1, "mod"),                  # V = 1, P = 1: every key 0
    ("zipf", 1, 777, 4, 9, "rand"),                 # V = 1, one owner of nine
    ("uniform", 50000, 9000, 20, 1024, "mod"),      # the most owners: 16 + 10 key bits, three 9-bit passes
    ("uniform", 50000, 9000, 20, 1024, "range"),
    ("uniform", (1 << 22) - 1, 9000, 4, 1024, "rand"),  # 22 + 10 = 32 key bits: four passes
    ("uniform", 1 << 21, 20000, 8, 16, "mod"),     # 21 + 4 = 25 key bits: three 9-bit passes (9, 9, 7)
    ("zipf", 256, 5000, 8, 2, "mod"),              # 8 + 1 = 9 key bits: one 9-bit pass
    ("uniform", (1 << 24) + 3, 9000, 4, 128, "mod"),    # 25 + 7 = 32 key bits, the widest that fits
    # 1536-key sort tiles (more than 32768 tokens): 8-bit digits, 9-bit digits, four passes
    ("zipf", 1 << 16, 40001, 8, 4, "range"),        # 16 + 2 = 18 key bits: two 9-bit passes
    ("uniform", 1 << 20, 33000, 8, 64, "rand"),     # 20 + 6 = 26 key bits: three 9-bit passes
    ("uniform", (1 << 22) - 1, 50000, 4, 1024, "rand"),  # 32 key bits: four 8-bit passes
    ("uniform", 1 << 20, 1 << 21, 4, 16, "mod"),   # two million tokens: 1366 sort tiles, 16384 reduction workgroups
    # the one-workgroup path (at most 2048 tokens): the most owners, 32 key bits, a device-side count
    ("uniform", 50000, 2048, 20, 1024, "rand"),
    ("uniform", (1 << 22) - 1, 1500, 4, 1024, "rand"),
    ("zipf", 5000, 1000, 256, 16, "mod"),
])
def test_by_owner_parity(law, V, T, D, P, rule):
    ids = ids_for(law, V + T + P, T, V)
    check_by_owner(ids, grads_for(V + D, T, D), V, owners(rule, V, P, seed=T), P)


@pytest.mark.parametrize("V,T,D,P", [(262144, 16384, 1024, 8), (1000, 3000, 10, 3)])
def test_by_owner_parity_bf16(V, T, D, P):
    ids = ids_for("zipf", V + T, T, V, 1.0)
    G = grads_for(V + D, T, D, 0.01, bf16=True)
    check_by_owner(ids, G, V, gen.owner_range(V, P), P, bf16=True)


@pytest.mark.parametrize("name", ["tiny", "transformer_shared_vocab", "two_table_translation",
                                  "lm_large_vocab_bf16", "lowdup_zipf13"])
def test_by_owner_workload_full_shape(name):
    """The call the benchmark's steps make, on each workload's own batches at full shape, every table:
    rows of 512 fp32 (shared vocabulary), 1024 fp32 (two tables), 1024 bf16 (large vocabulary)."""
    wl = configs.WORKLOADS[name]
    for k, sp in enumerate(wl.tables):
        print(f"[{name}] table {k}: V={sp.V} D={sp.D} T={sp.T} P={sp.P} {sp.owner_rule}", flush=True)
        ids, G = configs.make_batch(sp, 900 + k)
        check_by_owner(ids, G, sp.V, configs.row_owner(sp), sp.P, bf16=sp.grad_dtype == "bf16")


def test_by_owner_hot_row_spans_many_chunks():
    T, V, D, P = 20000, 5000, 256, 4
    ids = ids_for("zipf", 77, T, V, 2.5)
    check_by_owner(ids, grads_for(78, T, D, 0.01), V, gen.owner_mod(V, P), P)


@pytest.mark.parametrize("seed,rule,bad_frac", [(5, "range", 0.0), (6, "range", 0.01), (7, "mod", 0.0)])
def test_by_owner_runs_around_chunk_and_workgroup_boundaries(seed, rule, bad_frac):
    # with contiguous owners the sorted sequence is the runs in order (as for the plain call); with
    # id mod P each owner's runs follow one another
    V, P = 1 << 16, 4
    ids = runs_ids(seed, 300, V, bad_frac)
    G = grads_for(seed + 20, ids.size, 64)
    check_by_owner(ids, G, V, owners(rule, V, P), P)


def test_by_owner_lowdup_full_size():
    # the low-duplication stress shape: V = 2^20, D = 256, T = 65536 uniform ids, P = 16 by id mod P
    V, T, D, P = 1 << 20, 65536, 256, 16
    ids = ids_for("uniform", 51, T, V)
    check_by_owner(ids, grads_for(51, T, D, 0.01), V, gen.owner_mod(V, P), P)


def test_by_owner_bad_ids_and_owners_are_left_out():
    V, T, D, P = 1000, 3000, 16, 4
    ids = ids_for("zipf", 9, T, V)
    ids[::97] = -3
    ids[5::101] = V + 5
    own = gen.owner_mod(V, P)
    own[[0, 1, 7, 500]] = [P, -1, 1 << 20, P + 3]
    gpu, _ = check_by_owner(ids, grads_for(9, T, D), V, own, P)
    assert gpu["status"] == emb.EMB_DEV_ID_OUT_OF_RANGE | emb.EMB_DEV_OWNER_OUT_OF_RANGE


def test_by_owner_every_owner_bad():
    V, T, D, P = 100, 500, 4, 3
    own = np.full(V, 5, np.int32)
    gpu = gpu_by_owner(ids_for("uniform", 1, T, V), grads_for(1, T, D), V, own, P)
    assert gpu["U"] == 0 and gpu["send_offsets"].tolist() == [0] * (P + 1)
    assert gpu["send_counts"].tolist() == [0] * P and gpu["seg_offsets"].tolist() == [0]
    assert gpu["status"] == emb.EMB_DEV_OWNER_OUT_OF_RANGE


def test_by_owner_empty_batch():
    P = 5
    gpu = gpu_by_owner(np.zeros(0, np.int32), np.zeros((0, 8), np.float32), 50, gen.owner_mod(50, P), P)
    assert gpu["U"] == 0 and gpu["send_offsets"].tolist() == [0] * (P + 1)
    assert gpu["send_counts"].tolist() == [0] * P and gpu["status"] == 0


def test_by_owner_empty_owners_between_full_ones():
    # owners 0, 2 and 5 hold every row: 1, 3, 4 stay empty in the middle
    V, T, D, P = 600, 4000, 8, 6
    own = np.array([0, 2, 5], np.int32)[np.arange(V) % 3]
    check_by_owner(ids_for("zipf", 3, T, V), grads_for(3, T, D), V, own, P)


def test_by_owner_misaligned_gradient_rows_use_scalar_path():
    V, T, D, P = 2000, 3000, 64, 4
    ids = ids_for("zipf", 11, T, V)
    G = grads_for(11, T, D)
    buf = torch.zeros(T * D + 1, dtype=torch.float32, device="cuda")
    buf[1:] = to_dev(G.reshape(-1))
    check_by_owner(ids, G, V, gen.owner_mod(V, P), P, grad_dev=buf[1:].view(T, D))


def test_by_owner_is_bitwise_deterministic():
    V, T, D, P = 1 << 20, 65536, 256, 16
    ids = ids_for("zipf", 52, T, V, 1.3)
    G = to_dev(grads_for(52, T, D, 0.01))
    own = gen.owner_mod(V, P)
    a = gpu_by_owner(ids, None, V, own, P, grad_dev=G)
    b = gpu_by_owner(ids, None, V, own, P, grad_dev=G)
    assert a["U"] == b["U"] and np.array_equal(a["send_ids"], b["send_ids"])
    assert np.array_equal(a["send_rows"].view(np.uint32), b["send_rows"].view(np.uint32))


def test_by_owner_key_width_limit_is_unsupported():
    # bits(V) + bits(P) = 31 + 2 > 32: the call refuses before launching anything
    V, P, T, D = (1 << 31) - 1, 4, 16, 4
    ids = to_dev(np.arange(T, dtype=np.int32))
    own = torch.zeros(1, dtype=torch.int32, device="cuda")  # never read: the host check fails first
    g = to_dev(grads_for(1, T, D))
    outs = [torch.zeros(T + 1, dtype=torch.int32, device="cuda") for _ in range(5)]
    out_rows = torch.zeros((T, D), dtype=torch.float32, device="cuda")
    ws = emb.new_workspace(1 << 20)
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    code = emb.lib.emb_grad_coalesce_by_owner(p(ids), T, p(g), emb.EMB_F32, D, V, p(own), P, p(outs[0]), p(outs[1]),
                                              p(out_rows), p(outs[2]), p(outs[3]), p(outs[4]), p(ws), ws.numel(),
                                              None, None)
    assert code == emb.EMB_ERR_UNSUPPORTED
    # the binding refuses the owner map, one owner for 2^31 - 1 rows, before that
    with pytest.raises(emb.EmbError, match="row_owner"):
        emb.grad_coalesce_by_owner(ids, g, V, own, P)


# ------------------------------------------------------ vertical split (Algorithm 1)
def gpu_split(ids_np, next_np, grad_np, V, own_np, P, grad_dev=None):
    st = emb.new_status()
    g = to_dev(grad_np) if grad_dev is None else grad_dev
    out = emb.grad_coalesce_split(to_dev(ids_np.astype(np.int32)), to_dev(next_np.astype(np.int32)), g, V,
                                  to_dev(own_np.astype(np.int32)), P, dev_status=st)
    torch.cuda.synchronize()
    send_ids, seg, rows, counts, offs, nu = out
    U = int(nu.item())
    return dict(U=U, send_ids=host(send_ids[:U]), seg_offsets=host(seg[:U + 1]), send_rows=host(rows[:U]),
                send_counts=host(counts), send_offsets=host(offs), status=int(st.item()), dev=out)


def check_split(ids_np, next_np, grad_np, V, own_np, P, bf16=False):
    """GPU split vs the oracle's split_pack of its coalesce: ids, counts and offsets bit-exact, rows
    within the summation bound (bit-exact for one or two tokens), token counts per row exact."""
    orc = oracle.coalesce(ids_np, grad_np, V, grad_is_bf16=bf16)
    sp = oracle.split_pack(orc["uniq_ids"], orc["uniq_grad"], next_np, own_np, P)
    gpu = gpu_split(ids_np, next_np, grad_np, V, own_np, P)
    n = int(sp["send_offsets"][2 * P])
    assert gpu["U"] == n, (gpu["U"], n)
    for k in ("send_ids", "send_counts", "send_offsets"):
        assert np.array_equal(gpu[k], sp[k]), k
    idx = np.searchsorted(orc["uniq_ids"], sp["send_ids"])
    tolerance.assert_grad_close(gpu["send_rows"], orc["sum_f64"][idx], orc["absum"][idx], tolerance.RTOL_F32)
    seglen = np.diff(orc["seg_offsets"])[idx]
    assert gpu["seg_offsets"][0] == 0 and np.array_equal(np.diff(gpu["seg_offsets"]), seglen)
    short = seglen <= 2
    assert np.array_equal(gpu["send_rows"][short].view(np.uint32), orc["uniq_grad"][idx][short].view(np.uint32))
    return gpu, sp


@pytest.mark.parametrize("law,V,T,D,P,rule", [
    ("zipf", 1000, 512, 64, 2, "mod"),            # the tiny workload's shape
    ("zipf", 32768, 25000, 64, 4, "range"),       # shared-vocab shape, narrower rows
    ("uniform", 1 << 20, 20000, 16, 16, "mod"),   # 20 + 4 + 1 key bits: three 9-bit passes
    ("zipf", 5000, 2049, 3, 7, "rand"),           # ragged tile, scalar width path
    ("zipf", 1, 777, 4, 1, "mod"),                # V = 1, P = 1: keys 0 and 1 only
    ("uniform", 50000, 9000, 20, 1024, "mod"),    # the most owners: 16 + 10 + 1 = 27 key bits, 9 bits a pass
    ("uniform", (1 << 21) - 1, 9000, 4, 1024, "rand"),  # 21 + 10 + 1 = 32 key bits
    # the one-workgroup path: 2048 groups (the most), a hash set of next ids (V > 2^24)
    ("uniform", 50000, 2048, 20, 1024, "mod"),
    ("uniform", (1 << 24) + 5, 1800, 4, 4, "mod"),
])
def test_split_parity(law, V, T, D, P, rule):
    ids = ids_for(law, V + T + P, T, V)
    nxt = ids_for(law, V + T + P + 1, T, V)
    check_split(ids, nxt, grads_for(V + D, T, D), V, owners(rule, V, P, seed=T), P)


def test_split_lowdup_full_size():
    V, T, D, P = 1 << 20, 65536, 256, 16
    ids, nxt = ids_for("uniform", 51, T, V), ids_for("uniform", 52, T, V)
    gpu, sp = check_split(ids, nxt, grads_for(51, T, D, 0.01), V, gen.owner_mod(V, P), P)
    assert 0 < sp["n_prior"] < gpu["U"]


def test_split_bf16():
    V, T, D, P = 262144, 16384, 1024, 8
    ids, nxt = ids_for("zipf", 4, T, V, 1.0), ids_for("zipf", 5, T, V, 1.0)
    check_split(ids, nxt, grads_for(4, T, D, 0.01, bf16=True), V, gen.owner_range(V, P), P, bf16=True)


@pytest.mark.parametrize("case", ["same", "disjoint", "empty", "not_rows", "longer"])
def test_split_degenerate_next_batches(case):
    V, T, D, P = 3000, 4000, 8, 5
    ids = ids_for("zipf", 8, T, V)
    nxt = {"same": ids[::-1].copy(),
           "disjoint": np.setdiff1d(np.arange(V, dtype=np.int32), ids).astype(np.int32),
           "empty": np.zeros(0, np.int32), "not_rows": np.array([-5, V, V + 1, 1 << 30], np.int32),
           "longer": ids_for("uniform", 9, 3 * T, V)}[case]
    gpu, sp = check_split(ids, nxt, grads_for(8, T, D), V, gen.owner_mod(V, P), P)
    if case == "same":
        assert sp["n_prior"] == gpu["U"]
    if case in ("disjoint", "empty", "not_rows"):
        assert sp["n_prior"] == 0


def test_split_bad_ids_and_owners_are_left_out():
    V, T, D, P = 1000, 3000, 16, 4
    ids = ids_for("zipf", 9, T, V)
    ids[::97] = -3
    nxt = ids_for("zipf", 10, T, V)
    own = gen.owner_mod(V, P)
    own[[0, 1, 500]] = [P, -1, P + 3]
    gpu, _ = check_split(ids, nxt, grads_for(9, T, D), V, own, P)
    assert gpu["status"] == emb.EMB_DEV_ID_OUT_OF_RANGE | emb.EMB_DEV_OWNER_OUT_OF_RANGE


def test_split_empty_batch():
    P = 3
    gpu = gpu_split(np.zeros(0, np.int32), np.arange(5, dtype=np.int32), np.zeros((0, 4), np.float32), 50,
                    gen.owner_mod(50, P), P)
    assert gpu["U"] == 0 and gpu["send_offsets"].tolist() == [0] * (2 * P + 1)
    assert gpu["send_counts"].tolist() == [0] * (2 * P) and gpu["status"] == 0


def test_split_key_width_limit_is_unsupported():
    # bits(V) + bits(P) + 1 = 22 + 10 + 1 > 32: refused on the host
    V, P, T, D = (1 << 22) - 1, 1024, 16, 4
    ids = to_dev(np.arange(T, dtype=np.int32))
    own = torch.zeros(V, dtype=torch.int32, device="cuda")  # never read: the host check fails first
    with pytest.raises(emb.EmbError, match="unsupported"):
        emb.grad_coalesce_split(ids, ids, to_dev(grads_for(1, T, D)), V, own, P)


def test_split_hash_set_path_for_huge_tables():
    # above 2^24 rows the next-batch set is a hash set instead of a byte per row
    V, T, D, P = (1 << 24) + 5, 5000, 4, 4
    ids = ids_for("uniform", 71, T, V)
    nxt = np.concatenate([ids[: T // 3], ids_for("uniform", 72, T, V)]).astype(np.int32)
    gpu, sp = check_split(ids, nxt, grads_for(71, T, D), V, gen.owner_mod(V, P), P)
    assert 0 < sp["n_prior"] < gpu["U"]
    # hot rows repeated across the whole next batch (the per-workgroup LDS set drops repeats)
    nxt2 = np.concatenate([np.repeat(ids[:7], 3000), ids_for("zipf", 73, T, V, 1.3)]).astype(np.int32)
    check_split(ids, nxt2, grads_for(72, T, D), V, gen.owner_mod(V, P), P)
