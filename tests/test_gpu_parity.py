"""Parity of each C ABI call with the oracle at sizes the oracle finishes in
seconds: several sort tiles (1024 keys, 1536 above 32768 tokens) and reduction chunks (32 tokens) with
ragged tails, every gradient width path (vector and scalar), bf16 gradients,
hot rows spanning many chunks, empty and degenerate inputs."""
import numpy as np
import pytest
import torch

import oracle
import paper_2110_09132_amd as emb
import tolerance
from adam_inputs import eps_regime_grads
from gpu_helpers import (check_adam, check_coalesce, check_pack, gpu_coalesce, gpu_gather, host, runs_ids, to_dev)
from workloads import gen

pytestmark = pytest.mark.gpu

HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8)


def ids_for(law, seed, T, V, s=1.1):
    key = gen.stream_key(seed, 0, gen.PURPOSE_IDS)
    return gen.uniform_ids(key, T, V) if law == "uniform" else gen.zipf_ids(key, T, V, s)


def grads_for(seed, T, D, sigma=1.0, bf16=False):
    g = gen.normal_f32(gen.stream_key(seed, 0, gen.PURPOSE_GRADS), T * D, sigma).reshape(T, D)
    return gen.bf16_round(g).reshape(T, D) if bf16 else g


# ---------------------------------------------------------------------- gather
@pytest.mark.parametrize("D", [1, 3, 64, 65, 256, 1024])
@pytest.mark.parametrize("T", [1, 2047, 2049, 5000])
def test_gather_parity(D, T):
    V = 3000
    W = gen.normal_f32(gen.stream_key(D, T, gen.PURPOSE_WEIGHTS), V * D).reshape(V, D)
    ids = ids_for("zipf", D + T, T, V)
    out, st = gpu_gather(to_dev(W), ids)
    ref, bad = oracle.gather(W, ids)
    assert bad == 0 and st == 0
    assert np.array_equal(out.view(np.uint32), ref.view(np.uint32))


def test_gather_out_of_range_ids_give_zero_rows_and_flag():
    V, D, T = 100, 8, 300
    W = gen.normal_f32(gen.stream_key(1, 0, 1), V * D).reshape(V, D)
    ids = ids_for("uniform", 2, T, V)
    ids[[0, 17, 299]] = [-1, V, 1 << 30]
    out, st = gpu_gather(to_dev(W), ids)
    ref, bad = oracle.gather(W, ids)
    assert bad == 3 and st == emb.EMB_DEV_ID_OUT_OF_RANGE
    assert np.array_equal(out.view(np.uint32), ref.view(np.uint32))


def test_gather_empty():
    W = to_dev(np.ones((4, 4), np.float32))
    out = emb.gather(W, to_dev(np.zeros(0, np.int32)))
    torch.cuda.synchronize()
    assert out.shape == (0, 4)


# -------------------------------------------------------------------- coalesce
@pytest.mark.parametrize("law,V,T,D", [
    ("zipf", 1000, 512, 64),         # the tiny workload's shape
    ("zipf", 5000, 2048, 8),         # the most tokens of the one-workgroup path
    ("zipf", 5000, 3072, 8),         # exactly three sort tiles
    ("zipf", 5000, 2049, 3),         # two whole sort tiles and one key, scalar width path
    ("uniform", 1 << 20, 10000, 16),  # 20 key bits: three passes of 7 bits
    ("zipf", 32768, 25000, 65),      # odd width (scalar path), many chunks
    ("zipf", 300, 4001, 256),        # very heavy duplication; 9 key bits: one 9-bit pass
    ("uniform", 50, 33, 1),          # one chunk + 1, D = 1
    ("zipf", 1, 777, 4),             # V = 1: every key 0 (one pass), one segment over 25 chunks
    ("uniform", 5_000_000, 9000, 8),  # 23 key bits: three 8-bit passes
    ("uniform", (1 << 31) - 1, 5000, 4),  # 31 key bits: four passes
    ("zipf", 65535, 12000, 16),      # 16 key bits: two 8-bit passes
    ("zipf", 65537, 12000, 16),      # 17 key bits: two 9-bit passes
    ("uniform", (1 << 22) - 1, 20000, 4),  # 22 key bits
    ("uniform", 1 << 25, 20000, 4),  # 25 key bits: three 9-bit passes (9, 9, 7)
    ("uniform", (1 << 27) - 1, 9000, 4),  # 27 key bits: three 9-bit passes
    # batches of at most 2048 tokens (the one-workgroup path): four 8-bit passes in LDS, one
    # segment of all 2048 tokens, a hot row over many of them, a single token
    ("uniform", (1 << 31) - 1, 2000, 4),
    ("zipf", 1, 2048, 4),
    ("zipf", 300, 1999, 256),
    ("uniform", 7, 1, 5),
    # the largest batch of 1024-key sort tiles, and the smallest of 1536-key tiles (ragged: 21 whole
    # tiles and 513 keys)
    ("uniform", 1 << 20, 32768, 4),
    ("zipf", 1 << 20, 32769, 4),
    # 1536-key tiles with 9-bit digits: 17 key bits (two passes), 26 key bits (three passes), one
    # and a ragged tail of 1535 keys
    ("zipf", 65537, 49151, 8),
    ("uniform", (1 << 26) - 3, 40000, 4),
    # more than 1024 reduction workgroups: the head counts are scanned once by their own kernel
    ("zipf", 1 << 20, 200000, 8),
    ("uniform", 1 << 18, 131073, 4),
    # two million tokens: 1366 sort tiles to look back over, 16384 reduction workgroups
    ("uniform", 1 << 22, 1 << 21, 4),
    ("zipf", 1 << 20, (1 << 21) + 77, 4),
])
def test_coalesce_parity_fp32(law, V, T, D):
    ids = ids_for(law, V + T + D, T, V)
    G = grads_for(V + T, T, D)
    check_coalesce(ids, G, V)


@pytest.mark.parametrize("V,T,D", [(262144, 16384, 1024), (1000, 3000, 12), (1000, 3000, 10), (1000, 2000, 12),
                                   (1000, 2048, 16)])
def test_coalesce_parity_bf16(V, T, D):
    ids = ids_for("zipf", V + T, T, V, 1.0)
    G = grads_for(V + D, T, D, 0.01, bf16=True)
    _, _, r = check_coalesce(ids, G, V, bf16=True)
    assert r <= tolerance.RTOL_F32  # identical bf16 inputs: the fp32 bar holds too


def test_coalesce_hot_row_spans_many_chunks():
    # one id takes ~60% of 20000 tokens: ~375 chunk pieces in one segment
    T, V, D = 20000, 5000, 256
    ids = ids_for("zipf", 77, T, V, 2.5)
    G = grads_for(78, T, D, 0.01)
    check_coalesce(ids, G, V)


@pytest.mark.parametrize("seed,n_runs,bad_frac,D,bf16", [(1, 300, 0.0, 64, False), (2, 300, 0.0, 64, False),
                                                         (3, 250, 0.01, 64, False), (4, 40, 0.0, 64, False),
                                                         (5, 80, 0.0, 1024, False), (6, 120, 0.0, 256, True),
                                                         (7, 480, 0.0, 129, False), (8, 320, 0.0, 1024, False)])
def test_coalesce_runs_around_chunk_and_workgroup_boundaries(seed, n_runs, bad_frac, D, bf16):
    # ids that cross chunk boundaries inside a reduction workgroup are summed there, ids that
    # cross workgroups in pieces: every placement of a run's ends against both boundaries (with
    # rows of 1024 floats the columns are split over several workgroups per token range; the last
    # two cases leave each workgroup two column blocks in turn, scalar and float4)
    V = 1 << 16
    ids = runs_ids(seed, n_runs, V, bad_frac)
    G = grads_for(seed + 10, ids.size, D, 0.01, bf16=bf16)
    check_coalesce(ids, G, V, bf16=bf16)


def test_coalesce_all_one_id():
    T, D = 5000, 64
    check_coalesce(np.full(T, 7, np.int32), grads_for(3, T, D), 10)


def test_coalesce_all_distinct_is_a_permutation():
    V, T, D = 100000, 6000, 32
    ids = np.random.default_rng(4).permutation(V)[:T].astype(np.int32)
    G = grads_for(5, T, D)
    gpu, orc, _ = check_coalesce(ids, G, V)
    assert np.array_equal(gpu["uniq_grad"].view(np.uint32), G[np.argsort(ids)].view(np.uint32))


def test_coalesce_out_of_range_ids_are_left_out():
    V, T, D = 1000, 3000, 16
    ids = ids_for("zipf", 9, T, V)
    ids[::97] = -3
    ids[5::101] = V + 5
    check_coalesce(ids, grads_for(9, T, D), V)


def test_coalesce_all_ids_invalid():
    gpu = gpu_coalesce(np.full(100, -1, np.int32), grads_for(1, 100, 4), 50)
    assert gpu["U"] == 0 and gpu["seg_offsets"].tolist() == [0]
    assert gpu["status"] == emb.EMB_DEV_ID_OUT_OF_RANGE


def test_coalesce_empty_batch():
    gpu = gpu_coalesce(np.zeros(0, np.int32), np.zeros((0, 8), np.float32), 50)
    assert gpu["U"] == 0 and gpu["seg_offsets"].tolist() == [0] and gpu["status"] == 0


def test_coalesce_misaligned_gradient_rows_use_scalar_path():
    V, T, D = 2000, 3000, 64
    ids = ids_for("zipf", 11, T, V)
    G = grads_for(11, T, D)
    buf = torch.zeros(T * D + 1, dtype=torch.float32, device="cuda")
    buf[1:] = to_dev(G.reshape(-1))
    check_coalesce(ids, G, V, grad_dev=buf[1:].view(T, D))


def test_coalesce_is_bitwise_deterministic():
    V, T, D = 1 << 20, 65536, 256
    ids = ids_for("zipf", 52, T, V, 1.3)
    G = to_dev(grads_for(52, T, D, 0.01))
    a = gpu_coalesce(ids, None, V, grad_dev=G)
    b = gpu_coalesce(ids, None, V, grad_dev=G)
    assert a["U"] == b["U"]
    assert np.array_equal(a["uniq_grad"].view(np.uint32), b["uniq_grad"].view(np.uint32))


# ------------------------------------------------------------------------ pack
@pytest.mark.parametrize("P,rule", [(1, "mod"), (2, "mod"), (7, "range"), (16, "mod"), (1024, "mod"),
                                    (1024, "range"), (5, "rand")])
def test_pack_parity(P, rule):
    V, T, D = 50000, 9000, 20
    ids = ids_for("zipf", P, T, V, 1.05)
    G = grads_for(P + 1, T, D)
    gpu, _, _ = check_coalesce(ids, G, V)
    if rule == "mod":
        own = gen.owner_mod(V, P)
    elif rule == "range":
        own = gen.owner_range(V, P)
    else:
        own = np.random.default_rng(P).integers(0, P, V).astype(np.int32)
    check_pack(gpu["dev"], gpu["U"], own, P)


def test_pack_drops_rows_with_bad_owner():
    V, T, D, P = 500, 2000, 4, 4
    ids = ids_for("uniform", 3, T, V)
    gpu, _, _ = check_coalesce(ids, grads_for(3, T, D), V)
    own = gen.owner_mod(V, P)
    own[10] = 9
    own[11] = -2
    uid, _, ug, nu = gpu["dev"]
    st = emb.new_status()
    send_ids, send_rows, counts, offs = emb.pack_by_owner(uid, ug, nu, to_dev(own), P, dev_status=st)
    torch.cuda.synchronize()
    orc = oracle.pack_by_owner(host(uid[:gpu["U"]]), host(ug[:gpu["U"]]), own, P)
    n = int(offs[P].item())
    assert np.array_equal(host(send_ids[:n]), orc["send_ids"])
    assert np.array_equal(host(offs), orc["send_offsets"])
    assert int(st.item()) == emb.EMB_DEV_OWNER_OUT_OF_RANGE


def test_pack_empty():
    uid = torch.zeros(0, dtype=torch.int32, device="cuda")
    ug = torch.zeros((0, 4), dtype=torch.float32, device="cuda")
    nu = torch.zeros(1, dtype=torch.int32, device="cuda")
    own = to_dev(gen.owner_mod(10, 3))
    _, _, counts, offs = emb.pack_by_owner(uid, ug, nu, own, 3)
    torch.cuda.synchronize()
    assert host(counts).tolist() == [0, 0, 0] and host(offs).tolist() == [0, 0, 0, 0]


# ------------------------------------------------------------------------ adam
@pytest.mark.parametrize("D", [3, 64, 256])
def test_adam_parity_multi_step_by_shard(D):
    V, T, P = 20000, 6000, 4
    W0 = gen.normal_f32(gen.stream_key(D, 0, gen.PURPOSE_WEIGHTS), V * D).reshape(V, D)
    state = [to_dev(W0), torch.zeros((V, D), device="cuda"), torch.zeros((V, D), device="cuda")]
    own = gen.owner_range(V, P)
    for step in range(1, 4):
        ids = ids_for("zipf", 100 * D + step, T, V, 1.0)
        gpu, _, _ = check_coalesce(ids, grads_for(step, T, D, 0.01), V)
        pk = check_pack(gpu["dev"], gpu["U"], own, P)
        for s in range(P):  # each simulated owner applies its own block
            check_adam(state, pk["dev"], P, s, s + 1, HP, step)


@pytest.mark.parametrize("D", [1, 4, 64, 256, 1024])
def test_adam_eps_regime(D):
    """Gradients where the placement of eps decides the update (|g| near eps / sqrt(1 - b2^t)), zero
    gradients and whole zero rows, over three steps on the same rows, some rows skipped at step 2
    (lazy moments): each call against the oracle on the GPU's own pre-call state, W, m, v and the
    update W_after - W_before on its own scale (Sec. 5.7; Kingma & Ba, Algorithm 1)."""
    print(f"adam eps regime D={D}", flush=True)
    rng = np.random.default_rng(D)
    V, n = 3000, 700
    W0 = rng.normal(0.0, 1.0, (V, D)).astype(np.float32)
    state = [to_dev(W0), torch.zeros((V, D), device="cuda"), torch.zeros((V, D), device="cuda")]
    rows = np.sort(rng.choice(V, n, replace=False)).astype(np.int32)
    for step in (1, 2, 3):
        ids = rows if step != 2 else rows[::2]
        g = eps_regime_grads(rng, ids.size, D)
        pack = (to_dev(ids), to_dev(g), None, to_dev(np.array([0, ids.size], np.int32)))
        check_adam(state, pack, 1, 0, 1, HP, step)


@pytest.mark.parametrize("cap,n,D", [(1, 1, 4096), (3, 3, 4096), (2, 2, 8192), (5, 3, 9001), (7, 5, 2048),
                                     (4, 4, 16384), (16384, 4522, 1024), (300, 1, 4096), (50, 49, 1)])
def test_adam_few_wide_rows(cap, n, D):
    """Row capacities of a few rows with rows of many column steps (waves share a row's columns,
    never more sharing waves than the launch has), and the 4.5k rows of 4 KB of the translation
    workload."""
    print(f"adam few wide rows cap={cap} n={n} D={D}", flush=True)
    V = max(64, 2 * cap)
    W0 = gen.normal_f32(gen.stream_key(D, cap, gen.PURPOSE_WEIGHTS), V * D).reshape(V, D)
    state = [to_dev(W0), torch.zeros((V, D), device="cuda"), torch.zeros((V, D), device="cuda")]
    ids = np.sort(np.random.default_rng(cap + D).choice(V, cap, replace=False)).astype(np.int32)
    for step in (1, 2):
        pack = (to_dev(ids), to_dev(grads_for(700 + step, cap, D)), None, to_dev(np.array([0, n], np.int32)))
        check_adam(state, pack, 1, 0, 1, HP, step)


def test_adam_out_of_range_row_is_skipped_and_flagged():
    V, D = 100, 4
    W = to_dev(np.ones((V, D), np.float32))
    M = torch.zeros((V, D), device="cuda")
    S = torch.zeros((V, D), device="cuda")
    row_ids = to_dev(np.array([3, 200, 5], np.int32))
    rows = to_dev(np.full((3, D), 0.5, np.float32))
    offs = to_dev(np.array([0, 3], np.int32))
    st = emb.new_status()
    emb.sparse_adam_apply(W, M, S, row_ids, rows, offs, 1, 0, 1, **HP, step=1, dev_status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == emb.EMB_DEV_ID_OUT_OF_RANGE
    Wh = host(W)
    assert np.all(Wh[[0, 1, 2, 4, 6]] == 1.0) and np.all(Wh[[3, 5]] < 1.0)


# ----------------------------------------------------------- the whole step
def test_pipeline_on_streams_matches_default_stream():
    """All four calls enqueued on a side stream give the same bits."""
    V, T, D, P = 40000, 12000, 128, 8
    ids = ids_for("zipf", 5, T, V, 1.05)
    G = grads_for(5, T, D, 0.01)
    W0 = gen.normal_f32(gen.stream_key(5, 0, 1), V * D).reshape(V, D)
    own = to_dev(gen.owner_mod(V, P))

    def run(stream):
        with torch.cuda.stream(stream):
            W = to_dev(W0)
            M = torch.zeros_like(W)
            S = torch.zeros_like(W)
            out = emb.gather(W, to_dev(ids))
            uid, seg, ug, nu = emb.grad_coalesce(to_dev(ids), to_dev(G), V)
            send_ids, send_rows, counts, offs = emb.pack_by_owner(uid, ug, nu, own, P)
            emb.sparse_adam_apply(W, M, S, send_ids, send_rows, offs, P, 0, P, **HP, step=1)
        torch.cuda.synchronize()
        return [host(x) for x in (out, W, M, S, send_rows)]

    a = run(torch.cuda.current_stream())
    b = run(torch.cuda.Stream())
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))
