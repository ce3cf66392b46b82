"""The receiver side of the exchange, simulated for P workers on one device:
the block transpose (emb_exchange_simulated) moves exactly each worker's
owner blocks to their receivers (checked bit for bit against a numpy
transpose of the GPU's own send buffers), and the merge (emb_receive_merge)
equals the oracle's owner-major pack of the coalesce of all workers' tokens
together: ids, counts and offsets bit-exact, rows within the summation bound."""
import numpy as np
import pytest
import torch

import oracle
import paper_2110_09132_amd as emb
import tolerance
from gpu_helpers import host, to_dev
from workloads import gen

pytestmark = pytest.mark.gpu


def worker_batch(law, seed, T, V, D, s=1.1):
    key = gen.stream_key(seed, 0, gen.PURPOSE_IDS)
    ids = gen.uniform_ids(key, T, V) if law == "uniform" else gen.zipf_ids(key, T, V, s)
    g = gen.normal_f32(gen.stream_key(seed, 0, gen.PURPOSE_GRADS), T * D).reshape(T, D)
    return ids, g


def run_workers(batches, V, D, own_np, P, cap):
    """Each worker's owner-major coalesce, written side by side into [P, cap] buffers."""
    send_ids = torch.full((P, cap), -7, dtype=torch.int32, device="cuda")
    send_rows = torch.zeros((P, cap, D), dtype=torch.float32, device="cuda")
    send_offs = torch.zeros((P, P + 1), dtype=torch.int32, device="cuda")
    own = to_dev(own_np)
    for w, (ids, g) in enumerate(batches):
        T = ids.size
        seg = torch.empty(T + 1, dtype=torch.int32, device="cuda")
        cnt = torch.empty(P, dtype=torch.int32, device="cuda")
        nu = torch.empty(1, dtype=torch.int32, device="cuda")
        emb.grad_coalesce_by_owner(to_dev(ids.astype(np.int32)), to_dev(g), V, own, P,
                                   out=(send_ids[w, :T], seg, send_rows[w, :T], cnt, send_offs[w], nu))
    torch.cuda.synchronize()
    return send_ids, send_rows, send_offs


def check_exchange(send_ids, send_rows, send_offs, P, cap):
    st = emb.new_status()
    recv_ids, recv_rows, recv_offs, total = emb.exchange_simulated(send_ids, send_rows, send_offs)
    torch.cuda.synchronize()
    sid, srows, soffs = host(send_ids), host(send_rows), host(send_offs)
    exp_ids, exp_rows, exp_offs = [], [], np.zeros((P, P + 1), np.int64)
    pos = 0
    for p in range(P):
        for w in range(P):
            exp_offs[p, w] = pos
            a, b = soffs[w, p], soffs[w, p + 1]
            exp_ids.append(sid[w, a:b])
            exp_rows.append(srows[w, a:b])
            pos += b - a
        exp_offs[p, P] = pos
    n = int(total.item())
    assert n == pos
    assert np.array_equal(host(recv_offs), exp_offs)
    assert np.array_equal(host(recv_ids)[:n], np.concatenate(exp_ids))
    assert np.array_equal(host(recv_rows)[:n].view(np.uint32), np.concatenate(exp_rows).view(np.uint32))
    assert int(st.item()) == 0
    return recv_ids, recv_rows, total


@pytest.mark.parametrize("P,law,D,rule,T", [(1, "zipf", 16, "mod", 3000), (2, "uniform", 64, "mod", 3000),
                                            (4, "zipf", 3, "range", 3000), (16, "uniform", 32, "mod", 3000),
                                            (7, "zipf", 8, "rand", 3000),
                                            (2, "zipf", 16, "mod", 1000)])  # merge of 1903 of 2000 rows: one workgroup
def test_exchange_then_merge_equals_coalesce_of_all_tokens(P, law, D, rule, T):
    V = 20000
    sizes = [T - 97 * w for w in range(P)]  # ragged worker batches
    batches = [worker_batch(law, 900 + 31 * P + w, sizes[w], V, D) for w in range(P)]
    own_np = {"mod": gen.owner_mod(V, P), "range": gen.owner_range(V, P),
              "rand": np.random.default_rng(P).integers(0, P, V).astype(np.int32)}[rule]
    cap = max(sizes)
    send_ids, send_rows, send_offs = run_workers(batches, V, D, own_np, P, cap)
    recv_ids, recv_rows, total = check_exchange(send_ids, send_rows, send_offs, P, cap)
    st = emb.new_status()
    merged = emb.receive_merge(recv_ids, recv_rows, total, V, to_dev(own_np), P, dev_status=st)
    torch.cuda.synchronize()
    m_ids, m_seg, m_rows, m_cnt, m_offs, m_nu = merged
    U = int(m_nu.item())
    assert int(st.item()) == 0
    # the oracle: coalesce of all workers' tokens together, packed by owner
    all_ids = np.concatenate([b[0] for b in batches])
    all_g = np.concatenate([b[1] for b in batches])
    orc = oracle.coalesce(all_ids, all_g, V)
    pk = oracle.pack_by_owner(orc["uniq_ids"], orc["uniq_grad"], own_np, P)
    assert U == int(pk["send_offsets"][P])
    assert np.array_equal(host(m_ids)[:U], pk["send_ids"])
    assert np.array_equal(host(m_cnt), pk["send_counts"])
    assert np.array_equal(host(m_offs), pk["send_offsets"])
    idx = np.searchsorted(orc["uniq_ids"], pk["send_ids"])
    tolerance.assert_grad_close(host(m_rows)[:U], orc["sum_f64"][idx], orc["absum"][idx], tolerance.RTOL_F32)
    # each merged row sums one coalesced row per sender that had the id
    senders = np.zeros(V, np.int64)
    for ids, _ in batches:
        senders[np.unique(ids)] += 1
    assert np.array_equal(np.diff(host(m_seg)[:U + 1]), senders[pk["send_ids"]])


def test_exchange_with_an_empty_worker():
    V, D, P = 5000, 16, 3
    batches = [worker_batch("zipf", 11, 2000, V, D), (np.zeros(0, np.int32), np.zeros((0, D), np.float32)),
               worker_batch("zipf", 12, 1500, V, D)]
    own_np = gen.owner_mod(V, P)
    send_ids, send_rows, send_offs = run_workers(batches, V, D, own_np, P, 2000)
    recv_ids, recv_rows, total = check_exchange(send_ids, send_rows, send_offs, P, 2000)
    merged = emb.receive_merge(recv_ids, recv_rows, total, V, to_dev(own_np), P)
    torch.cuda.synchronize()
    all_ids = np.concatenate([batches[0][0], batches[2][0]])
    orc = oracle.coalesce(all_ids, np.concatenate([batches[0][1], batches[2][1]]), V)
    pk = oracle.pack_by_owner(orc["uniq_ids"], orc["uniq_grad"], own_np, P)
    assert np.array_equal(host(merged[4]), pk["send_offsets"])
    assert np.array_equal(host(merged[0])[:int(merged[5].item())], pk["send_ids"])


def test_merge_of_nothing():
    V, D, P = 100, 4, 2
    recv_ids = torch.zeros(8, dtype=torch.int32, device="cuda")
    recv_rows = torch.zeros((8, D), dtype=torch.float32, device="cuda")
    total = torch.zeros(1, dtype=torch.int32, device="cuda")
    merged = emb.receive_merge(recv_ids, recv_rows, total, V, to_dev(gen.owner_mod(V, P)), P)
    torch.cuda.synchronize()
    assert int(merged[5].item()) == 0 and host(merged[4]).tolist() == [0, 0, 0]


def test_exchange_and_merge_at_the_benchmark_shape():
    """The launch configuration the benchmark times: 16 workers, each the owner-major coalesce of a
    65536-token batch over 2^20 rows of 256 floats (worker w takes batch w mod 8, as there).  The
    merge's ids, counts and offsets bit for bit against the oracle's owner-major pack of the coalesce
    of all 16 batches together; rows sampled within the summation bound."""
    V, D, P, T = 1 << 20, 256, 16, 65536
    print(f"exchange + merge at V={V} D={D} P={P} T={T}", flush=True)
    own_np = gen.owner_mod(V, P)
    base = [worker_batch("uniform", 1500 + b, T, V, D) for b in range(8)]
    batches = [base[w % 8] for w in range(P)]
    send_ids, send_rows, send_offs = run_workers(batches, V, D, own_np, P, T)
    recv_ids, recv_rows, recv_offs, total = emb.exchange_simulated(send_ids, send_rows, send_offs)
    del send_rows
    st = emb.new_status()
    m_ids, m_seg, m_rows, m_cnt, m_offs, m_nu = emb.receive_merge(recv_ids, recv_rows, total, V, to_dev(own_np), P,
                                                                 dev_status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    U = int(m_nu.item())
    all_ids = np.concatenate([b[0] for b in batches])
    all_g = np.concatenate([b[1] for b in batches])
    orc = oracle.coalesce(all_ids, all_g, V)
    del all_g
    pk = oracle.pack_by_owner(orc["uniq_ids"], orc["uniq_grad"], own_np, P)
    assert U == int(pk["send_offsets"][P])
    assert np.array_equal(host(m_ids[:U]), pk["send_ids"])
    assert np.array_equal(host(m_cnt), pk["send_counts"]) and np.array_equal(host(m_offs), pk["send_offsets"])
    sample = np.sort(np.random.default_rng(5).choice(U, 4096, replace=False))
    idx = np.searchsorted(orc["uniq_ids"], pk["send_ids"][sample])
    got = host(m_rows[torch.from_numpy(sample).to(m_rows.device)])
    tolerance.assert_grad_close(got, orc["sum_f64"][idx], orc["absum"][idx], tolerance.RTOL_F32)
