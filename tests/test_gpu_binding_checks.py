"""The Python binding checks every buffer against the sizes the call will use
and raises before anything is enqueued: a gradient of the wrong dtype or row
count, outputs too small, an owner map shorter than the table, a batch larger
than the pipeline's buffers.  Each case here must raise EmbError (no kernel of
these calls is launched)."""
import numpy as np
import pytest
import torch

import paper_2110_09132_amd as emb
from paper_2110_09132_amd.step import EmbeddingTable, StepPipeline

pytestmark = pytest.mark.gpu

i32, f32 = torch.int32, torch.float32


def z(*shape, dtype=f32):
    return torch.zeros(shape, dtype=dtype, device="cuda")


def ids(n, V=100):
    return torch.arange(n, dtype=i32, device="cuda") % V


def test_gather_checks():
    with pytest.raises(emb.EmbError):
        emb.gather(z(100, 8), ids(10), out=z(9, 8))
    with pytest.raises(emb.EmbError):
        emb.gather(z(100, 8), ids(10), out=z(10, 4))
    with pytest.raises(emb.EmbError):
        emb.gather(z(800), ids(10))  # not [V, D]


def test_coalesce_checks():
    g = z(10, 8)
    with pytest.raises(emb.EmbError):  # bf16 bits in an integer tensor are not a gradient
        emb.grad_coalesce(ids(10), torch.zeros((10, 8), dtype=torch.int16, device="cuda"), 100)
    with pytest.raises(emb.EmbError):
        emb.grad_coalesce(ids(10), z(9, 8), 100)  # a row per token
    with pytest.raises(emb.EmbError):
        emb.grad_coalesce(ids(10), g, 100, out=(z(10, dtype=i32), z(10, dtype=i32), z(10, 8), z(1, dtype=i32)))
    with pytest.raises(emb.EmbError):
        emb.grad_coalesce(ids(10), g, 100, out=(z(10, dtype=i32), z(11, dtype=i32), z(10, 7), z(1, dtype=i32)))
    with pytest.raises(emb.EmbError):
        emb.grad_coalesce_by_owner(ids(10), g, 100, z(99, dtype=i32), 4)  # owners of 99 rows for V = 100
    with pytest.raises(emb.EmbError):
        emb.grad_coalesce_by_owner(ids(10), g, 100, z(100, dtype=i32), 4,
                                   out=(z(10, dtype=i32), z(11, dtype=i32), z(10, 8), z(3, dtype=i32),
                                        z(5, dtype=i32), z(1, dtype=i32)))
    with pytest.raises(emb.EmbError):
        emb.grad_coalesce_split(ids(10), ids(5), g, 100, z(100, dtype=i32), 4,
                                out=(z(10, dtype=i32), z(11, dtype=i32), z(10, 8), z(4, dtype=i32),
                                     z(5, dtype=i32), z(1, dtype=i32)))  # 2P groups


def test_request_exchange_pack_checks():
    with pytest.raises(emb.EmbError):
        emb.lookup_request(ids(10), 100, z(100, dtype=i32), 4,
                           out=(z(10, dtype=i32), z(4, dtype=i32), z(5, dtype=i32), z(1, dtype=i32), z(9, dtype=i32)))
    with pytest.raises(emb.EmbError):
        emb.lookup_request(ids(10), 100, z(50, dtype=i32), 4)
    with pytest.raises(emb.EmbError):
        emb.exchange_simulated(z(4, 10, dtype=i32), z(4, 10, 8), z(4, 4, dtype=i32))  # offsets [P, P + 1]
    with pytest.raises(emb.EmbError):
        emb.exchange_simulated(z(4, 10, dtype=i32), z(4, 9, 8), z(4, 5, dtype=i32))
    with pytest.raises(emb.EmbError):
        emb.receive_merge(z(40, dtype=i32), z(39, 8), z(1, dtype=i32), 100, z(100, dtype=i32), 4)
    with pytest.raises(emb.EmbError):
        emb.pack_by_owner(z(10, dtype=i32), z(10, 8), z(1, dtype=i32), z(100, dtype=i32), 4,
                          out=(z(10, dtype=i32), z(9, 8), z(4, dtype=i32), z(5, dtype=i32)))


def test_column_and_adam_checks():
    with pytest.raises(emb.EmbError):
        emb.pack_by_column(z(10, 8), 2, out=(z(79), z(2, dtype=i32)))
    with pytest.raises(emb.EmbError):
        emb.gather_by_column(z(799), 100, 8, 2, ids(10))
    with pytest.raises(emb.EmbError):
        emb.assemble_by_column(z(80), 10, 8, 2, out=z(9, 8))
    W = z(100, 8)
    with pytest.raises(emb.EmbError):
        emb.sparse_adam_apply(W, z(100, 8), z(99, 8), ids(10), z(10, 8), z(2, dtype=i32), 1, 0, 1, 1e-3, 0.9, 0.999,
                              1e-8, 1)
    with pytest.raises(emb.EmbError):
        emb.sparse_adam_apply(W, z(100, 8), z(100, 8), ids(10), z(9, 8), z(2, dtype=i32), 1, 0, 1, 1e-3, 0.9, 0.999,
                              1e-8, 1)
    with pytest.raises(emb.EmbError):
        emb.sparse_adam_apply(W, z(100, 8), z(100, 8), ids(10), z(10, 8), z(2, dtype=i32), 4, 0, 4, 1e-3, 0.9,
                              0.999, 1e-8, 1)  # offsets [P + 1]


def test_pipeline_checks():
    with pytest.raises(emb.EmbError):
        EmbeddingTable(z(100, 8), z(99, dtype=i32), 4, 64)
    tb = EmbeddingTable(z(100, 8), torch.arange(100, dtype=i32, device="cuda") % 4, 4, 64)
    pipe = StepPipeline([tb], 1e-3, 0.9, 0.999, 1e-8)
    for bad in ((ids(65), z(65, 8)),  # more tokens than the buffers hold
                (ids(10), z(10, 4)),  # rows of the wrong width
                (ids(10), torch.zeros((10, 8), dtype=torch.int16, device="cuda")),  # not a gradient dtype
                (ids(10).to(torch.int64), z(10, 8))):
        with pytest.raises(emb.EmbError):
            pipe.step([bad], 1)
    with pytest.raises(emb.EmbError):
        pipe.step([], 1)
    assert pipe.count == 0  # nothing was enqueued
    pipe.step([(ids(10), z(10, 8))], 1)  # a good step still runs
    pipe.finish()
    torch.cuda.synchronize()
    assert np.all(np.isfinite(tb.W.cpu().numpy()))
