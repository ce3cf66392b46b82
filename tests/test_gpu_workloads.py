"""Every workload at its full size, in the launch configuration the benchmark
uses, chained over training steps: gather, coalesce, pack and the per-owner
Adam updates of each step, each call compared with the oracle on identical
inputs (the GPU's state before the call), as the step of one GPU's share of
sparse embedding training (Sec. 4.1.1: lookup, gradient exchange payload,
update; Sec. 4.2.2: coalescing)."""
import numpy as np
import pytest
import torch

import oracle
import tolerance
from gpu_helpers import check_adam, check_coalesce, check_pack, gpu_gather, host, to_dev
from workloads import configs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", list(configs.WORKLOADS))
def test_workload_parity(name):
    wl = configs.WORKLOADS[name]
    hp = dict(lr=wl.lr, beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps)
    for spec in wl.tables:
        print(f"[{name}] V={spec.V} D={spec.D} T={spec.T} P={spec.P} seed={spec.seed}", flush=True)
        W = to_dev(configs.make_weights(spec))
        state = [W, torch.zeros_like(W), torch.zeros_like(W)]
        own = configs.row_owner(spec)
        bf16 = spec.grad_dtype == "bf16"
        for step in range(1, wl.steps + 1):
            ids, G = configs.make_batch(spec, step)
            # gather reads the table as left by the previous step's update
            out, st = gpu_gather(W, ids)
            assert st == 0
            rows = np.unique(ids)
            Wrows = host(W[torch.from_numpy(rows.astype(np.int64)).to(W.device)])
            ref, _ = oracle.gather(Wrows, np.searchsorted(rows, ids).astype(np.int32))
            assert np.array_equal(out.view(np.uint32), ref.view(np.uint32))
            gpu, orc, r = check_coalesce(ids, G, spec.V, bf16=bf16,
                                         rtol=tolerance.RTOL_BF16 if bf16 else tolerance.RTOL_F32)
            pk = check_pack(gpu["dev"], gpu["U"], own, spec.P)
            worst = 0.0
            for s in range(spec.P):
                worst = max(worst, check_adam(state, pk["dev"], spec.P, s, s + 1, hp, step))
            print(f"  step {step}: U={gpu['U']} grad_err={r:.2e} adam_err={worst:.2e} "
                  f"counts={pk['send_counts'].tolist()[:8]}", flush=True)
        del W, state
        torch.cuda.empty_cache()
