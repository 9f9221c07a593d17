"""Host AdamW after a global batch (atom_optimizer_step), against the oracle.

A global batch of two steps on the GPU fills the fp32 host accumulators; the
library's AdamW (fp32 on the host) then updates the master weights and
refreshes the working copy.  The oracle applies AdamW in fp64 to the same
accumulated gradients (read back from the host, so the comparison measures the
optimizer alone).  Tolerance: fp32 rounding of an update of size about lr,
relative to the weights (max-norm), 1e-6; the bf16 copy equals the master
rounded to nearest even, within one bf16 ulp near rounding ties and a few
fp32 ulp of the largest weight for weights the update drives through zero.
A second global batch checks the moments carry over and the accumulators
were zeroed.
"""
import numpy as np
import pytest

import synthetic
from oracle import adamw as O
from paper_2403_10504_amd import Session
from paper_2403_10504_amd import atom as A
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

TINY = synthetic.CONFIGS["tiny"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_adamw_after_global_batch_matches_oracle(dtype):
    cfg = TINY.with_(n_layer=2, dtype=dtype)
    n = cfg.n_nodes
    plan = A.atom_plan_fixed(A.make_config(cfg), list(range(n)), 2)
    toks = [np.stack([synthetic.gen_tokens(cfg, seed=700 + 2 * b + s) for s in range(2)]) for b in range(2)]
    # the library takes fp32 hyper-parameters: the oracle gets the same values
    hp = {k: float(np.float32(v)) for k, v in dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1).items()}
    with Session(cfg, plan=plan) as s:
        s.load_weights()
        params = [{k: v.astype(np.float64) for k, v in p.items()} for p in s.weights()]
        A.atom_optimizer_init(s.ctx)
        state = None
        for b, tok in enumerate(toks, start=1):
            s.steps(tok)
            g = s.grads(A.GRAD_ACC)
            g = [{k: v.astype(np.float64) / 2 for k, v in p.items()} for p in g]
            A.atom_optimizer_step(s.ctx, hp["lr"], 0.5, b, hp["beta1"], hp["beta2"], hp["eps"], hp["weight_decay"])
            params, state = O.model_step(params, g, state, b, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"],
                                         hp["weight_decay"])
            got = s.weights()
            acc = s.grads(A.GRAD_ACC)
            assert all(not np.any(acc[i][k]) for i in range(n) for k in acc[i])  # accumulators zeroed
            for i in range(n):
                for k, ref in params[i].items():
                    if dtype == "f32":
                        assert U.rel_err(got[i][k], ref) < 1e-6, (b, i, k)
                    else:
                        want = U.rep(ref.astype(np.float32), "bf16")
                        # the master is fp32: its bf16 rounding may differ from the fp64
                        # oracle's by one bf16 ulp where the value sits near a rounding tie,
                        # and a weight that the update drives through zero keeps the fp32
                        # master's absolute rounding error (a few ulp of the largest weight)
                        d = np.abs(got[i][k].astype(np.float64) - want)
                        bound = 2.0 ** -7 * np.abs(want) + 4 * 2.0 ** -24 * np.max(np.abs(ref))
                        w = np.unravel_index(np.argmax(d - bound), d.shape)
                        assert np.all(d <= bound), (b, i, k, w, got[i][k][w], want[w], ref[w])
                        assert np.mean(got[i][k] == want) > 0.99, (b, i, k)
