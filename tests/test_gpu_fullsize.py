"""Whole-step parity at the full widths of the GPT-3 Small, XL, 6.7B and 13B steps.

One decoder block (n_layer = 1) with every other size of the configuration
(d_model, heads, MLP width, vocabulary 50257, batch x 2048 tokens): the
GEMM, attention, LayerNorm, embedding and cross-entropy kernels run at the
shapes and tile configurations the benchmark times, and the step swaps (one
node per group, two weight slots).  bf16 with fp32 accumulation against the
fp64 oracle on the same bf16-rounded weights: loss and every gradient tensor
within 2e-2 normwise (max|g - r| / max|r|).
"""
import time

import numpy as np
import pytest

import synthetic
from oracle import gpt
from paper_2403_10504_amd import Session
from paper_2403_10504_amd import atom as A
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

TOL = 2e-2


@pytest.mark.parametrize("name", ["small", "xl", "6.7b", "13b"])
def test_full_width_block_matches_oracle(name):
    cfg = synthetic.CONFIGS[name].with_(n_layer=1)
    t0 = time.time()
    w = synthetic.gen_weights(cfg)
    tok = synthetic.gen_tokens(cfg)
    plan = A.atom_plan_fixed(A.make_config(cfg), list(range(cfg.n_nodes)), 2)
    with Session(cfg, plan=plan) as s:
        s.set_weights(w)
        loss = s.step(tok)
        got = s.grads(A.GRAD_LAST)
    print(f"{name}: GPU step done ({time.time() - t0:.1f} s)", flush=True)
    ref_loss, ref = gpt.step(cfg, w, tok)
    print(f"{name}: oracle done ({time.time() - t0:.1f} s); loss {loss:.6f} vs {ref_loss:.6f}", flush=True)
    assert abs(loss - ref_loss) <= TOL * abs(ref_loss)
    errs = {}
    for node in range(cfg.n_nodes):
        for k, g in got[node].items():
            errs[(node, k)] = U.rel_err(g, ref[node][k])
    print(name, {f"{n}.{k}": f"{e:.1e}" for (n, k), e in errs.items()}, flush=True)
    bad = {k: e for k, e in errs.items() if e > TOL}
    assert not bad, bad
