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


def _raw(s, which):
    """Raw bytes of every node's host buffer `which` (bitwise comparisons)."""
    import ctypes

    out = []
    for node in range(s.n_nodes):
        ptr, nbytes = A.atom_host_tensor(s.ctx, node, which)
        out.append(ctypes.string_at(ptr, nbytes))
    return out


# Section III-E / V-B: the update of a global batch applied group by group as
# each group's last gradients are accumulated (atom_optimizer_arm) must equal
# the update applied after the call (atom_optimizer_step), bit for bit: the
# host model, the fp32 master weights, both moments and the zeroed
# accumulators, and the next global batch's losses.  Plans: one group per
# node in two weight slots and the minimum of two gradient slots (the backward
# waits on the copies out, so updates run while later groups still compute),
# and a two-group plan; one and three steps per call; C = 2 micro-batches.
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n_steps,accum,plan_kind", [(1, 1, "per_node"), (3, 1, "per_node"), (2, 2, "two_groups")])
def test_armed_update_equals_update_after_the_call(dtype, n_steps, accum, plan_kind):
    cfg = TINY.with_(n_layer=3, dtype=dtype, accum=accum)
    n = cfg.n_nodes
    c = A.make_config(cfg)
    if plan_kind == "per_node":
        plan = A.atom_plan_fixed(c, list(range(n)), 2, 2)
    else:
        plan = A.atom_plan_fixed(c, [1, n - 1], 2, 2)
    toks = [np.stack([synthetic.gen_tokens(cfg, seed=900 + 7 * b + s) for s in range(n_steps)]) for b in range(3)]
    hp = dict(beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1)
    with Session(cfg, plan=plan) as ref, Session(cfg, plan=plan) as fused:
        for s in (ref, fused):
            s.load_weights()
            A.atom_optimizer_init(s.ctx)
        for b, tok in enumerate(toks, start=1):
            lr = 1e-3 * b
            l_ref = ref.steps(tok)
            A.atom_optimizer_step(ref.ctx, lr, 1.0 / n_steps, b, **hp)
            A.atom_optimizer_arm(fused.ctx, lr, 1.0 / n_steps, b, **hp)
            l_fused = fused.steps(tok)
            st = fused.stats()
            assert st.updated_groups == len(plan.groups()), (b, st.updated_groups)
            assert st.host_update_s > 0
            assert np.array_equal(l_ref, l_fused), (b, l_ref, l_fused)
            for which in (A.WEIGHTS, A.GRAD_ACC, A.MASTER, A.MOMENT1, A.MOMENT2):
                for node, (x, y) in enumerate(zip(_raw(ref, which), _raw(fused, which))):
                    assert x == y, (b, which, node)
            assert not any(np.any(a[k]) for a in fused.grads(A.GRAD_ACC) for k in a)
        # the arm is one-shot: a plain call afterwards updates nothing
        fused.steps(toks[0])
        assert fused.stats().updated_groups == 0


def test_arm_requires_optimizer_state():
    cfg = TINY.with_(n_layer=1)
    plan = A.atom_plan_fixed(A.make_config(cfg), list(range(cfg.n_nodes)), 2)
    with Session(cfg, plan=plan) as s:
        with pytest.raises(A.AtomError) as e:
            A.atom_optimizer_arm(s.ctx, 1e-3, 1.0, 1)
        assert e.value.status == A.ATOM_ESTATE
        with pytest.raises(A.AtomError):
            A.atom_host_tensor(s.ctx, 0, A.MASTER)
