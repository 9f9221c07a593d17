"""Whole-step parity on the GPU, through the C ABI (atom_step and the per-group calls).

* fp32 mode matches the fp64 oracle within 1e-4 (normwise per tensor and
  for the loss), bf16 mode within 2e-2 (the oracle consumes the same
  bf16-rounded weights, so the error measured is compute error);
* a swapped plan (one node per group, two weight slots, so groups are reloaded
  in the backward) gives bit-identical loss and gradients to a plan that keeps
  everything resident;
* two runs of the same step are bit-identical; accumulators sum steps.
"""
import math

import numpy as np
import pytest

import synthetic
from oracle import gpt
from paper_2403_10504_amd import Session
from paper_2403_10504_amd import atom as A
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

TINY = synthetic.CONFIGS["tiny"]


def run_step(cfg, plan=None, weights=None, tokens=None, steps=1):
    with Session(cfg, plan=plan) as s:
        if weights is None:
            s.load_weights()
        else:
            s.set_weights(weights)
        tok = synthetic.gen_tokens(cfg) if tokens is None else tokens
        losses = [s.step(tok) for _ in range(steps)]
        return losses, s.grads(A.GRAD_LAST), s.grads(A.GRAD_ACC), s.stats()


def swapped_plan(cfg, k=2):
    n = cfg.n_layer + 2
    return A.atom_plan_fixed(A.make_config(cfg), list(range(n)), k)


def resident_plan(cfg):
    n = cfg.n_layer + 2
    return A.atom_plan_fixed(A.make_config(cfg), [n - 1], 1)


def compare_to_oracle(cfg, tol, tokens=None, weights=None):
    w = synthetic.gen_weights(cfg) if weights is None else weights
    tok = synthetic.gen_tokens(cfg) if tokens is None else tokens
    loss, grads, _, _ = run_step(cfg, plan=swapped_plan(cfg), weights=w, tokens=tok)
    ref_loss, ref = gpt.step(cfg, w, tok)
    assert abs(loss[0] - ref_loss) <= tol * abs(ref_loss), (loss[0], ref_loss)
    worst = {}
    for node in range(cfg.n_nodes):
        for name, g in grads[node].items():
            worst[(node, name)] = U.rel_err(g, ref[node][name])
    bad = {k: v for k, v in worst.items() if v > tol}
    assert not bad, bad
    return worst


def test_tiny_fp32_matches_oracle():
    compare_to_oracle(TINY, 1e-4)


def test_tiny_bf16_matches_oracle():
    compare_to_oracle(TINY.with_(dtype="bf16"), 2e-2)


@pytest.mark.parametrize("dtype,tol", [("f32", 1e-4), ("bf16", 2e-2)])
def test_accumulated_step_matches_oracle(dtype, tol):
    cfg = TINY.with_(dtype=dtype, accum=2, n_layer=1)
    compare_to_oracle(cfg, tol)


def test_ragged_sequence_and_vocab_match_oracle():
    # T = 100 (not a tile multiple), V = 1000 (not a multiple of 128), d_head 128
    cfg = synthetic.Config("ragged", 1, 256, 2, 512, 1000, 100, 2, 1, "f32")
    compare_to_oracle(cfg, 1e-4)


def test_single_token_sequences():
    cfg = synthetic.Config("t1", 1, 128, 2, 256, 64, 1, 8, 1, "f32")
    compare_to_oracle(cfg, 1e-4)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_swap_and_no_swap_are_bit_exact(dtype):
    cfg = TINY.with_(dtype=dtype, n_layer=3)
    l_res, g_res, _, st_res = run_step(cfg, plan=resident_plan(cfg))
    l_sw, g_sw, _, st_sw = run_step(cfg, plan=swapped_plan(cfg))
    assert st_sw.h2d_bytes > st_res.h2d_bytes  # the swapped plan really reloaded
    assert l_res == l_sw
    for node in range(cfg.n_nodes):
        for name in g_res[node]:
            assert np.array_equal(g_res[node][name], g_sw[node][name]), (node, name)


def test_planner_budget_of_one_block_swaps_and_matches():
    cfg = TINY
    c = A.make_config(cfg)
    _, blk = A.atom_node_layout(c, 1)
    _, emb = A.atom_node_layout(c, 0)
    _, head = A.atom_node_layout(c, cfg.n_layer + 1)
    slot = max(blk, emb, head)
    budget = A.atom_reserve_bytes(c) + 4 * slot  # two weight slots + two gradient slots
    plan = A.atom_plan_partition(c, budget)
    assert plan.n_slots == 2 and plan.n_groups > 2
    l1, g1, _, st = run_step(cfg, plan=plan)
    assert st.swap_ins > plan.n_groups
    l0, g0, _, _ = run_step(cfg, plan=resident_plan(cfg))
    assert l0 == l1
    for node in range(cfg.n_nodes):
        for name in g0[node]:
            assert np.array_equal(g0[node][name], g1[node][name]), (node, name)


def test_repeat_steps_bit_identical_and_accumulate():
    cfg = TINY.with_(dtype="bf16")
    losses, last, acc, _ = run_step(cfg, plan=swapped_plan(cfg), steps=3)
    assert losses[0] == losses[1] == losses[2]
    for node in range(cfg.n_nodes):
        for name in last[node]:
            np.testing.assert_allclose(acc[node][name], 3 * last[node][name], rtol=1e-6, atol=1e-12)


def test_loss_near_ln_vocab_at_init():
    losses, _, _, _ = run_step(TINY.with_(dtype="bf16"))
    assert abs(losses[0] - (math.log(1024) + 0.5 * 0.02 ** 2 * 256)) < 0.05


def test_manual_calls_enforce_order():
    cfg = TINY
    with Session(cfg, plan=swapped_plan(cfg)) as s:
        s.load_weights()
        ctx = s.ctx
        tok = synthetic.gen_tokens(cfg)
        A.atom_set_tokens(ctx, tok)
        with pytest.raises(A.AtomError) as e:
            A.atom_block_fwd(ctx, 0, 0)  # group 0 not swapped in
        assert e.value.status == A.ATOM_ESTATE
        A.atom_swap_in(ctx, 0)
        with pytest.raises(A.AtomError) as e:
            A.atom_swap_in(ctx, 0)
        assert e.value.status == A.ATOM_ESTATE
        with pytest.raises(A.AtomError) as e:
            A.atom_block_fwd(ctx, 1, 0)  # input of node 1 not computed (and not resident)
        assert e.value.status == A.ATOM_ESTATE
        A.atom_block_fwd(ctx, 0, 0)
        with pytest.raises(A.AtomError) as e:
            A.atom_block_bwd(ctx, 0, 0)  # gradient of node 0's output not computed
        assert e.value.status == A.ATOM_ESTATE
        with pytest.raises(A.AtomError) as e:
            A.atom_swap_out(ctx, 0)
        assert e.value.status == A.ATOM_ESTATE
        with pytest.raises(A.AtomError) as e:
            A.atom_set_tokens(ctx, np.full_like(tok, cfg.vocab))
        assert e.value.status == A.ATOM_EINVAL
        A.atom_sync(ctx)


def test_manual_schedule_equals_atom_step():
    cfg = TINY.with_(n_layer=2)
    plan = swapped_plan(cfg, k=4)
    tok = synthetic.gen_tokens(cfg)
    ref_loss, ref_g, _, _ = run_step(cfg, plan=plan, tokens=tok)
    with Session(cfg, plan=plan) as s:
        s.load_weights()
        ctx = s.ctx
        A.atom_set_tokens(ctx, tok)
        n = cfg.n_nodes
        for g in range(n):
            A.atom_swap_in(ctx, g)
        for node in range(n):
            A.atom_block_fwd(ctx, node, 0)
        for node in range(n - 1, -1, -1):
            if node <= cfg.n_layer:
                A.atom_block_bwd(ctx, node, 0)
            A.atom_swap_out(ctx, node)
        loss = A.atom_sync(ctx)
        got = s.grads(A.GRAD_LAST)
    assert loss == ref_loss[0]
    for node in range(n):
        for name in got[node]:
            assert np.array_equal(got[node][name], ref_g[node][name]), (node, name)


def test_arena_is_the_device_budget():
    """The context holds exactly the plan's arena on the device; the step
    itself allocates nothing more through torch."""
    import gc

    t = U.torch()
    cfg = TINY.with_(dtype="bf16")
    gc.collect()  # sessions of earlier tests that are garbage now
    t.cuda.synchronize()
    base = t.cuda.memory_allocated()
    plan = swapped_plan(cfg)
    with Session(cfg, plan=plan) as s:
        held = t.cuda.memory_allocated() - base
        assert plan.arena_bytes <= held <= plan.arena_bytes + (4 << 20), (held, plan.arena_bytes)
        t.cuda.reset_peak_memory_stats()
        s.load_weights()
        s.step(synthetic.gen_tokens(cfg))
        t.cuda.synchronize()
        assert t.cuda.max_memory_allocated() - base <= held + (4 << 20)


def test_measured_costs_plan_gives_same_step():
    """Node costs measured on the GPU (the per-layer profile the planner
    consumes) are positive, loading time grows with bytes, and a plan made from
    them runs the step bitwise like the analytic plan (a plan moves data, it
    changes no arithmetic)."""
    cfg = TINY.with_(n_layer=4, dtype="bf16")
    tok = synthetic.gen_tokens(cfg)
    c = A.make_config(cfg)
    with Session(cfg, plan=swapped_plan(cfg)) as s:
        s.load_weights()
        costs = A.atom_profile_nodes(s.ctx, c, tok)
        profiled = s.grads(A.GRAD_LAST)
    n = cfg.n_nodes
    assert len(costs) == n
    analytic_costs = A.atom_node_costs(c)
    N = cfg.batch * cfg.seq_len
    for i, x in enumerate(costs):
        assert x.weight_bytes > 0 and x.t_load > 0 and x.t_store > 0 and x.t_fwd > 0
        assert (x.t_bwd > 0) == (i <= cfg.n_layer)
        # working memory: how far the node's kernels wrote into the workspace,
        # within what the arena carves for it (the embedding uses none)
        assert x.mem_bytes <= analytic_costs[i].mem_bytes, (i, x.mem_bytes, analytic_costs[i].mem_bytes)
        if i == 0:
            assert x.mem_bytes == 0
        else:
            assert x.mem_bytes >= analytic_costs[i].mem_bytes // 2, (i, x.mem_bytes)
        assert x.cut_bytes == (N * cfg.d_model * 4 if i <= cfg.n_layer else 4)
    # the profiled step (workspace filled with a marker before every node)
    # computed exactly what an ordinary step computes
    _, last, _, _ = run_step(cfg, plan=swapped_plan(cfg), tokens=tok)
    for node in range(n):
        for name in last[node]:
            assert np.array_equal(profiled[node][name], last[node][name]), (node, name)
    budget = A.atom_reserve_bytes(c) + 8 * costs[1].weight_bytes
    measured = A.atom_plan_partition(c, budget, costs)
    analytic = A.atom_plan_partition(c, budget)
    l1, g1, _, _ = run_step(cfg, plan=measured, tokens=tok)
    l2, g2, _, _ = run_step(cfg, plan=analytic, tokens=tok)
    assert l1 == l2
    for node in range(n):
        for name in g1[node]:
            assert np.array_equal(g1[node][name], g2[node][name]), (node, name)
