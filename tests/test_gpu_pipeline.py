"""Pipelined steps (atom_steps) on the GPU, through the C ABI.

Several steps of one global batch run back to back with the next step's first
groups swapped in during the current step's backward.  The result must be
bitwise that of the same steps run one call at a time: every loss, the fp32
host accumulators and the last step's gradients; every step must still move
every weight in and every gradient out.
"""
import numpy as np
import pytest

import synthetic
from paper_2403_10504_amd import Session
from paper_2403_10504_amd import atom as A

pytestmark = pytest.mark.gpu

TINY = synthetic.CONFIGS["tiny"]


def tokens_for(cfg, n):
    return np.stack([synthetic.gen_tokens(cfg, seed=100 + s) for s in range(n)])


def plan_for(cfg, last, k, gslots=2):
    return A.atom_plan_fixed(A.make_config(cfg), last, k, gslots)


def sequential(cfg, plan, tok):
    with Session(cfg, plan=plan) as s:
        s.load_weights()
        losses = [s.step(t) for t in tok]
        st = s.stats()
        return np.array(losses, np.float32), s.grads(A.GRAD_ACC), s.grads(A.GRAD_LAST), st


def pipelined(cfg, plan, tok):
    with Session(cfg, plan=plan) as s:
        s.load_weights()
        losses = s.steps(tok)
        st = s.stats()
        return losses, s.grads(A.GRAD_ACC), s.grads(A.GRAD_LAST), st


def assert_same(a, b):
    for node, (ga, gb) in enumerate(zip(a, b)):
        for name in ga:
            assert np.array_equal(ga[name], gb[name]), (node, name)


CASES = {
    # one node per group, two slots: reloads in the backward, G > K
    "f32_singletons_k2": (TINY.with_(n_layer=3), lambda n: list(range(n)), 2),
    # bf16, three slots, two micro-batches (fp32 accumulation slot)
    "bf16_accum2_k3": (TINY.with_(dtype="bf16", accum=2, n_layer=3), lambda n: list(range(n)), 3),
    # everything resident in one group (G = K = 1)
    "f32_resident": (TINY.with_(n_layer=2), lambda n: [n - 1], 1),
    # groups of two nodes, G = K (no reload, every slot handed to the next step)
    "bf16_pairs_all_slots": (TINY.with_(dtype="bf16", n_layer=4), lambda n: [1, 3, 5], 3),
    # odd number of groups with K = 2 (slot order alternates between steps)
    "f32_three_groups_k2": (TINY.with_(n_layer=3), lambda n: [0, 2, 4], 2),
    # more gradient slots than groups per step: copies lag across the step boundary
    "bf16_singletons_k2_g7": (TINY.with_(dtype="bf16", n_layer=3), lambda n: list(range(n)), 2, 7),
    # three gradient slots with five groups (claims wrap unevenly across steps)
    "f32_singletons_k3_g3": (TINY.with_(n_layer=3), lambda n: list(range(n)), 3, 3),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_pipelined_steps_equal_sequential_steps(case):
    cfg, last_fn, k, *gs = CASES[case]
    n = cfg.n_layer + 2
    last = last_fn(n)
    if last[-1] != n - 1:
        last = last + [n - 1]
    plan = plan_for(cfg, last, k, *gs)
    tok = tokens_for(cfg, 3)
    l_seq, acc_seq, last_seq, st_seq = sequential(cfg, plan, tok)
    l_pipe, acc_pipe, last_pipe, st_pipe = pipelined(cfg, plan, tok)
    print(case, l_seq, l_pipe, flush=True)
    assert np.array_equal(l_seq, l_pipe)
    assert len(set(l_seq.tolist())) == 3  # the three steps saw different tokens
    assert_same(acc_seq, acc_pipe)
    assert_same(last_seq, last_pipe)
    # per call: the pipelined call moved three steps' worth of weights and gradients
    assert st_pipe.h2d_bytes == 3 * st_seq.h2d_bytes
    assert st_pipe.d2h_bytes == 3 * st_seq.d2h_bytes
    assert st_pipe.swap_outs == 3 * st_seq.swap_outs


def test_single_step_after_pipelined_call():
    cfg = TINY.with_(n_layer=3)
    plan = plan_for(cfg, list(range(cfg.n_nodes)), 2)
    tok = tokens_for(cfg, 3)
    with Session(cfg, plan=plan) as s:
        s.load_weights()
        s.steps(tok[:2])  # ends with the slots in the odd step's order
        s.zero_grads()
        l_after = s.step(tok[2])
        g_after = s.grads(A.GRAD_ACC)
    with Session(cfg, plan=plan) as s:
        s.load_weights()
        l_fresh = s.step(tok[2])
        g_fresh = s.grads(A.GRAD_ACC)
    assert l_after == l_fresh
    assert_same(g_after, g_fresh)


def test_steps_rejects_bad_count_and_bad_ids():
    cfg = TINY.with_(n_layer=1)
    with Session(cfg) as s:
        s.load_weights()
        tok = tokens_for(cfg, 2)
        with pytest.raises(ValueError):
            A.atom_steps(s.ctx, tok[:0])
        # shapes the C side would read out of bounds are refused by the binding
        with pytest.raises(ValueError):
            s.steps(tok[:, :, :, :-1])
        with pytest.raises(ValueError):
            s.step(tok[0, 0])
        with pytest.raises(ValueError):
            A.atom_step(s.ctx, tok)
        bad = tok.copy()
        bad[1, 0, 0, 0] = cfg.vocab
        with pytest.raises(A.AtomError):
            s.steps(bad)
        # nothing ran: the accumulators are still zero
        assert all(not np.any(g[k]) for g in s.grads(A.GRAD_ACC) for k in g)
        good = s.steps(tok[:1])
    with Session(cfg) as s:
        s.load_weights()
        ref = s.step(tok[0])
    assert good[0] == ref


def test_gradient_slot_count_does_not_change_results():
    cfg = TINY.with_(dtype="bf16", n_layer=3)
    last = list(range(cfg.n_nodes))
    tok = tokens_for(cfg, 2)
    ref = pipelined(cfg, plan_for(cfg, last, 2, 2), tok)
    for gslots in (3, 16):
        plan = plan_for(cfg, last, 2, gslots)
        assert plan.n_gslots == gslots
        got = pipelined(cfg, plan, tok)
        assert np.array_equal(ref[0], got[0])
        assert_same(ref[1], got[1])
    with pytest.raises(A.AtomError):
        plan_for(cfg, last, 2, 1)
    with pytest.raises(A.AtomError):
        plan_for(cfg, last, 2, A.ATOM_MAX_GSLOTS + 1)


def pipelined_retained(cfg, plan, tok, on=True):
    with Session(cfg, plan=plan) as s:
        s.load_weights()
        s.set_retention(on)
        losses = s.steps(tok)
        st = s.stats()
        # a second call loads everything again, and gives the same results
        s.zero_grads()
        again = s.steps(tok)
        st2 = s.stats()
        return losses, s.grads(A.GRAD_ACC), s.grads(A.GRAD_LAST), st, again, st2


RETAIN_CASES = {
    # one node per group, a slot each
    "f32_singletons_all_slots": (TINY.with_(n_layer=3), lambda n: list(range(n)), 5),
    # bf16 pairs, G = K = 3
    "bf16_pairs_all_slots": (TINY.with_(dtype="bf16", n_layer=4), lambda n: [1, 3, 5], 3),
    # bf16, two micro-batches per step (fp32 accumulation slot), G = K = 5
    "bf16_accum2_all_slots": (TINY.with_(dtype="bf16", accum=2, n_layer=3), lambda n: list(range(n)), 5),
    # fewer slots than groups: retention has no effect
    "f32_singletons_k2": (TINY.with_(n_layer=3), lambda n: list(range(n)), 2),
}


@pytest.mark.parametrize("case", sorted(RETAIN_CASES))
def test_retained_weights_equal_reloaded_weights(case):
    cfg, last_fn, k = RETAIN_CASES[case]
    n = cfg.n_nodes
    last = last_fn(n)
    if last[-1] != n - 1:
        last = last + [n - 1]
    plan = plan_for(cfg, last, k)
    tok = tokens_for(cfg, 3)
    l_ref, acc_ref, last_ref, st_ref = pipelined(cfg, plan, tok)
    l_ret, acc_ret, last_ret, st_ret, again, st2 = pipelined_retained(cfg, plan, tok)
    print(case, l_ref, l_ret, st_ref.h2d_bytes, st_ret.h2d_bytes, flush=True)
    assert np.array_equal(l_ref, l_ret)
    assert np.array_equal(l_ref, again)
    assert_same(acc_ref, acc_ret)
    assert_same(last_ref, last_ret)
    assert st_ret.d2h_bytes == st_ref.d2h_bytes  # gradients still leave every step
    assert st_ret.swap_outs == st_ref.swap_outs
    assert st2.h2d_bytes == st_ret.h2d_bytes
    if plan.n_slots >= plan.n_groups:
        # each group loaded once per call instead of once per step
        assert st_ret.h2d_bytes * 3 == st_ref.h2d_bytes
        assert st_ret.swap_ins == plan.n_groups
    else:
        assert st_ret.h2d_bytes == st_ref.h2d_bytes


def test_single_step_after_retained_call():
    cfg = TINY.with_(n_layer=3)
    plan = plan_for(cfg, list(range(cfg.n_nodes)), cfg.n_nodes)
    tok = tokens_for(cfg, 3)
    with Session(cfg, plan=plan) as s:
        s.load_weights()
        s.set_retention(True)
        s.steps(tok[:2])
        s.zero_grads()
        l_after = s.step(tok[2])
        g_after = s.grads(A.GRAD_ACC)
    with Session(cfg, plan=plan) as s:
        s.load_weights()
        l_fresh = s.step(tok[2])
        g_fresh = s.grads(A.GRAD_ACC)
    assert l_after == l_fresh
    assert_same(g_after, g_fresh)
