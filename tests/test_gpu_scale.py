"""The benchmarked schedules at production widths, through the C ABI.

The step the benchmark times runs many groups in many weight slots, lets
gradient copies lag the backward through up to 16 gradient slots, keeps the
13B block inputs in a host ring, reloads XL groups in the backward, keeps
GPT-3 Small's one resident group on the device across the steps of a call,
and pipelines the steps of a global batch.  None of that changes arithmetic: the
same kernels run in the same order on the same weights, so every loss, the
fp32 host accumulators and the last step's gradients must be bitwise those of

* the same plan run one atom_step call at a time, and
* a plan that keeps the whole model resident in one group (no swapping inside
  the step), with device checkpoints.

Each case uses the full width of its GPT-3 configuration (d_model, heads, MLP,
vocabulary 50257, batch x 2048 tokens) with fewer blocks, so the kernels run
at the benchmark's shapes and tile configurations and the schedule has enough
groups for slots, gradient slots and the checkpoint ring to wrap.  Host
buffers are compared through per-node SHA-256 digests of their raw bytes.
"""
import time

import numpy as np
import pytest

import synthetic
from paper_2403_10504_amd import Session
from paper_2403_10504_amd import atom as A
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

N_STEPS = 3


def tokens_for(cfg, n):
    return np.stack([synthetic.gen_tokens(cfg, seed=synthetic.TOKEN_SEED + 1000 + s) for s in range(n)])


def say(msg):
    print(f"[scale] {msg}", flush=True)


def run(cfg, plan, tok, pipelined, label, rows=False, retain=False):
    t0 = time.time()
    say(f"{label}: {plan.n_groups} groups, {plan.n_slots} slots, {plan.n_gslots} gradient slots, "
        f"arena {plan.arena_bytes / 1e9:.2f} GB, {'pipelined' if pipelined else 'sequential'}"
        f"{', embedding rows only' if rows else ''}{', weights retained' if retain else ''}")
    with Session(cfg, plan=plan) as s:
        s.load_weights()
        s.set_embedding_rows(rows)
        s.set_retention(retain)
        if pipelined:
            losses = s.steps(tok)
        else:
            losses = np.array([s.step(t) for t in tok], np.float32)
        st = s.stats()
        acc = U.host_digests(s, A.GRAD_ACC)
        last = U.host_digests(s, A.GRAD_LAST)
    say(f"{label}: losses {losses.tolist()} ({time.time() - t0:.1f} s)")
    return np.asarray(losses, np.float32), acc, last, st


def assert_same(ref, got, what):
    l_ref, acc_ref, last_ref, _ = ref
    l_got, acc_got, last_got, _ = got
    assert np.array_equal(l_ref, l_got), (what, l_ref, l_got)
    bad_acc = [n for n, (a, b) in enumerate(zip(acc_ref, acc_got)) if a != b]
    bad_last = [n for n, (a, b) in enumerate(zip(last_ref, last_got)) if a != b]
    assert not bad_acc and not bad_last, (what, "accumulators differ at nodes", bad_acc, "last step at", bad_last)


def resident(cfg):
    """One group holding every node (one weight slot), device checkpoints."""
    dev = cfg.with_(ckpt_host=False)
    return dev, A.atom_plan_fixed(A.make_config(dev), [dev.n_nodes - 1], 1, 2)


def test_6p7b_width_bench_plan_pipelined():
    # the 6.7B benchmark plan's structure (a slot per one-node group, 14
    # gradient slots, so copies out lag the backward across the step
    # boundary), and what atom_plan_partition makes of the same budget
    cfg = synthetic.CONFIGS["6.7b"].with_(n_layer=4)
    c = A.make_config(cfg)
    bench = A.atom_plan_fixed(c, list(range(cfg.n_nodes)), cfg.n_nodes, 14)
    budget = bench.arena_bytes
    planned = A.atom_plan_partition(c, budget)
    say(f"6.7B width plan for {budget / 1e9:.2f} GB: {planned.groups()}, {planned.n_slots} slots, "
        f"{planned.n_gslots} gradient slots")
    assert planned.n_slots == planned.n_groups and planned.arena_bytes <= budget
    tok = tokens_for(cfg, N_STEPS)
    pipe = run(cfg, bench, tok, True, "6.7B width, bench plan")
    seq = run(cfg, bench, tok, False, "6.7B width, bench plan")
    assert_same(seq, pipe, "pipelined vs sequential")
    assert pipe[3].h2d_bytes == N_STEPS * seq[3].h2d_bytes
    assert len(set(pipe[0].tolist())) == N_STEPS
    rcfg, rplan = resident(cfg)
    res = run(rcfg, rplan, tok, False, "6.7B width, resident")
    assert_same(res, pipe, "swapped vs resident")
    got = run(cfg, planned, tok, True, "6.7B width, planned")
    assert_same(res, got, "planned vs resident")
    # the bench line's default: only the embedding rows a step uses cross the link
    rows = run(cfg, bench, tok, True, "6.7B width, bench plan", rows=True)
    assert_same(pipe, rows, "embedding rows only vs whole rows")
    unused = sum(cfg.vocab - len(np.unique(t[..., :-1])) for t in tok) * cfg.d_model * 2
    assert pipe[3].h2d_bytes - rows[3].h2d_bytes == unused
    assert pipe[3].d2h_bytes - rows[3].d2h_bytes == unused


def test_13b_width_host_checkpoint_ring_evicts():
    # six blocks: block inputs 0..2 leave the four-entry device ring for the
    # host in the forward and come back before their backward; eight one-node
    # groups in six slots reload two groups in the backward (the 13B plan's
    # shape: more groups than slots, two gradient slots)
    cfg = synthetic.CONFIGS["13b"].with_(n_layer=6)
    assert cfg.ckpt_host
    c = A.make_config(cfg)
    plan = A.atom_plan_fixed(c, list(range(cfg.n_nodes)), 6, 2)
    expect_ckpt = (cfg.n_layer + 1 - 4) * cfg.batch * cfg.seq_len * cfg.d_model * 4
    tok = tokens_for(cfg, N_STEPS)
    pipe = run(cfg, plan, tok, True, "13B width, host checkpoints")
    seq = run(cfg, plan, tok, False, "13B width, host checkpoints")
    assert_same(seq, pipe, "pipelined vs sequential (host checkpoints)")
    weights = sum(A.atom_node_layout(c, n)[1] for n in range(cfg.n_nodes))
    reload = sum(A.atom_node_layout(c, n)[1] for n in range(cfg.n_nodes - 6))
    assert seq[3].h2d_bytes == weights + reload + expect_ckpt, (seq[3].h2d_bytes, weights, reload, expect_ckpt)
    assert seq[3].d2h_bytes == weights + expect_ckpt
    dcfg = cfg.with_(ckpt_host=False)
    dev = run(dcfg, A.atom_plan_fixed(A.make_config(dcfg), list(range(cfg.n_nodes)), 6, 2), tok, True,
              "13B width, device checkpoints")
    assert_same(dev, pipe, "host vs device checkpoints")
    rcfg, rplan = resident(cfg)
    res = run(rcfg, rplan, tok, False, "13B width, resident")
    assert_same(res, pipe, "swapped vs resident")
    # only the embedding rows a step uses, with group 0 reloaded in the backward
    rows = run(cfg, plan, tok, True, "13B width, host checkpoints", rows=True)
    assert_same(pipe, rows, "embedding rows only vs whole rows (host checkpoints)")
    unused = sum(cfg.vocab - len(np.unique(t[..., :-1])) for t in tok) * cfg.d_model * 2
    assert pipe[3].d2h_bytes - rows[3].d2h_bytes == unused
    assert pipe[3].h2d_bytes - rows[3].h2d_bytes == 2 * unused  # loaded in the forward and the backward


def test_xl_width_planned_with_backward_reloads():
    # a budget under which the planner keeps fewer slots than groups, so the
    # backward reloads the first groups (the XL benchmark plan does the same
    # under 8 GB)
    cfg = synthetic.CONFIGS["xl"].with_(n_layer=6)
    c = A.make_config(cfg)
    per_node = A.atom_plan_fixed(c, list(range(cfg.n_nodes)), 2, 2)
    budget = per_node.reserve_bytes + 6 * per_node.slot_bytes
    plan = A.atom_plan_partition(c, budget)
    say(f"XL width plan: {plan.groups()}, {plan.n_slots} slots")
    assert plan.n_slots < plan.n_groups, (plan.n_slots, plan.n_groups)
    tok = tokens_for(cfg, N_STEPS)
    pipe = run(cfg, plan, tok, True, "XL width, planned")
    seq = run(cfg, plan, tok, False, "XL width, planned")
    assert_same(seq, pipe, "pipelined vs sequential")
    assert seq[3].h2d_bytes > sum(A.atom_node_layout(c, n)[1] for n in range(cfg.n_nodes))  # reloads happened
    rcfg, rplan = resident(cfg)
    res = run(rcfg, rplan, tok, False, "XL width, resident")
    assert_same(res, pipe, "swapped vs resident")


def test_small_width_resident_retained():
    # GPT-3 Small's bench default: no device budget, so the planner makes the
    # whole model one group in one slot, and the weights stay on the device
    # across the steps of the call (loaded once instead of once per step);
    # d_h = 64 kernels at the full width
    cfg = synthetic.CONFIGS["small"].with_(n_layer=3)
    c = A.make_config(cfg)
    plan = A.atom_plan_partition(c, 1 << 50)
    assert plan.n_groups == 1 and plan.n_slots == 1, plan.groups()
    tok = tokens_for(cfg, N_STEPS)
    ret = run(cfg, plan, tok, True, "Small width, resident", retain=True)
    pipe = run(cfg, plan, tok, True, "Small width, resident")
    seq = run(cfg, plan, tok, False, "Small width, resident")
    assert_same(seq, pipe, "pipelined vs sequential")
    assert_same(pipe, ret, "retained vs loaded every step")
    weights = sum(A.atom_node_layout(c, n)[1] for n in range(cfg.n_nodes))
    assert pipe[3].h2d_bytes == N_STEPS * weights and ret[3].h2d_bytes == weights
    assert ret[3].d2h_bytes == pipe[3].d2h_bytes == N_STEPS * weights
