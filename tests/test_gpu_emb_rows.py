"""Row-sparse embedding transfers (atom_set_embedding_rows) on the GPU.

A step reads only the rows of wte its tokens name and only those rows of the
wte gradient are nonzero, so with the option on the swap-in of group 0 copies
just the step's distinct rows and its swap-out just their gradients.  The
results must be bitwise those of whole-row transfers: every loss, the fp32
host accumulators and the last step's gradients (node 0's spread back to full
rows), for sequential and pipelined steps, with reloads in the backward,
several micro-batches and group 0 holding more than the embedding; the bytes
saved must be exactly the rows no token names.
"""
import numpy as np
import pytest

import synthetic
from oracle import gpt
from paper_2403_10504_amd import Session
from paper_2403_10504_amd import atom as A
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

TINY = synthetic.CONFIGS["tiny"]


def tokens_for(cfg, n):
    return np.stack([synthetic.gen_tokens(cfg, seed=300 + s) for s in range(n)])


def distinct_rows(cfg, tok):
    """Distinct input ids of one step's tokens [accum][batch][seq_len + 1]."""
    return len(np.unique(tok[..., :-1]))


def run(cfg, plan, tok, rows, pipelined):
    with Session(cfg, plan=plan) as s:
        s.load_weights()
        s.set_embedding_rows(rows)
        losses = s.steps(tok) if pipelined else np.array([s.step(t) for t in tok], np.float32)
        st = s.stats()
        return np.asarray(losses, np.float32), s.grads(A.GRAD_ACC), s.grads(A.GRAD_LAST), st


def assert_same(a, b):
    for node, (ga, gb) in enumerate(zip(a, b)):
        for name in ga:
            assert np.array_equal(ga[name], gb[name]), (node, name)


CASES = {
    # one node per group, two slots: group 0 is loaded again in the backward
    "f32_singletons_k2": (TINY.with_(n_layer=3), lambda n: list(range(n)), 2),
    # bf16, two micro-batches (fp32 accumulation slot), three slots
    "bf16_accum2_k3": (TINY.with_(dtype="bf16", accum=2, n_layer=3), lambda n: list(range(n)), 3),
    # fp32, three micro-batches (the gradient slot accumulates in place)
    "f32_accum3_k2": (TINY.with_(accum=3, n_layer=2), lambda n: list(range(n)), 2),
    # the whole model in one group: wte is followed by every other tensor
    "f32_resident": (TINY.with_(n_layer=2), lambda n: [n - 1], 1),
    # groups of two nodes: group 0 is the embedding and the first block
    "bf16_pairs_all_slots": (TINY.with_(dtype="bf16", n_layer=4), lambda n: [1, 3, 5], 3),
    # gradient copies lagging across the step boundary (seven gradient slots)
    "bf16_singletons_k2_g7": (TINY.with_(dtype="bf16", n_layer=3), lambda n: list(range(n)), 2, 7),
}


@pytest.mark.parametrize("pipelined", [False, True], ids=["sequential", "pipelined"])
@pytest.mark.parametrize("case", sorted(CASES))
def test_row_sparse_embedding_equals_whole_rows(case, pipelined):
    cfg, last_fn, k, *gs = CASES[case]
    n = cfg.n_layer + 2
    last = last_fn(n)
    if last[-1] != n - 1:
        last = last + [n - 1]
    plan = A.atom_plan_fixed(A.make_config(cfg), last, k, *gs)
    tok = tokens_for(cfg, 3)
    print(case, "pipelined" if pipelined else "sequential", flush=True)
    l_full, acc_full, last_full, st_full = run(cfg, plan, tok, False, pipelined)
    l_rows, acc_rows, last_rows, st_rows = run(cfg, plan, tok, True, pipelined)
    assert np.array_equal(l_full, l_rows), (l_full, l_rows)
    assert_same(acc_full, acc_rows)
    assert_same(last_full, last_rows)
    # exactly the rows no token of a step names stay on the host, each way
    # (the stats are the last call's: every step pipelined, or the last one)
    row = cfg.d_model * (2 if cfg.dtype == "bf16" else 4)
    unused = sum(cfg.vocab - distinct_rows(cfg, t) for t in (tok if pipelined else tok[-1:])) * row
    assert unused > 0
    assert st_full.d2h_bytes - st_rows.d2h_bytes == unused
    saved_in = st_full.h2d_bytes - st_rows.h2d_bytes
    loads_of_group0 = saved_in // unused
    assert saved_in == loads_of_group0 * unused and loads_of_group0 in (1, 2), (saved_in, unused)
    assert st_full.swap_ins == st_rows.swap_ins and st_full.swap_outs == st_rows.swap_outs


def test_every_id_used_and_oracle_parity():
    """A vocabulary every step uses in full (no row saved), and a bf16 step
    with the option on against the fp64 oracle (2e-2, normwise per tensor)."""
    cfg = TINY.with_(dtype="bf16", vocab=16)
    plan = A.atom_plan_fixed(A.make_config(cfg), list(range(cfg.n_layer + 2)), 2)
    tok = tokens_for(cfg, 1)
    assert distinct_rows(cfg, tok[0]) == cfg.vocab
    l_full, acc_full, last_full, st_full = run(cfg, plan, tok, False, False)
    l_rows, acc_rows, last_rows, st_rows = run(cfg, plan, tok, True, False)
    assert np.array_equal(l_full, l_rows)
    assert_same(last_full, last_rows)
    assert st_full.h2d_bytes == st_rows.h2d_bytes and st_full.d2h_bytes == st_rows.d2h_bytes
    ref_loss, ref = gpt.step(cfg, synthetic.gen_weights(cfg), tok[0])
    assert abs(float(l_rows[0]) - ref_loss) <= 2e-2 * abs(ref_loss), (l_rows[0], ref_loss)
    bad = {(node, name): U.rel_err(g, ref[node][name]) for node in range(cfg.n_nodes)
           for name, g in last_rows[node].items()}
    assert all(v <= 2e-2 for v in bad.values()), bad


def test_manual_calls_with_row_sparse_embedding():
    cfg = TINY.with_(n_layer=2)
    n = cfg.n_nodes
    plan = A.atom_plan_fixed(A.make_config(cfg), list(range(n)), 4)
    tok = synthetic.gen_tokens(cfg, seed=77)
    ref_loss, _, ref_last, _ = run(cfg, plan, tok[None], False, False)
    with Session(cfg, plan=plan) as s:
        s.load_weights()
        s.set_embedding_rows(True)
        ctx = s.ctx
        A.atom_set_tokens(ctx, tok)
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
    assert_same(ref_last, got)


def test_row_sparse_embedding_and_retention_exclude_each_other():
    cfg = TINY.with_(n_layer=2)
    plan = A.atom_plan_fixed(A.make_config(cfg), list(range(cfg.n_nodes)), cfg.n_nodes)
    with Session(cfg, plan=plan) as s:
        s.set_retention(True)
        with pytest.raises(A.AtomError) as e:
            s.set_embedding_rows(True)
        assert e.value.status == A.ATOM_ESTATE
        s.set_retention(False)
        s.set_embedding_rows(True)
        with pytest.raises(A.AtomError) as e:
            s.set_retention(True)
        assert e.value.status == A.ATOM_ESTATE
        s.set_embedding_rows(False)
        s.set_retention(True)
