"""C-ABI library tests that need no GPU: symbols, validation, layout, planner.

The planner (atom_plan_search, C++) is compared with the brute-force oracle
(oracle/plan.py) on random cost graphs: same partition, slot count, byte
counts, overlap flag and bit-identical predicted times.
"""
import os
import re

import numpy as np
import pytest

from oracle import plan as OP
from paper_2403_10504_amd import atom as A
from synthetic import CONFIGS, Config, param_specs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    names = []
    for h in ("atom.h", "atom_kernels.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names += re.findall(r"\b(atom_\w+)\s*\(", src)
    return sorted(set(names))


def test_library_exports_every_declared_function():
    lib = A.lib()
    declared = header_functions()
    assert len(declared) >= 32
    for name in declared:
        assert hasattr(lib, name), name
    assert set(declared) == set(A.EXPORTED)


def test_version_and_status_strings():
    assert "gfx950" in A.atom_version()
    assert A.status_string(A.ATOM_ENOPLAN).startswith("no partition")


TINY = CONFIGS["tiny"]


def test_config_validation():
    bad = [TINY.with_(n_head=3), TINY.with_(d_model=200, n_head=2), TINY.with_(n_layer=0),
           TINY.with_(dtype="f16")]
    for cfg in bad:
        c = A.make_config(cfg)
        if cfg.dtype == "f16":
            c.dtype = 7
        with pytest.raises(A.AtomError) as e:
            A.atom_plan_partition(c, 1 << 40)
        assert e.value.status == A.ATOM_EINVAL


def test_node_layout_matches_parameter_list():
    for cfg in (TINY, CONFIGS["small"], CONFIGS["6.7b"]):
        c = A.make_config(cfg)
        esz = 2 if cfg.dtype == "bf16" else 4
        for node in (0, 1, cfg.n_layer + 1):
            tens, nbytes = A.atom_node_layout(c, node)
            specs = param_specs(cfg, node)
            assert [t[0] for t in tens] == [s[0] for s in specs]
            for (name, rows, cols, off, tb), (_, shape, _) in zip(tens, specs):
                assert off % 256 == 0
                n = int(np.prod(shape))
                if name == "w_head":
                    vp = (cfg.vocab + 127) // 128 * 128
                    assert (rows, cols) == (vp, cfg.d_model) and tb == vp * cfg.d_model * esz
                else:
                    assert rows * cols == n and tb == n * esz
            assert nbytes % 256 == 0 and nbytes >= tens[-1][3] + tens[-1][4]
    with pytest.raises(A.AtomError):
        A.atom_node_layout(A.make_config(TINY), TINY.n_layer + 2)


def test_reserve_and_partition_fit_budget():
    for name in ("tiny", "small", "xl", "6.7b"):
        cfg = CONFIGS[name]
        c = A.make_config(cfg)
        r = A.atom_reserve_bytes(c)
        budget = cfg.budget_bytes or (1 << 45)
        p = A.atom_plan_partition(c, budget)
        assert p.reserve_bytes == r
        assert p.arena_bytes <= budget
        assert p.arena_bytes == r + p.n_slots * p.slot_bytes + p.n_gslots * p.slot_bytes
        assert p.n_slots >= min(p.n_groups, 2)
        # leftover budget becomes gradient slots, up to the limit
        assert 2 <= p.n_gslots <= A.ATOM_MAX_GSLOTS
        assert p.n_gslots == A.ATOM_MAX_GSLOTS or budget - p.arena_bytes < p.slot_bytes
        # the reserve holds the largest working memory of a node (m_i)
        costs = A.atom_node_costs(c)
        assert p.work_bytes == max(x.mem_bytes for x in costs) > 0
        q = A.atom_plan_search(c, budget, r - p.work_bytes, costs)
        assert q.groups() == p.groups() and q.n_slots == p.n_slots and q.n_gslots == p.n_gslots
        groups = p.groups()
        assert groups[0][0] == 0 and groups[-1][1] == cfg.n_layer + 1


def test_budget_too_small_is_enoplan():
    c = A.make_config(CONFIGS["small"])
    with pytest.raises(A.AtomError) as e:
        A.atom_plan_partition(c, A.atom_reserve_bytes(c) + 1000)
    assert e.value.status == A.ATOM_ENOPLAN


def test_6p7b_plan_keeps_all_weights_resident_under_24gb():
    cfg = CONFIGS["6.7b"]
    p = A.atom_plan_partition(A.make_config(cfg), cfg.budget_bytes)
    assert p.n_slots == p.n_groups
    assert p.h2d_bytes == p.d2h_bytes == p.forced_h2d_bytes


def test_13b_host_checkpoints_plan():
    """13B under 24 GB with block inputs on the host: the weights no longer fit
    (26.2 GB), so groups reload in the backward; every block input the
    four-entry device ring overwrites crosses the link once each way."""
    cfg = CONFIGS["13b"]
    assert cfg.ckpt_host
    c = A.make_config(cfg)
    p = A.atom_plan_partition(c, cfg.budget_bytes)
    assert p.arena_bytes <= cfg.budget_bytes
    assert p.n_slots < p.n_groups
    ck = (cfg.n_layer + 1 - 4) * cfg.accum * cfg.batch * cfg.seq_len * cfg.d_model * 4
    dev = A.make_config(cfg.with_(ckpt_host=False))
    # same partition and slots with device checkpoints would need (L+1-4) more [N][d] fp32 entries
    assert A.atom_reserve_bytes(dev) - A.atom_reserve_bytes(c) == ck
    W = sum(A.atom_node_layout(c, i)[1] for i in range(cfg.n_nodes))
    assert p.d2h_bytes == W + ck
    assert p.h2d_bytes > W + ck  # reloads in the backward
    assert p.forced_h2d_bytes >= W + ck


def test_plan_fixed():
    c = A.make_config(TINY)
    n = TINY.n_layer + 2
    p = A.atom_plan_fixed(c, list(range(n)), 2)
    assert p.n_groups == n and p.n_slots == 2
    assert p.groups() == [(i, i) for i in range(n)]
    one = A.atom_plan_fixed(c, [n - 1], 1)
    assert one.n_groups == 1 and one.slot_bytes > p.slot_bytes
    for last, k in (([1, 1, n - 1], 2), ([n - 2], 1), (list(range(n)), 1), (list(range(n)), n + 1)):
        with pytest.raises(A.AtomError):
            A.atom_plan_fixed(c, last, k)


def random_costs(rng, n, tiers=True):
    out = []
    for i in range(n):
        w = int(rng.integers(1, 6)) * 256 if tiers else int(rng.integers(1, 10 ** 6))
        out.append(dict(weight_bytes=w, mem_bytes=int(rng.integers(0, 4)) * 128, cut_bytes=int(rng.choice([64, 64, 96])),
                        t_fwd=float(rng.choice([0.5, 1.0, 1.5, 2.0])), t_bwd=float(rng.choice([1.0, 2.0, 3.0])),
                        t_load=float(rng.choice([0.25, 1.0, 2.0, 4.0])), t_store=float(rng.choice([0.5, 1.0, 3.0]))))
    out[-1]["t_bwd"] = 0.0  # the head's backward runs inside its forward
    return out


def ck_times(cfg, costs):
    """Host-checkpoint copy times the C planner derives: one node's block input
    (all micro-batches) at the costs' average link rates."""
    if not cfg.ckpt_host:
        return {}
    ckb = float(cfg.accum * cfg.batch * cfg.seq_len * cfg.d_model * 4)
    w = sum(x["weight_bytes"] for x in costs)
    tl = sum(x["t_load"] for x in costs)
    ts = sum(x["t_store"] for x in costs)
    return dict(n_layer=cfg.n_layer, ck_host=True, t_ck_in=ckb * (tl / w), t_ck_out=ckb * (ts / w))


def _compare(c, cfg, costs, budget, base, want, strict=False, duplex=A.ATOM_DEFAULT_DUPLEX):
    try:
        got = A.atom_plan_search(c, budget, base, costs, strict=strict, duplex=duplex)
    except A.AtomError as e:
        assert e.status == A.ATOM_ENOPLAN and want is None
        return None
    assert want is not None
    assert got.groups() == want["groups"]
    assert (got.n_slots, got.n_gslots) == (want["n_slots"], want["n_gslots"])
    assert got.slot_bytes == want["slot_bytes"]
    assert got.arena_bytes == want["arena_bytes"]
    assert got.cut_bytes == want["cut_bytes"]
    assert got.rule == (A.ATOM_RULE_PAPER if want["rule"] == "paper" else A.ATOM_RULE_TIME)
    # bit-identical: the same sums, maxima and event arithmetic
    assert got.pred_step_s == want["pred_step_s"]
    assert got.pred_first_step_s == want["pred_first_step_s"]
    assert got.pred_fwd_s == want["pred_fwd_s"]
    assert bool(got.overlap_ok) == want["overlap_ok"]
    ck = cfg.accum * cfg.batch * cfg.seq_len * cfg.d_model * 4 * max(0, cfg.n_layer + 1 - 4) if cfg.ckpt_host else 0
    assert (got.h2d_bytes, got.d2h_bytes) == (want["h2d_bytes"] + ck, want["d2h_bytes"] + ck)
    return got


@pytest.mark.parametrize("seed", range(64))
def test_planner_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(3, 11))
    costs = random_costs(rng, n)
    accum = int(rng.choice([1, 2, 4]))
    dtype = int(rng.choice([OP.F32, OP.BF16]))
    ck_host = n >= 6 and bool(rng.integers(0, 2))
    strict = bool(rng.integers(0, 2))
    duplex = float(rng.choice([0.5, 0.85, 1.0]))
    base = int(rng.integers(0, 4096))
    total = sum(c["weight_bytes"] for c in costs)
    budget = base + 384 + int(rng.integers(total // 2 + 256, 5 * total // 2 + 1024))
    cfg = TINY.with_(n_layer=n - 2, accum=accum, dtype="bf16" if dtype == OP.BF16 else "f32", ckpt_host=ck_host)
    c = A.make_config(cfg)
    want = OP.brute_force(costs, budget, base, accum, dtype, strict=strict, duplex=duplex, **ck_times(cfg, costs))
    _compare(c, cfg, costs, budget, base, want, strict, duplex)


def test_planner_rules_through_the_abi():
    # the oracle's hand cases, through the C planner
    cfg = TINY.with_(n_layer=2)
    c = A.make_config(cfg)
    def uni(tf, tb, tu, ts, cut=7):
        out = [dict(weight_bytes=100, mem_bytes=0, cut_bytes=cut, t_fwd=tf, t_bwd=tb, t_load=tu, t_store=ts)
               for _ in range(4)]
        out[3]["t_bwd"] = 0.0
        return out
    # minimum cut among overlapping partitions beats the faster one
    got = A.atom_plan_search(c, 4 * 200, 0, uni(2.0, 4.0, 1.0, 1.0))
    assert got.groups() == [(0, 1), (2, 3)] and got.rule == A.ATOM_RULE_PAPER and got.overlap_ok
    # nothing overlaps: strict mode has no plan, the fallback is the fastest
    slow = uni(0.1, 0.2, 5.0, 5.0)
    with pytest.raises(A.AtomError) as e:
        A.atom_plan_search(c, 600, 0, slow, strict=True)
    assert e.value.status == A.ATOM_ENOPLAN
    got = A.atom_plan_search(c, 600, 0, slow)
    assert got.rule == A.ATOM_RULE_TIME and not got.overlap_ok


@pytest.mark.parametrize("seed", range(6))
def test_planner_structured_search_for_long_chains(seed):
    rng = np.random.default_rng(100 + seed)
    L = int(rng.integers(15, 30))
    blk = dict(weight_bytes=4096, mem_bytes=1024, cut_bytes=64, t_fwd=1.0, t_bwd=3.0,
               t_load=float(rng.choice([0.5, 2.0, 8.0])), t_store=2.0)
    emb = dict(weight_bytes=int(rng.choice([2048, 8192])), mem_bytes=0, cut_bytes=64, t_fwd=0.1, t_bwd=0.1,
               t_load=1.0, t_store=1.0)
    head = dict(weight_bytes=int(rng.choice([4096, 12288])), mem_bytes=2048, cut_bytes=4, t_fwd=2.0, t_bwd=0.0,
                t_load=3.0, t_store=3.0)
    costs = [emb] + [dict(blk) for _ in range(L)] + [head]
    base = 10000
    budget = base + 2048 + int(rng.integers(6, 3 * L)) * 4096
    cfg = TINY.with_(n_layer=L)
    c = A.make_config(cfg)
    want = OP.best(OP.structured_candidates(L), costs, budget, base, 1, OP.F32, duplex=A.ATOM_DEFAULT_DUPLEX)
    got = _compare(c, cfg, costs, budget, base, want)
    if got is not None:
        assert got.exhaustive == (L + 2 <= 16)


def test_plan_predict_matches_the_oracle_schedule():
    cfg = CONFIGS["13b"].with_(n_layer=6)
    c = A.make_config(cfg)
    plan = A.atom_plan_fixed(c, list(range(cfg.n_nodes)), 6, 3)
    costs = [x.as_dict() for x in A.atom_node_costs(c)]
    for n_steps, duplex in ((1, 0.85), (5, 0.5), (3, 1.0)):
        ends, fwd = A.atom_plan_predict(c, plan, costs, duplex, n_steps)
        t_fwd, want = OP.simulate(plan.groups(), costs, 1, 6, 3, n_steps, duplex, **ck_times(cfg, costs))
        assert ends == want and fwd == t_fwd
    # retention (a slot per group): only step 0 loads
    full = A.atom_plan_fixed(c, list(range(cfg.n_nodes)), cfg.n_nodes, 3)
    for n_steps, duplex in ((1, 0.85), (4, 0.5), (3, 1.0)):
        ends, fwd = A.atom_plan_predict(c, full, costs, duplex, n_steps, retain=True)
        t_fwd, want = OP.simulate(full.groups(), costs, 1, cfg.n_nodes, 3, n_steps, duplex, retain=True,
                                  **ck_times(cfg, costs))
        assert ends == want and fwd == t_fwd
        assert ends[-1] <= A.atom_plan_predict(c, full, costs, duplex, n_steps)[0][-1] * (1 + 1e-12)
    # 6 slots for 8 groups: every group is loaded again each step, as without retention
    assert A.atom_plan_predict(c, plan, costs, 0.5, 3, retain=True) == A.atom_plan_predict(c, plan, costs, 0.5, 3)
    # the plan's own predictions are the default-duplex ones
    ends, _ = A.atom_plan_predict(c, plan, None, 0.0, OP.PIPE_STEPS)
    assert plan.pred_step_s == (ends[-1] - ends[-3]) / 2.0
    assert plan.pred_first_step_s == A.atom_plan_predict(c, plan, None, 0.0, 1)[0][0]


def test_ctx_create_rejects_bad_arguments_without_gpu():
    c = A.make_config(TINY)
    p = A.atom_plan_partition(c, 1 << 40)
    with pytest.raises(A.AtomError) as e:
        A.atom_ctx_create(c, p, 0, p.arena_bytes, 1)
    assert e.value.status == A.ATOM_EINVAL
    with pytest.raises(A.AtomError) as e:
        A.atom_ctx_create(c, p, 4096, p.arena_bytes, 0)  # no compute stream
    assert e.value.status == A.ATOM_EINVAL
    p2 = A.atom_plan_partition(c, 1 << 40)
    p2.n_slots = 0
    with pytest.raises(A.AtomError) as e:
        A.atom_ctx_create(c, p2, 4096, p.arena_bytes, 1)
    assert e.value.status == A.ATOM_EINVAL
    with pytest.raises(A.AtomError) as e:
        A.atom_ctx_create(c, p, 4096, p.arena_bytes - 256, 1)
    assert e.value.status == A.ATOM_EBUDGET


def test_context_calls_reject_a_null_context_without_gpu():
    for call in (lambda: A.atom_set_retention(None, True), lambda: A.atom_optimizer_init(None),
                 lambda: A.atom_set_embedding_rows(None, True)):
        with pytest.raises(A.AtomError) as e:
            call()
        assert e.value.status == A.ATOM_EINVAL


def test_kernel_entry_points_validate_before_launch():
    # dtype and null-pointer checks return EINVAL without touching a device
    with pytest.raises(A.AtomError) as e:
        A.atom_k_gemm(5, 1, 1, 0, 16, 16, 16, 4096, 16, 4096, 16, 4096, 16)
    assert e.value.status == A.ATOM_EINVAL
    with pytest.raises(A.AtomError) as e:
        A.atom_k_gemm(A.ATOM_BF16, 1, 1, A.ATOM_EPI_BIAS, 16, 16, 16, 4096, 16, 4096, 16, 4096, 16)
    assert e.value.status == A.ATOM_EINVAL
    with pytest.raises(A.AtomError) as e:  # K not a multiple of 8
        A.atom_k_gemm(A.ATOM_BF16, 1, 1, 0, 16, 16, 12, 4096, 16, 4096, 16, 4096, 16)
    assert e.value.status == A.ATOM_EINVAL
    with pytest.raises(A.AtomError) as e:  # head dim 96 unsupported
        A.atom_k_attn_fwd(A.ATOM_BF16, 4096, 4096, 4096, 1, 16, 1, 96)
    assert e.value.status == A.ATOM_EINVAL
    assert A.atom_k_layernorm_bwd_part_floats(100, 64) == 7 * 2 * 64
    assert A.atom_k_colsum_part_floats(130, 10) == 9 * 10  # blocks of 16 rows
