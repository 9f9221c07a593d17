"""Pins of the planner oracle: enumeration, schedule closed forms, paper sizes."""
import math
import os

import numpy as np
import pytest

from oracle import plan as P
from synthetic import CONFIGS, Config, param_count

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def costs_uniform(n, w=100, tf=1.0, tb=2.0, tu=3.0, ts=3.0):
    return [dict(weight_bytes=w, t_fwd=tf, t_bwd=tb, t_load=tu, t_store=ts) for _ in range(n)]


def test_compositions_are_all_distinct_contiguous_partitions():
    for n in range(1, 9):
        parts = list(P.compositions(n))
        assert len(parts) == 2 ** (n - 1)
        assert len({tuple(p) for p in parts}) == len(parts)
        for p in parts:
            assert p[0][0] == 0 and p[-1][1] == n - 1
            for (a, b), (c, _) in zip(p, p[1:]):
                assert c == b + 1
            assert all(a <= b for a, b in p)


def test_single_group_schedule_is_serial():
    c = costs_uniform(3)
    t_fwd, t_step = P.simulate([(0, 2)], c, accum=2, K=1)
    # load all, compute forward of 2 micro-batches, backward, store all
    assert t_fwd == 9.0 + 2 * 3.0
    assert t_step == 9.0 + 6.0 + 12.0 + 9.0


def test_link_bound_resident_schedule_is_sum_of_transfers():
    c = costs_uniform(5, tf=0.0, tb=0.0, tu=1.5, ts=2.5)
    groups = [(i, i) for i in range(5)]
    t_fwd, t_step = P.simulate(groups, c, accum=1, K=5)
    assert t_fwd == 7.5 and t_step == 7.5 + 12.5


def test_compute_bound_schedule_exposes_only_first_load_and_last_store():
    c = costs_uniform(4, tf=10.0, tb=20.0, tu=1.0, ts=1.0)
    groups = [(i, i) for i in range(4)]
    t_fwd, t_step = P.simulate(groups, c, accum=1, K=4)
    assert t_fwd == 1.0 + 40.0
    assert t_step == 1.0 + 40.0 + 80.0 + 1.0


def test_two_slots_force_reloads_in_backward():
    c = costs_uniform(4, w=10)
    groups = [(i, i) for i in range(4)]
    ok, K, S, arena = P.memory(groups, c, budget=1000 + 4 * 10, reserve=1000, accum=1, dtype=P.BF16)
    assert ok and K == 2 and S == 10 and arena == 1040
    h2d, d2h = P.transfer_bytes(groups, c, K)
    assert h2d == 40 + 20 and d2h == 40


def test_memory_rejects_budget_below_two_slots():
    c = costs_uniform(4, w=10)
    groups = [(i, i) for i in range(4)]
    assert not P.memory(groups, c, budget=1000 + 3 * 10, reserve=1000, accum=1, dtype=P.BF16)[0]
    # a single group needs one weight slot only
    assert P.memory([(0, 3)], c, budget=1000 + 3 * 40, reserve=1000, accum=1, dtype=P.BF16)[0]
    # bf16 with accumulation adds an fp32 slot of 2S
    assert not P.memory(groups, c, budget=1000 + 5 * 10, reserve=1000, accum=2, dtype=P.BF16)[0]
    assert P.memory(groups, c, budget=1000 + 6 * 10, reserve=1000, accum=2, dtype=P.BF16)[0]
    assert P.memory(groups, c, budget=1000 + 4 * 10, reserve=1000, accum=2, dtype=P.F32)[0]


def test_brute_force_prefers_fine_groups_when_link_bound():
    c = costs_uniform(6, tf=0.1, tb=0.2, tu=1.0, ts=1.0)
    best = P.brute_force(c, budget=10 ** 9, reserve=0, accum=1, dtype=P.BF16)
    # link-bound: all loads, then the last group's forward and backward, then
    # all stores; a small last group minimises the exposed compute, and the
    # fewest-groups tie-break then merges everything before it
    assert best["pred_step_s"] == pytest.approx(6.0 + 0.1 + 0.2 + 6.0, abs=1e-12)
    assert best["groups"] == [(0, 4), (5, 5)]
    assert not best["overlap_ok"]


def test_brute_force_tie_breaks_bytes_then_groups():
    # no transfer cost: every partition has the same predicted time
    c = costs_uniform(5, tu=0.0, ts=0.0)
    # everything stays resident in any partition (same bytes): fewest groups
    best = P.brute_force(c, budget=10 ** 9, reserve=0, accum=1, dtype=P.BF16)
    assert best["groups"] == [(0, 4)]
    # 800 bytes beside the reserve: groups of two nodes get slots of 200 and
    # gradient slots of 400, so two weight slots, and three groups reload one
    # group in the backward; single nodes get six slots of 100 next to 200 of
    # gradient slots, so nothing reloads: fewest bytes wins over fewest groups
    best = P.brute_force(c, budget=400 + 4 * 200, reserve=400, accum=1, dtype=P.BF16)
    assert best["groups"] == [(i, i) for i in range(5)]
    assert best["h2d_bytes"] == 5 * 100
    # among the three-group plans, the one reloading the smallest group wins
    # ((1,2,2): 100 bytes; (2,1,2) and (2,2,1): 200), although [0,2,4] is also
    # the smallest end list
    three = P.best([[(0, 0), (1, 2), (3, 4)], [(0, 1), (2, 2), (3, 4)], [(0, 1), (2, 3), (4, 4)]], c,
                   400 + 4 * 200, 400, 1, P.BF16)
    assert [b for _, b in three["groups"]] == [0, 2, 4] and three["h2d_bytes"] == 600


def test_brute_force_none_when_nothing_fits():
    c = costs_uniform(3, w=100)
    assert P.brute_force(c, budget=350, reserve=0, accum=1, dtype=P.BF16) is None


def test_structured_candidates_are_valid_partitions():
    for L in (1, 2, 3, 7, 12):
        n = L + 2
        cands = list(P.structured_candidates(L))
        assert cands
        for g in cands:
            assert g[0][0] == 0 and g[-1][1] == n - 1
            for (a, b), (c, _) in zip(g, g[1:]):
                assert c == b + 1 and a <= b
        assert [(i, i) for i in range(n)] in cands


def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def test_table2_activation_payload_is_one_fp32_block_cut():
    # Table II: payload of a [1, 2048, d_model] fp32 activation at a block cut
    for model, L, d, h, mib in _read_golden("table2_activation_payload.txt"):
        assert 1 * int(L) * int(d) * 4 == int(mib) * 2 ** 20, model


def test_paper_printed_sizes():
    g = {r[0]: float(r[1]) for r in _read_golden("paper_sizes.txt")}
    d, L, V, T = 12288, 96, 50257, 2048
    cfg175 = Config("175b", L, d, 96, 4 * d, V, T, 1)
    n = param_count(cfg175)
    # GPT-3 175B is "175B" parameters; untied head adds V*d
    assert 174e9 < n - V * d < 176e9
    fp32_gb = (n - V * d) * 4 / 1e9
    assert fp32_gb == pytest.approx(g["gpt3_175b_fp32_params_GB"], rel=0.01)
    assert 4 * fp32_gb / 1e3 == pytest.approx(g["gpt3_175b_with_optimizer_TB"], rel=0.01)
    assert 50000 * d * 4 / 1e9 == pytest.approx(g["gpt3_175b_embedding_fp32_GB"], rel=0.04)


def test_config_param_counts():
    # 12 d^2 + 13 d per block, plus two V x d matrices, T x d and the final LN
    exp = {"tiny": 2.137e6, "small": 163.8e6, "xl": 1.419e9, "6.7b": 6.864e9, "13b": 13.111e9}
    for k, v in exp.items():
        assert param_count(CONFIGS[k]) == pytest.approx(v, rel=2e-3), k
