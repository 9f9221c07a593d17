"""Pins of the planner oracle: enumeration, schedule closed forms, the
selection rule of Section III-D, paper sizes."""
import os

import pytest

from oracle import plan as P
from synthetic import CONFIGS, Config, param_count

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def costs_uniform(n, w=100, tf=1.0, tb=2.0, tu=3.0, ts=3.0, mem=0, cut=10):
    return [dict(weight_bytes=w, mem_bytes=mem, cut_bytes=cut, t_fwd=tf, t_bwd=tb, t_load=tu, t_store=ts)
            for _ in range(n)]


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


# ------------------------------------------------------------------ schedule
def test_single_group_step_is_serial():
    # one group of three nodes (embedding, block, head): load all, forward of
    # two micro-batches, backward (the head has none), store all
    c = costs_uniform(3)
    c[2]["t_bwd"] = 0.0
    t_fwd, ends = P.simulate([(0, 2)], c, accum=2, K=1, R=2)
    assert t_fwd == 9.0 + 2 * 3.0
    assert ends == [9.0 + 6.0 + 2 * 4.0 + 9.0]


def test_link_bound_resident_step_is_sum_of_transfers():
    # no compute, every group in its own slot: loads back to back, then the
    # stores back to back (the backward needs the loss, so nothing overlaps)
    c = costs_uniform(5, tf=0.0, tb=0.0, tu=1.5, ts=2.5)
    groups = [(i, i) for i in range(5)]
    t_fwd, ends = P.simulate(groups, c, accum=1, K=5, R=2, duplex=0.5)
    assert t_fwd == 7.5 and ends == [7.5 + 12.5]


def test_compute_bound_exposes_first_load_and_last_store():
    c = costs_uniform(4, tf=10.0, tb=20.0, tu=1.0, ts=1.0)
    c[3]["t_bwd"] = 0.0
    groups = [(i, i) for i in range(4)]
    t_fwd, ends = P.simulate(groups, c, accum=1, K=4, R=2)
    assert t_fwd == 1.0 + 40.0
    assert ends == [1.0 + 40.0 + 60.0 + 1.0]
    # pipelined: the next step's loads hide under this step's backward
    _, ends = P.simulate(groups, c, accum=1, K=4, R=2, n_steps=4)
    assert [b - a for a, b in zip(ends, ends[1:])] == [100.0, 100.0, 100.0]


@pytest.mark.parametrize("duplex,want", [(1.0, [5.0, 8.0]), (0.5, [7.0, 10.0])])
def test_shared_link_between_steps(duplex, want):
    # one group, no compute: step 0's gradient copy (3 s alone) and step 1's
    # load (2 s alone) start together after step 0's backward.  Full duplex:
    # they run side by side.  duplex 0.5: both at half rate until the load
    # ends at 2 + 2/0.5 = 6 with 1 s of the copy left, which ends at 7; step
    # 1's copy then runs alone from 7 to 10.
    c = [dict(weight_bytes=1, mem_bytes=0, cut_bytes=1, t_fwd=0.0, t_bwd=0.0, t_load=t, t_store=s)
         for t, s in ((0.5, 1.0), (1.0, 1.0), (0.5, 1.0))]
    _, ends = P.simulate([(0, 2)], c, accum=1, K=1, R=2, n_steps=2, duplex=duplex)
    assert ends == want


def test_retained_weights_load_once_per_call():
    # one group of three nodes (load 1 s each, forward 2 s, backward 3 s, the
    # head none, store 1 s each), one slot: T_c = 3 x 2 + 2 x 3 = 12 s of
    # compute per step.  Retained, only step 0 loads and each later step's
    # compute follows the previous one's at once: end of step s = load +
    # (s + 1) T_c + store, whatever the link sharing (the engines never run
    # together).  Reloaded with the link shared (duplex 1): (s + 1)(load +
    # T_c) + store; at duplex 0.5 each load runs beside the previous step's
    # gradient copy at half rate (3 s of each: 6 s), so step 0's copy ends at
    # 15 + 6 = 21, step 1's (beside step 2's load) at 21 + 12 + 6 = 39 and
    # step 2's at 39 + 12 + 3 = 54.
    c = [dict(weight_bytes=1, mem_bytes=0, cut_bytes=1, t_fwd=2.0, t_bwd=b, t_load=1.0, t_store=1.0)
         for b in (3.0, 3.0, 0.0)]
    for duplex in (1.0, 0.5):
        _, ends = P.simulate([(0, 2)], c, accum=1, K=1, R=2, n_steps=3, duplex=duplex, retain=True)
        assert ends == [3.0 + 12.0 * (s + 1) + 3.0 for s in range(3)]
    _, ends = P.simulate([(0, 2)], c, accum=1, K=1, R=2, n_steps=3, duplex=1.0)
    assert ends == [15.0 * (s + 1) + 3.0 for s in range(3)]
    _, ends = P.simulate([(0, 2)], c, accum=1, K=1, R=2, n_steps=3, duplex=0.5)
    assert ends == [21.0, 39.0, 54.0]
    # a call of one step is the same either way; with fewer slots than groups
    # retention changes nothing (every group is loaded again each step)
    assert P.simulate([(0, 2)], c, 1, 1, 2, 1, 0.5, retain=True) == P.simulate([(0, 2)], c, 1, 1, 2, 1, 0.5)
    two = [(0, 0), (1, 2)]
    assert P.simulate(two, c, 1, 1, 2, 3, 1.0, retain=True) == P.simulate(two, c, 1, 1, 2, 3, 1.0)


def test_gradient_slots_throttle_the_backward():
    # five one-node groups, all resident, slow copies out: with R gradient
    # slots, the backward of the group R claims later waits for the copy out
    # of the slot it reuses.  Claims: head (group 4) at its forward, then
    # groups 3, 2, 1, 0 in the backward.
    c = costs_uniform(5, tf=0.0, tb=1.0, tu=0.0, ts=10.0)
    c[4]["t_bwd"] = 0.0
    groups = [(i, i) for i in range(5)]
    # R = 16: copies queue on the engine; backward runs 4 x 1 s unhindered;
    # the five copies of 10 s run back to back from t = 0 (the head's copy
    # waits only for the head's forward)
    _, ends = P.simulate(groups, c, accum=1, K=5, R=16)
    assert ends == [50.0]
    # R = 2: group 2's backward (third claim) waits for the head's copy
    # (0..10), group 1's for group 3's copy (10..20), group 0's for group 2's
    # (20..30); the last copy, group 0's, runs 40..50: the same end, but the
    # backward now ends at 31
    jobs = P.build_jobs(groups, c, 1, 5, 2, 1)
    end = P.run_jobs(jobs, 1.0)
    bwd_end = max(e for e, j in zip(end, jobs) if j[4] == "bwd")
    assert bwd_end == 31.0
    assert P.step_ends(jobs, end, 1) == [50.0]


def test_reload_waits_for_the_slot_it_reuses():
    # four one-node groups in two slots: groups 0 and 1 are loaded again in
    # the backward, each after the backward of the group two later
    c = costs_uniform(4, tf=1.0, tb=1.0, tu=2.0, ts=0.0)
    c[3]["t_bwd"] = 0.0
    jobs = P.build_jobs([(i, i) for i in range(4)], c, 1, 2, 2, 1)
    kinds = [(j[0], j[4]) for j in jobs]
    assert kinds.count(("I", "reload")) == 2
    end = P.run_jobs(jobs, 1.0)
    # forward: load0 0-2, fwd0 2-3, load1 2-4 (queued), fwd1 4-5, load2 after
    # fwd0 and load1: 4-6, fwd2 6-7, load3 6-8, fwd3 (head) 8-9.  Backward:
    # the head has no backward, so its group's last compute is its forward
    # (9) and reload1 (into its slot) runs 9-11; bwd2 9-10 (resident);
    # reload0 after bwd2 and behind reload1: 11-13; bwd1 11-12; bwd0 13-14
    assert P.step_ends(jobs, end, 1) == [14.0]
    reloads = [e for e, j in zip(end, jobs) if j[4] == "reload"]
    assert reloads == [11.0, 13.0]


def test_host_checkpoint_ring():
    # five blocks, one group, no weights to move and no compute: only the
    # block inputs 0 and 1 leave the four-entry ring (1 s each way).  ckout0
    # 0-1 (after fwd0), ckout1 1-2; fwd4 waits ckout0, fwd5 waits ckout1 (2);
    # the head's restore of input 1 runs 2-3, bwd5's restore of input 0 3-4;
    # bwd2 waits input 1 (3), bwd1 waits input 0 (4)
    c = [dict(weight_bytes=1, mem_bytes=0, cut_bytes=1, t_fwd=0.0, t_bwd=0.0, t_load=0.0, t_store=0.0)
         for _ in range(7)]
    t_fwd, ends = P.simulate([(0, 6)], c, accum=1, K=1, R=2, n_layer=5, ck_host=True, t_ck_out=1.0, t_ck_in=1.0)
    assert t_fwd == 2.0 and ends == [4.0]
    jobs = P.build_jobs([(0, 6)], c, 1, 1, 2, 1, n_layer=5, ck_host=True, t_ck_out=1.0, t_ck_in=1.0)
    assert sum(j[4] == "ckout" for j in jobs) == 2 and sum(j[4] == "restore" for j in jobs) == 2


# ------------------------------------------------------------------ memory
def test_memory_slots_and_working_memory():
    c = costs_uniform(4, w=10)
    groups = [(i, i) for i in range(4)]
    # base 1000, two gradient slots of 10: two weight slots fit in 40
    ok, K, R, S, arena = P.memory(groups, c, budget=1000 + 4 * 10, base=1000, accum=1, dtype=P.BF16)
    assert ok and (K, R, S, arena) == (2, 2, 10, 1040)
    assert P.transfer_bytes(groups, c, K) == (40 + 20, 40)
    # the largest working memory m_i joins the reserve (max, not sum)
    c[2]["mem_bytes"] = 500
    c[1]["mem_bytes"] = 300
    assert not P.memory(groups, c, budget=1000 + 4 * 10, base=1000, accum=1, dtype=P.BF16)[0]
    ok, K, R, S, arena = P.memory(groups, c, budget=1500 + 4 * 10, base=1000, accum=1, dtype=P.BF16)
    assert ok and K == 2 and arena == 1540
    # budget left after the weight slots becomes gradient slots, up to 16
    ok, K, R, S, arena = P.memory(groups, c, budget=1500 + 4 * 10 + 2 * 10 + 7 * 10, base=1000, accum=1,
                                  dtype=P.BF16)
    assert (K, R) == (4, 9) and arena == 1500 + 4 * 10 + 9 * 10
    ok, K, R, S, arena = P.memory(groups, c, budget=10 ** 9, base=1000, accum=1, dtype=P.BF16)
    assert (K, R) == (4, 16)


def test_memory_rejects_budget_below_two_slots():
    c = costs_uniform(4, w=10)
    groups = [(i, i) for i in range(4)]
    assert not P.memory(groups, c, budget=1000 + 3 * 10, base=1000, accum=1, dtype=P.BF16)[0]
    # a single group needs one weight slot only
    assert P.memory([(0, 3)], c, budget=1000 + 3 * 40, base=1000, accum=1, dtype=P.BF16)[0]
    # bf16 with accumulation adds an fp32 slot of 2S
    assert not P.memory(groups, c, budget=1000 + 5 * 10, base=1000, accum=2, dtype=P.BF16)[0]
    assert P.memory(groups, c, budget=1000 + 6 * 10, base=1000, accum=2, dtype=P.BF16)[0]
    assert P.memory(groups, c, budget=1000 + 4 * 10, base=1000, accum=2, dtype=P.F32)[0]


# ------------------------------------------------------------------ overlap
def test_overlap_constraint():
    c = costs_uniform(4, tf=1.0, tb=2.0, tu=3.0)
    g = [(i, i) for i in range(4)]
    assert not P.overlap_ok(g, c, accum=1, K=4)  # forward 1 < load 3
    assert P.overlap_ok(g, c, accum=3, K=4)  # C = 3: 3 >= 3 (the paper's remedy)
    # backward: a reloaded group j needs C t^b(g_{j+1}) >= t^u(g_j)
    c2 = costs_uniform(4, tf=3.0, tb=1.0, tu=2.0)
    assert P.overlap_ok(g, c2, accum=1, K=4)  # nothing reloaded
    assert not P.overlap_ok(g, c2, accum=1, K=2)  # groups 0, 1 reloaded: 1 < 2
    assert P.overlap_ok(g, c2, accum=2, K=2)
    # a single group has no neighbour: the constraint holds vacuously
    assert P.overlap_ok([(0, 3)], c, accum=1, K=1)


# ------------------------------------------------------------------ selection
def test_minimum_cut_beats_a_faster_partition():
    # everything overlaps; the whole model in one group has no cut at all and
    # wins, although loading it whole exposes 4 s of transfers at each end
    c = costs_uniform(4, tf=2.0, tb=4.0, tu=1.0, ts=1.0, cut=7)
    c[3]["t_bwd"] = 0.0
    best = P.brute_force(c, budget=10 ** 6, base=0, accum=1, dtype=P.BF16)
    assert best["groups"] == [(0, 3)] and best["rule"] == "paper" and best["cut_bytes"] == 0
    singles = P.evaluate([(i, i) for i in range(4)], c, 10 ** 6, 0, 1, P.BF16)
    assert singles["overlap_ok"] and singles["pred_first_step_s"] < best["pred_first_step_s"]
    # with a budget that cannot hold the whole model in one slot, the fewest
    # cuts among overlapping partitions win: two groups of two nodes
    # (S = 200: 3 S + 2 S gradient slots... K = 2, no reload)
    best = P.brute_force(c, budget=4 * 200, base=0, accum=1, dtype=P.BF16)
    assert best["rule"] == "paper" and len(best["groups"]) == 2 and best["cut_bytes"] == 7
    assert best["groups"] == [(0, 1), (2, 3)]


def test_cut_sizes_decide_between_equal_group_counts():
    # cuts differ per edge: the partition with the cheaper edge wins
    c = costs_uniform(4, tf=2.0, tb=4.0, tu=1.0, ts=1.0)
    for i, cb in enumerate((50, 5, 50, 0)):
        c[i]["cut_bytes"] = cb
    best = P.best([[(0, 0), (1, 3)], [(0, 1), (2, 3)], [(0, 2), (3, 3)]], c, 4 * 300, 0, 1, P.BF16)
    assert best["groups"] == [(0, 1), (2, 3)] and best["cut_bytes"] == 5


def test_no_overlapping_partition_strict_and_fallback():
    # loads dwarf compute and the budget forbids one group: nothing overlaps
    c = costs_uniform(4, tf=0.1, tb=0.2, tu=5.0, ts=5.0)
    c[3]["t_bwd"] = 0.0
    budget = 4 * 100 + 2 * 100  # singletons: four slots and two gradient slots
    assert P.brute_force(c, budget, 0, 1, P.BF16, strict=True) is None
    best = P.brute_force(c, budget, 0, 1, P.BF16)
    assert best["rule"] == "time" and not best["overlap_ok"]
    # the fallback is the fastest memory-feasible partition
    for g in P.compositions(4):
        p = P.evaluate(g, c, budget, 0, 1, P.BF16)
        assert p is None or p["pred_step_s"] >= best["pred_step_s"]
    # and C large enough restores the paper's rule
    best = P.brute_force(c, budget, 0, 100, P.F32)
    assert best["rule"] == "paper" and best["overlap_ok"]


def test_brute_force_none_when_nothing_fits():
    c = costs_uniform(3, w=100)
    assert P.brute_force(c, budget=350, base=0, accum=1, dtype=P.BF16) is None


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


# ------------------------------------------------------------------ paper sizes
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
