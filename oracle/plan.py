"""Oracle for the partition planner: brute-force enumeration.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Algorithm 1 (Section III-D) searches, with step size 1, the ways to cut the
topologically sorted layer chain into contiguous sub-models such that the
executing sub-model and the one being preloaded both fit the GPU, and the
executing sub-model's compute (scaled by the gradient-accumulation degree C)
covers the next sub-model's load time.  Among the valid partitions Atom keeps
the one with the smallest total cut-tensor size; the paper's objective also
minimises computation time.

Because step size 1 makes the search exhaustive, its result is defined by the
set of all compositions of the chain into contiguous groups, which this module
enumerates directly (2^(n-1) of them, so only small n).  The readings of the
constraints and of the objective:

Memory (hard).  Groups are staged in equal weight slots of S = the largest
group's weight bytes.  Gradients drain through two gradient slots of S bytes;
a bf16 step with C > 1 also keeps an fp32 accumulation slot of 2S bytes.  With
R reserved bytes (activations, checkpoints, workspace) the number of weight
slots is K = min(G, floor((budget - R - grad_slots) / S)), and a partition is
feasible when K >= min(G, 2): the executing group and the prefetched one are
co-resident.

Schedule (used for the predicted step time).  Group j uses weight slot j mod
K.  Forward: the load stream loads groups in order, group j waiting for the
forward of group j-K to free its slot; compute runs groups in order, each
after its load.  The last K groups stay resident into the backward.
Backward runs groups in reverse; a group that is not resident is reloaded
into its slot once group j+K's backward has freed it; group j's backward
also waits for the gradient slot it shares with group j+2 to have drained;
after it, the store stream copies its gradients out.  Per group:
F = C * sum(t_fwd), B = C * sum(t_bwd), U = sum(t_load), S = sum(t_store),
sums in ascending node order.  Step time = max(compute end, store end).

Overlap (soft, reported).  Forward: C*t_fwd(g_j) >= t_load(g_{j+1}) for all
consecutive groups; backward: C*t_bwd(g_{j+1}) >= t_load(g_j) for every
group that has to be reloaded.

Selection.  Among feasible partitions: smallest predicted step time, then
fewest bytes loaded (the schedule model runs loads and stores at full rate
each, so reloads that overlap the gradient stores look free although both
directions share the host link), then fewest groups (the smallest total cut
size, since every cut is one [B,T,d] activation), then the lexicographically
smallest list of group end nodes.
"""
from __future__ import annotations

import itertools

F32, BF16 = 0, 1


def compositions(n):
    """All partitions of nodes 0..n-1 into contiguous groups, as lists of (first, last)."""
    for mask in range(1 << (n - 1)):
        groups, start = [], 0
        for i in range(n - 1):
            if mask >> i & 1:
                groups.append((start, i))
                start = i + 1
        groups.append((start, n - 1))
        yield groups


def _group_sums(groups, costs, accum):
    F, B, U, S, W = [], [], [], [], []
    for a, b in groups:
        tf = tb = tu = ts = 0.0
        w = 0
        for i in range(a, b + 1):
            tf += costs[i]["t_fwd"]
            tb += costs[i]["t_bwd"]
            tu += costs[i]["t_load"]
            ts += costs[i]["t_store"]
            w += costs[i]["weight_bytes"]
        F.append(accum * tf)
        B.append(accum * tb)
        U.append(tu)
        S.append(ts)
        W.append(w)
    return F, B, U, S, W


def memory(groups, costs, budget, reserve, accum, dtype):
    """(feasible, K, slot_bytes, arena_bytes) under the slot model in the module docstring."""
    W = _group_sums(groups, costs, accum)[4]
    G = len(groups)
    S = max(W)
    grad = 2 * S + (2 * S if (accum > 1 and dtype == BF16) else 0)
    if S == 0 or budget < reserve + grad:
        return False, 0, S, 0
    kmax = (budget - reserve - grad) // S
    K = min(G, kmax)
    if K < min(G, 2):
        return False, 0, S, 0
    return True, K, S, reserve + K * S + grad


def simulate(groups, costs, accum, K):
    """Predicted (forward end, step end) of the three-stream schedule."""
    F, B, U, S, _ = _group_sums(groups, costs, accum)
    G = len(groups)
    h = c = d = 0.0
    fend = [0.0] * G
    for j in range(G):
        free = fend[j - K] if j >= K else 0.0
        ls = max(h, free)
        le = ls + U[j]
        h = le
        cs = max(c, le)
        fend[j] = cs + F[j]
        c = fend[j]
    t_fwd = c
    bend = [0.0] * G
    dend = [0.0] * G
    for j in range(G - 1, -1, -1):
        if j >= G - K:
            ready = 0.0
        else:
            ls = max(h, bend[j + K])
            le = ls + U[j]
            h = le
            ready = le
        gfree = dend[j + 2] if j + 2 <= G - 1 else 0.0
        bs = max(c, ready, gfree)
        bend[j] = bs + B[j]
        c = bend[j]
        ds = max(d, bend[j])
        dend[j] = ds + S[j]
        d = dend[j]
    return t_fwd, max(c, d)


def overlap_ok(groups, costs, accum, K):
    F, B, U, _, _ = _group_sums(groups, costs, accum)
    G = len(groups)
    for j in range(G - 1):
        if F[j] < U[j + 1]:
            return False
    for j in range(G - 1):
        if j < G - K and B[j + 1] < U[j]:
            return False
    return True


def transfer_bytes(groups, costs, K):
    """(bytes loaded, bytes stored) by the schedule."""
    W = [sum(costs[i]["weight_bytes"] for i in range(a, b + 1)) for a, b in groups]
    G = len(groups)
    h2d = sum(W) + sum(W[j] for j in range(G) if j < G - K)
    return h2d, sum(W)


def evaluate(groups, costs, budget, reserve, accum, dtype):
    ok, K, S, arena = memory(groups, costs, budget, reserve, accum, dtype)
    if not ok:
        return None
    t_fwd, t_step = simulate(groups, costs, accum, K)
    h2d, d2h = transfer_bytes(groups, costs, K)
    return dict(groups=groups, n_slots=K, slot_bytes=S, arena_bytes=arena, pred_fwd_s=t_fwd,
                pred_step_s=t_step, overlap_ok=overlap_ok(groups, costs, accum, K),
                h2d_bytes=h2d, d2h_bytes=d2h)


def rank_key(plan):
    return (plan["pred_step_s"], plan["h2d_bytes"], len(plan["groups"]), [b for _, b in plan["groups"]])


def best(candidates, costs, budget, reserve, accum, dtype):
    """Best plan among `candidates` (iterable of group lists), or None if none fits."""
    out = None
    for groups in candidates:
        p = evaluate(groups, costs, budget, reserve, accum, dtype)
        if p is not None and (out is None or rank_key(p) < rank_key(out)):
            out = p
    return out


def brute_force(costs, budget, reserve, accum, dtype):
    return best(compositions(len(costs)), costs, budget, reserve, accum, dtype)


def structured_candidates(n_layer):
    """Partitions that use the chain's structure: identical decoder blocks.

    Node 0 (embedding) forms a group alone or with the first block; node L+1
    (head) alone or with the last block; the remaining blocks are cut into
    groups of s consecutive blocks, the remainder forming the first of them.
    Section III-D notes that identical blocks shrink the search space.
    """
    L = n_layer
    seen = set()
    for e, h in itertools.product((0, 1), (0, 1)):
        lo, hi = 1 + e, L - h  # middle blocks lo..hi inclusive
        m = hi - lo + 1
        if m < 0:
            continue
        for s in range(1, max(m, 1) + 1):
            groups = [(0, e)]
            if m > 0:
                r = m % s
                start = lo
                if r:
                    groups.append((start, start + r - 1))
                    start += r
                while start <= hi:
                    groups.append((start, start + s - 1))
                    start += s
            groups.append((L + 1 - h, L + 1))
            key = tuple(groups)
            if key not in seen:
                seen.add(key)
                yield groups
