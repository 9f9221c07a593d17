"""Oracle for the partition planner: brute-force enumeration and a plain
event simulation of the swap schedule.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

What Section III-D defines.  The layer chain (topologically sorted nodes
0..l) carries per node its maximum working memory m_i, forward time t^f,
backward time t^b and loading time t^u.  Algorithm 1 searches, with step size
1, the ways to cut the chain into contiguous sub-models such that the
sub-model that executes and the one being preloaded both fit the GPU, and the
executing sub-model's compute (scaled by the gradient-accumulation degree C)
covers the next sub-model's load time.  Among the valid partitions Atom keeps
the one with the smallest total size of the tensors on the cut edges.

Because step size 1 makes the search exhaustive, its result is defined by the
set of all compositions of the chain into contiguous groups, which this module
enumerates directly (2^(n-1) of them, so only small n).  The readings:

Memory (hard).  Groups are staged in K equal weight slots of S = the largest
group's weight bytes.  The executing group and the prefetched one must be
co-resident, so K >= min(G, 2).  Working memory: every node's activations are
recomputed in its backward from its input checkpoint, so nothing of a node's
working memory outlives it and one workspace serves every node in turn; the
sub-model sum of m_i in the paper's constraint becomes the maximum over nodes
here.  Gradients drain through R >= 2 gradient slots of S bytes; a bf16 step
with C > 1 also keeps an fp32 accumulation slot of 2S.  With `base` bytes of
other device memory (checkpoints, tokens, residual gradient), a partition is
feasible when base + max m_i + K*S + 2S (+ 2S) <= budget with K = min(G,
floor(room / S)); budget left after that becomes extra gradient slots,
R = min(16, 2 + floor(left / S)).

Overlap (the paper's second constraint).  Forward: C * t^f(g_j) >= t^u(g_{j+1})
for every pair of consecutive groups.  Backward: C * t^b(g_{j+1}) >= t^u(g_j)
for every group j that must be loaded again (j < G - K).

Selection.  Among partitions that satisfy memory and overlap: smallest total
cut size (sum of cut_bytes of each group's last node except the last group's),
then smallest predicted step time, then the lexicographically smallest list
of group end nodes.  When no partition satisfies overlap the paper's search
returns nothing: in strict mode so does this one; otherwise (a reading, not
the paper's rule) the memory-feasible partition with the smallest predicted
step time is taken, then fewest bytes loaded, then smallest cut, then the end
list.

Schedule (for the predicted times).  Three servers run jobs in the order they
are issued: the compute stream (X), the host-to-device engine (I) and the
device-to-host engine (O).  A job starts when the previous job of its server
has ended and every job it depends on has ended.  Compute jobs take their
time; a copy takes its time alone, but while both copy engines are busy each
progresses at `duplex` times its rate alone (both directions share the host
link).  The jobs of a call of n steps, in issue order (group j uses weight
slot j mod K in even steps and K-1-(j mod K) in odd ones):

* before step 0: load(0, j) for j < min(G, K);
* step s, forward, for each group j in order: for each node of j, fwd(s, node)
  (time C * t^f; its group's first node waits for the group's load; the head
  waits for the gradient slot it claims; with host checkpoints a block input
  i written by fwd(s, i) with i <= L - 4 is copied out by ckout(s, i) after
  it, fwd(s, i) waits for ckout(s, i - 4), and after the head restore(s, L-4)
  is issued); then load(s, j + K) if j + K < G, after fwd of j's last node;
* step s, backward, for j = G-1 .. 0: for each block node of j from the last,
  bwd(s, node) (time C * t^b; its group's first job waits for the group's
  weights, the reload if j < G - K, and for the gradient slot it claims; with
  host checkpoints a block waits for the restore of its input if that input
  was evicted, and after bwd(s, n) restore(s, n - 5) is issued if n >= 5);
  then gcopy(s, j) (time sum of t_store, after j's last compute job); then
  load(s, j - K) if j >= K (a reload), else load(s + 1, K - 1 - j) if another
  step follows, each after j's last compute job.

Gradient slots are claimed round-robin in claim order (the head's group at its
forward, the others at their first backward job); a claim waits for the copy
out of the claim R claims earlier.  A step ends when both its last compute job
and its last gradient copy have ended.  Micro-batches of one node are one
job; the host accumulation and token uploads are not modelled.
"""
from __future__ import annotations

import itertools

F32, BF16 = 0, 1
MAX_GSLOTS = 16
CKPT_RING = 4


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


def group_weights(groups, costs):
    return [sum(costs[i]["weight_bytes"] for i in range(a, b + 1)) for a, b in groups]


def memory(groups, costs, budget, base, accum, dtype):
    """(feasible, K, R, slot_bytes, arena_bytes) under the slot model of the module docstring."""
    W = group_weights(groups, costs)
    G = len(groups)
    S = max(W)
    work = max(c.get("mem_bytes", 0) for c in costs)
    acc = 2 * S if (accum > 1 and dtype == BF16) else 0
    fixed = base + work + 2 * S + acc
    if S == 0 or budget < fixed:
        return False, 0, 0, S, 0
    K = min(G, (budget - fixed) // S)
    if K < min(G, 2):
        return False, 0, 0, S, 0
    left = budget - fixed - K * S
    R = min(MAX_GSLOTS, 2 + left // S)
    return True, K, R, S, fixed + K * S + (R - 2) * S


def cut_bytes(groups, costs):
    return sum(costs[b]["cut_bytes"] for _, b in groups[:-1])


def overlap_ok(groups, costs, accum, K):
    G = len(groups)
    F = [accum * sum(costs[i]["t_fwd"] for i in range(a, b + 1)) for a, b in groups]
    B = [accum * sum(costs[i]["t_bwd"] for i in range(a, b + 1)) for a, b in groups]
    U = [sum(costs[i]["t_load"] for i in range(a, b + 1)) for a, b in groups]
    for j in range(G - 1):
        if F[j] < U[j + 1]:
            return False
    for j in range(G - 1):
        if j < G - K and B[j + 1] < U[j]:
            return False
    return True


def transfer_bytes(groups, costs, K, ckpt_bytes=0):
    """(bytes loaded, bytes stored) by one step of the schedule."""
    W = group_weights(groups, costs)
    G = len(groups)
    h2d = sum(W) + sum(W[j] for j in range(G) if j < G - K)
    return h2d + ckpt_bytes, sum(W) + ckpt_bytes


def build_jobs(groups, costs, accum, K, R, n_steps, n_layer=None, ck_host=False, t_ck_out=0.0, t_ck_in=0.0,
               retain=False):
    """Jobs of a call of n_steps steps: (server, duration, deps, step, kind) in issue order.

    retain: when each group has its own slot (K = G) its weights stay on the
    device for the whole call (the host model changes only between global
    batches, Section III-C), so the steps after the first load nothing: their
    loads keep their place in the order with no length.  With fewer slots
    than groups every group is loaded again each step and retain changes
    nothing."""
    retain = retain and K >= len(groups)
    G = len(groups)
    L = len(costs) - 2 if n_layer is None else n_layer
    head = L + 1
    jobs = []

    def add(server, dur, deps, step, kind):
        jobs.append((server, dur, [d for d in deps if d is not None], step, kind))
        return len(jobs) - 1

    def evicted(i):
        return ck_host and 0 <= i and i + CKPT_RING <= L

    load = {}
    for j in range(min(G, K)):
        load[(0, j)] = add("I", sum(costs[i]["t_load"] for i in range(groups[j][0], groups[j][1] + 1)), [], 0, "load")
    claims = []  # per claim, the gradient copy that releases its slot (filled later)

    def claim_dep():
        k = len(claims)
        claims.append(None)
        return claims[k - R] if k >= R else None

    for s in range(n_steps):
        fwd, ckout, restore, last_c, claim_of = {}, {}, {}, {}, {}
        for j, (a, b) in enumerate(groups):
            for node in range(a, b + 1):
                deps = []
                if node == a:
                    deps.append(load[(s, j)])
                if node == head:
                    claim_of[j] = len(claims)
                    deps.append(claim_dep())
                if evicted(node - CKPT_RING):
                    deps.append(ckout[node - CKPT_RING])
                fwd[node] = add("X", accum * costs[node]["t_fwd"], deps, s, "fwd")
                if evicted(node):
                    ckout[node] = add("O", t_ck_out, [fwd[node]], s, "ckout")
                if ck_host and node == head and L - CKPT_RING >= 0:
                    restore[L - CKPT_RING] = add("I", t_ck_in, [fwd[node], ckout[L - CKPT_RING]], s, "restore")
            last_c[j] = fwd[b]
            if j + K < G:
                jb = groups[j + K]
                load[(s, j + K)] = add("I", sum(costs[i]["t_load"] for i in range(jb[0], jb[1] + 1)),
                                       [fwd[b]], s, "load")
        for j in range(G - 1, -1, -1):
            a, b = groups[j]
            first = True
            for node in range(min(b, L), a - 1, -1):
                deps = []
                if first:
                    if j < G - K:
                        deps.append(load[(s, j, "re")])
                    if j not in claim_of:
                        claim_of[j] = len(claims)
                        deps.append(claim_dep())
                    first = False
                if node >= 1 and evicted(node - 1):
                    deps.append(restore[node - 1])
                last_c[j] = add("X", accum * costs[node]["t_bwd"], deps, s, "bwd")
                if ck_host and node - 1 - CKPT_RING >= 0:
                    i = node - 1 - CKPT_RING
                    restore[i] = add("I", t_ck_in, [last_c[j], ckout[i]], s, "restore")
            gc = add("O", sum(costs[i]["t_store"] for i in range(a, b + 1)), [last_c[j]], s, "gcopy")
            claims[claim_of[j]] = gc
            if j - K >= 0:
                jb = groups[j - K]
                load[(s, j - K, "re")] = add("I", sum(costs[i]["t_load"] for i in range(jb[0], jb[1] + 1)),
                                             [last_c[j]], s, "reload")
            elif s + 1 < n_steps:
                jn = K - 1 - j
                jb = groups[jn]
                t_in = 0.0 if retain else sum(costs[i]["t_load"] for i in range(jb[0], jb[1] + 1))
                load[(s + 1, jn)] = add("I", t_in, [last_c[j]], s, "load")
    return jobs


def run_jobs(jobs, duplex):
    """End time of every job (processor sharing between the two copy engines)."""
    servers = ("X", "I", "O")
    queue = {sv: [i for i, jb in enumerate(jobs) if jb[0] == sv] for sv in servers}
    nxt = {sv: 0 for sv in servers}
    run = {sv: -1 for sv in servers}
    rem = {sv: 0.0 for sv in servers}
    end = [None] * len(jobs)
    t = 0.0
    while True:
        progress = True
        while progress:
            progress = False
            for sv in servers:
                if run[sv] < 0 and nxt[sv] < len(queue[sv]):
                    k = queue[sv][nxt[sv]]
                    if all(end[d] is not None for d in jobs[k][2]):
                        nxt[sv] += 1
                        progress = True
                        if jobs[k][1] <= 0.0:
                            end[k] = t
                        else:
                            run[sv] = k
                            rem[sv] = jobs[k][1]
        active = [sv for sv in servers if run[sv] >= 0]
        if not active:
            break
        both = run["I"] >= 0 and run["O"] >= 0
        rate = {sv: (duplex if (both and sv != "X") else 1.0) for sv in servers}
        tau = {sv: rem[sv] / rate[sv] for sv in active}
        dt = min(tau.values())
        t_new = t + dt
        for sv in active:
            if tau[sv] == dt:
                end[run[sv]] = t_new
                run[sv] = -1
                rem[sv] = 0.0
            else:
                rem[sv] = rem[sv] - rate[sv] * dt
        t = t_new
    if any(e is None for e in end):
        raise RuntimeError("schedule deadlock")
    return end


def step_ends(jobs, end, n_steps):
    out = []
    for s in range(n_steps):
        out.append(max(end[i] for i, jb in enumerate(jobs) if jb[3] == s and (jb[0] == "X" or jb[4] == "gcopy")))
    return out


def simulate(groups, costs, accum, K, R, n_steps=1, duplex=1.0, retain=False, **ck):
    """(forward end of step 0, list of step end times) of a call of n_steps steps."""
    jobs = build_jobs(groups, costs, accum, K, R, n_steps, retain=retain, **ck)
    end = run_jobs(jobs, duplex)
    t_fwd = max(end[i] for i, jb in enumerate(jobs) if jb[3] == 0 and jb[4] == "fwd")
    return t_fwd, step_ends(jobs, end, n_steps)


PIPE_STEPS = 4


def evaluate(groups, costs, budget, base, accum, dtype, duplex=1.0, **ck):
    ok, K, R, S, arena = memory(groups, costs, budget, base, accum, dtype)
    if not ok:
        return None
    t_fwd, one = simulate(groups, costs, accum, K, R, 1, duplex, **ck)
    _, ends = simulate(groups, costs, accum, K, R, PIPE_STEPS, duplex, **ck)
    h2d, d2h = transfer_bytes(groups, costs, K)
    return dict(groups=groups, n_slots=K, n_gslots=R, slot_bytes=S, arena_bytes=arena, pred_fwd_s=t_fwd,
                pred_first_step_s=one[0], pred_step_s=(ends[-1] - ends[-3]) / 2.0,
                overlap_ok=overlap_ok(groups, costs, accum, K), cut_bytes=cut_bytes(groups, costs),
                h2d_bytes=h2d, d2h_bytes=d2h)


def paper_key(p):
    return (p["cut_bytes"], p["pred_step_s"], [b for _, b in p["groups"]])


def time_key(p):
    return (p["pred_step_s"], p["h2d_bytes"], p["cut_bytes"], [b for _, b in p["groups"]])


def best(candidates, costs, budget, base, accum, dtype, strict=False, duplex=1.0, **ck):
    """Selected plan among `candidates` (iterable of group lists), or None.

    The returned dict carries rule = "paper" (minimum cut among partitions
    that satisfy memory and overlap) or "time" (the fallback)."""
    feas = [p for p in (evaluate(g, costs, budget, base, accum, dtype, duplex, **ck) for g in candidates)
            if p is not None]
    ok = [p for p in feas if p["overlap_ok"]]
    if ok:
        out = min(ok, key=paper_key)
        return dict(out, rule="paper")
    if strict or not feas:
        return None
    return dict(min(feas, key=time_key), rule="time")


def brute_force(costs, budget, base, accum, dtype, strict=False, duplex=1.0, **ck):
    return best(compositions(len(costs)), costs, budget, base, accum, dtype, strict, duplex, **ck)


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
