#!/usr/bin/env python3
"""Throughput of the swapped GPT training step on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 6.7b] [--accum C]

One step = the whole hot path over one batch: swap-in of every group,
forward, LM head and cross-entropy, backward with recompute, gradient
swap-out and host fp32 accumulation.  The timed steps are the steps of one
global batch, run by one pipelined call (atom_steps: the next step's first
groups are swapped in during the current step's backward; every step still
loads every weight and copies out every gradient); --sequential times one
atom_step call per step instead, each starting with no weights on the device.
Inputs are synthetic and seeded (weights N(0, 0.02), uniform tokens, a
different batch per step) with the shapes of the named GPT-3 configuration;
the host model is already in pinned memory when timing starts.

Prints one JSON line.  `value` is training tokens/s.  `roofline` is the
dominant kernel (the weight-gradient GEMM) against the bf16 MFMA peak, its
average launch time measured with HIP events on the compute stream inside
the timed steps.  `step_roofline` is the step against max(FLOP time at MFMA
peak, forced host-to-device bytes at the link rate measured in the same run).
`cpu_baseline` is the fp64 oracle on a bounded sample on this host's cores.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
HBM_PEAK_GBS = 8000.0

# HBM traffic of the weight-gradient GEMM per launch in the default workload
# (6.7B, C = 1), from two rocprofv3 --pmc passes (FETCH_SIZE, then
# WRITE_SIZE) over `bench.py --steps 2 --warmup 1 --no-cpu-baseline
# --copy-calibration 2147483648`, each scaled by what the counter reads for
# the plain copy kernel of known size (profiles/gemm_wgrad_6.7b_hbm_traffic.md).
# Valid only for the kernel sources it was measured on.
WGRAD_TRAFFIC = {"sources_sha256": "5b2c7ed08ef49c4e14822aaf57262fccd09a2efe914ec142e5b6281a7b7cd87c",
                 "bytes_per_launch": 725832891}
TRAFFIC_SOURCES = ("gemm.hip", "common.h", "launch.h")


def wgrad_kernel_name(cfg, epi):
    """The kernel the weight-gradient GEMMs (k = tokens of a micro-batch) launch."""
    if cfg.dtype != "bf16":
        return f"gemm_kernel<f32, A not k-contiguous, B not k-contiguous, epilogue {epi}> (weight gradients)"
    if (cfg.batch * cfg.seq_len) % 128 == 0:
        return (f"gemm_p4_kernel<A not k-contiguous, B not k-contiguous, epilogue {epi}> (weight gradients; "
                "four waves of 128x128 with double-buffered fragments, four-stage direct-to-LDS pipeline)")
    return (f"gemm_p3_kernel<A not k-contiguous, B not k-contiguous, epilogue {epi}> (weight gradients; "
            "sixteen waves, four-stage direct-to-LDS pipeline)")


def kernel_sources_sha256():
    import hashlib

    h = hashlib.sha256()
    for name in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, "paper_2403_10504_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def host_digests(sess, which):
    """SHA-256 of each node's host buffer `which` (raw bytes), hashed in parallel."""
    import ctypes
    import hashlib
    from concurrent.futures import ThreadPoolExecutor

    from paper_2403_10504_amd import atom as A

    def one(node):
        ptr, nbytes = A.atom_host_tensor(sess.ctx, node, which)
        return hashlib.sha256((ctypes.c_char * nbytes).from_address(ptr)).hexdigest()

    with ThreadPoolExecutor(8) as ex:
        return list(ex.map(one, range(sess.n_nodes)))


def blas_info():
    """The BLAS numpy uses here: library, version, threading layer and thread count."""
    from threadpoolctl import threadpool_info

    out = []
    for i in threadpool_info():
        if i.get("user_api") == "blas":
            out.append({k: i.get(k) for k in ("internal_api", "version", "threading_layer", "num_threads")})
    return out


RULES = {0: "paper: minimum cut among partitions meeting memory and overlap",
         1: "fallback: no partition meets overlap; fastest memory-feasible", 2: "fixed partition"}


def link_fit(sess, plan):
    """Copy time against size on the step's DMA engines (Section III-B: loading
    time grows linearly with a layer's size): t = a + bytes / r fitted by least
    squares for each direction, with R^2."""
    import numpy as np

    from paper_2403_10504_amd import atom as A

    cap = plan.n_slots * plan.slot_bytes // 2
    sizes = [s for s in (4 << 20, 16 << 20, 64 << 20, 256 << 20, 1 << 30) if s <= cap]
    rows = []
    for size in sizes:
        iters = max(2, (1 << 30) // size)
        h, d, _ = A.atom_link_bench(sess.ctx, size, iters)
        rows.append((size, size / (h * 1e9), size / (d * 1e9)))
    out = {"sizes_mb": [round(r[0] / 2 ** 20, 1) for r in rows]}
    x = np.array([r[0] for r in rows], np.float64)
    for k, name in ((1, "h2d"), (2, "d2h")):
        t = np.array([r[k] for r in rows])
        b, a = np.polyfit(x, t, 1)
        pred = a + b * x
        r2 = 1.0 - float(np.sum((t - pred) ** 2)) / float(np.sum((t - t.mean()) ** 2))
        out[name] = {"t_ms": [round(v * 1e3, 3) for v in t], "a_ms": round(a * 1e3, 4), "r_gbs": round(1 / b / 1e9, 2),
                     "r2": round(r2, 6)}
    return out


def step_flops(cfg):
    """Algorithmic FLOPs of one training step (forward + backward, no recompute):
    6 per parameter per token for the linear layers (blocks and LM head) plus
    6 T d per token per layer for causal attention (half of the T x T scores)."""
    N = cfg.accum * cfg.batch * cfg.seq_len
    L, d, V, T = cfg.n_layer, cfg.d_model, cfg.vocab, cfg.seq_len
    per_block = 4 * d * d + 2 * d * cfg.d_mlp
    return N * (6.0 * (L * per_block + V * d) + 6.0 * L * T * d)


def cpu_baseline(cfg):
    """The fp64 oracle on a bounded sample of the workload, extrapolated to one step.

    Sample: one decoder block forward + backward on one whole sequence of T
    tokens (its causal attention forward + backward also timed alone) and the
    LM head + cross-entropy forward + backward on batch x T tokens (about 10-15 s of
    CPU work at the 6.7B width).  Weights are converted to fp64 before the
    clock starts.  Extrapolation: x (accum * batch) sequences x layers for the
    block, x tokens for the head.
    """
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits

    import synthetic
    from oracle import gpt

    cores = len(os.sched_getaffinity(0))
    T, d, H, V = cfg.seq_len, cfg.d_model, cfg.n_head, cfg.vocab
    Ts = T
    n_head_tok = cfg.batch * T
    with threadpool_limits(limits=cores):
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        blas = blas_info()
        rng = np.random.default_rng(0)
        # weights handed over in fp64 so the timed region holds only the step's arithmetic
        p = {name: synthetic.gen_param(cfg, 1, name).astype(np.float64) for name, _, _ in synthetic.param_specs(cfg, 1)}
        x = rng.standard_normal((1, Ts, d))
        dout = rng.standard_normal((1, Ts, d)) * 1e-3
        t0 = time.perf_counter()
        _, cache = gpt.block_forward(x, p, H)
        gpt.block_backward(dout, cache, p, H)
        t_block = time.perf_counter() - t0
        t0 = time.perf_counter()
        gpt.causal_attention(cache["qkv"], H)
        gpt.causal_attention_backward(cache["o"], cache["qkv"], H)
        t_attn = time.perf_counter() - t0
        del cache, p
        ph = {name: synthetic.gen_param(cfg, cfg.n_layer + 1, name).astype(np.float64)
              for name in ("lnf_g", "lnf_b", "w_head")}
        xh = rng.standard_normal((1, n_head_tok, d))
        tgt = rng.integers(0, V, (1, n_head_tok))
        t0 = time.perf_counter()
        gpt.head_forward_backward(xh, ph, tgt, n_head_tok)
        t_head = time.perf_counter() - t0
    r = T / Ts
    t_block_seq = (t_block - t_attn) * r + t_attn * r * r
    n_tok = cfg.accum * cfg.batch * T
    t_step = cfg.accum * cfg.batch * cfg.n_layer * t_block_seq + t_head * n_tok / n_head_tok
    return {
        "value": n_tok / t_step,
        "unit": "tokens/s",
        "cores": threads,
        "affinity_cores": cores,
        "blas": blas,
        "kind": "oracle",
        "sample": (f"fp64 NumPy oracle: one decoder block forward+backward on a {Ts}-token sequence "
                   f"({t_block:.2f} s, of which causal attention {t_attn:.2f} s) and the LM head + "
                   f"cross-entropy forward+backward on {n_head_tok} tokens ({t_head:.2f} s); extrapolated to "
                   f"{cfg.accum}x{cfg.batch} sequences of {T} tokens x {cfg.n_layer} blocks and "
                   f"{n_tok} head tokens"),
        "extrapolated_step_s": t_step,
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64,
                    help="timed steps: one global batch in one pipelined call (64, the most one atom_steps call "
                         "takes; the paper synchronises once per global batch of 256 mini-batches)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="6.7b")
    ap.add_argument("--accum", type=int, default=None, help="gradient-accumulation degree C")
    ap.add_argument("--budget-gb", type=float, default=None, help="device budget (default: the config's)")
    ap.add_argument("--ckpt-host", action="store_true",
                    help="keep block-input checkpoints beyond a four-entry device ring in host memory (the 13B "
                         "configuration's policy; needed for large C under 24 GB)")
    ap.add_argument("--layers", type=int, default=None,
                    help="override the layer count (kernel profiling at the configuration's shapes in less time; "
                         "not a benchmark of the named model)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sequential", action="store_true", help="one atom_step call per step (no cross-step overlap)")
    ap.add_argument("--schedule", choices=["atom", "paper"], default="atom",
                    help="atom: the planner's partition and slots (Algorithm 1 with retention of the last K groups); "
                         "paper: one node per group in two weight slots (load g+1 while g runs, only the last "
                         "groups stay for the backward, every other group is loaded again in the backward)")
    ap.add_argument("--optimizer", action="store_true",
                    help="after the timed global batch, run the host AdamW step once (timed on its own, "
                         "not part of the step throughput, as in the paper), then time one more global batch "
                         "followed by the update, and one with the update armed (applied group by group as the "
                         "last step's gradients land)")
    ap.add_argument("--measured-plan", action="store_true",
                    help="profile every node on the GPU (atom_profile_nodes) and plan the timed steps with those "
                         "costs instead of the analytic ones")
    ap.add_argument("--retain", action="store_true",
                    help="keep every group's weights on the device across the steps of the call when each group "
                         "has a slot of its own (atom_set_retention: loaded once per global batch, gradients "
                         "still copied out every step); the default only for a configuration without a device "
                         "budget (the whole model resident, GPT-3 Small); under a budget every weight is loaded "
                         "every step")
    ap.add_argument("--no-retain", action="store_true",
                    help="load every weight every step also when the whole model is resident")
    ap.add_argument("--dense-embedding", action="store_true",
                    help="move the whole token-embedding matrix and its gradient every step (default: only the "
                         "rows the step's tokens use cross the host link, atom_set_embedding_rows; the same "
                         "results bit for bit)")
    ap.add_argument("--seq-steps", type=int, default=3,
                    help="after the timed steps, time this many single-step calls (the survey-literal step: no "
                         "cross-step overlap) and report their median beside the headline")
    ap.add_argument("--link-fit", action="store_true",
                    help="fit copy time against size (t = a + bytes / r, R^2) on the step's DMA engines")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="run one plain device copy of BYTES before the timed steps (calibrates HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the data-parallel path across GPUs is a design, not an implementation).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synthetic
    from paper_2403_10504_amd import Session
    from paper_2403_10504_amd import atom as A

    cfg = synthetic.CONFIGS[args.config]
    if args.accum:
        cfg = cfg.with_(accum=args.accum)
    if args.ckpt_host:
        cfg = cfg.with_(ckpt_host=True)
    if args.layers:
        cfg = cfg.with_(n_layer=args.layers)
    budget = int(args.budget_gb * 1e9) if args.budget_gb else (cfg.budget_bytes or (1 << 50))
    torch.cuda.set_device(0)

    t0 = time.time()
    if args.schedule == "paper":
        sess = Session(cfg, plan=A.atom_plan_fixed(A.make_config(cfg), list(range(cfg.n_layer + 2)), 2))
        if sess.plan.arena_bytes > budget:
            raise SystemExit(f"the paper schedule needs {sess.plan.arena_bytes / 1e9:.2f} GB, over the budget")
    else:
        sess = Session(cfg, budget=budget)
    plan = sess.plan
    log(f"plan: {plan.n_groups} groups, {plan.n_slots} slots of {plan.slot_bytes / 1e6:.1f} MB, "
        f"arena {plan.arena_bytes / 1e9:.2f} GB, H2D/step {plan.h2d_bytes / 1e9:.2f} GB ({time.time() - t0:.1f} s)")
    t0 = time.time()
    sess.load_weights()
    log(f"host model filled ({time.time() - t0:.1f} s)")
    n_batches = max(args.steps, args.warmup, 1)
    tokens = np.stack([synthetic.gen_tokens(cfg, seed=synthetic.TOKEN_SEED + i) for i in range(n_batches)])

    c = A.make_config(cfg)
    link_bytes = min(1 << 30, plan.n_slots * plan.slot_bytes // 2)
    h2d_gbs, d2h_gbs, bidir_gbs = A.atom_link_bench(sess.ctx, link_bytes, 4)
    duplex = min(1.0, bidir_gbs / (h2d_gbs + d2h_gbs))
    log(f"host link: H2D {h2d_gbs:.1f} GB/s, D2H {d2h_gbs:.1f} GB/s, both {bidir_gbs:.1f} GB/s "
        f"(each direction at {duplex:.3f} of its rate alone while both run)")
    fit = link_fit(sess, plan) if args.link_fit else None

    # measured node costs (t^u, t^f, t^b, m_i of Section III-D) predict the
    # timed call through the planner's schedule model
    t0 = time.time()
    costs = A.atom_profile_nodes(sess.ctx, c, tokens[0])
    blk = costs[1]
    log(f"node profile ({time.time() - t0:.1f} s): block load {blk.t_load * 1e3:.2f} ms, fwd {blk.t_fwd * 1e3:.2f} "
        f"ms, bwd {blk.t_bwd * 1e3:.2f} ms, working memory {blk.mem_bytes / 1e6:.1f} MB")
    plan_info = {"schedule": args.schedule, "costs": "analytic", "rule": RULES.get(plan.rule, plan.rule),
                 "overlap_ok": bool(plan.overlap_ok), "cut_mb": round(plan.cut_bytes / 1e6, 1),
                 "pred_step_ms_analytic": round(plan.pred_step_s * 1e3, 1),
                 "pred_first_step_ms_analytic": round(plan.pred_first_step_s * 1e3, 1)}
    plan_info["node_costs"] = {
        name: {"t_load_ms": round(x.t_load * 1e3, 3), "t_store_ms": round(x.t_store * 1e3, 3),
               "t_fwd_ms": round(x.t_fwd * 1e3, 3), "t_bwd_ms": round(x.t_bwd * 1e3, 3),
               "mem_mb": round(x.mem_bytes / 1e6, 1), "weight_mb": round(x.weight_bytes / 1e6, 1)}
        for name, x in (("embed", costs[0]), ("block", blk), ("head", costs[-1]))}
    if args.measured_plan:
        mplan = A.atom_plan_partition(c, budget, costs, duplex=duplex)
        plan_info.update(costs="measured", rule=RULES.get(mplan.rule, mplan.rule),
                         analytic_groups=plan.n_groups, analytic_slots=plan.n_slots)
        log(f"measured-cost plan: {mplan.n_groups} groups, {mplan.n_slots} slots, "
            f"predicted {mplan.pred_step_s * 1e3:.1f} ms per pipelined step")
        if mplan.groups() != plan.groups() or mplan.n_slots != plan.n_slots or mplan.n_gslots != plan.n_gslots:
            sess.close()
            del sess
            sess = Session(cfg, plan=mplan)
            sess.load_weights()
        plan = mplan
    sess.zero_grads()

    def run(n, arm=None):
        """n steps (tokens[i] for step i); returns the losses.  arm(): called
        before the call that runs the last step (an armed optimizer update)."""
        if args.sequential:
            if arm:
                raise SystemExit("--optimizer times pipelined calls; drop --sequential")
            out = []
            for i in range(n):
                out.append(sess.step(tokens[i]))
                log(f"step {i}: loss {out[-1]:.5f} ({sess.stats().step_s * 1e3:.1f} ms)")
            return out
        out = []
        for i0 in range(0, n, A.MAX_STEPS_PER_CALL):
            if arm and i0 + A.MAX_STEPS_PER_CALL >= n:
                arm()
            out.extend(sess.steps(tokens[i0:min(n, i0 + A.MAX_STEPS_PER_CALL)]).tolist())
            log(f"steps {i0}..{i0 + len(out) - 1}: {sess.stats().step_s * 1e3:.1f} ms/step")
        return out

    # a configuration without a device budget keeps its weights on the device
    # across the steps of a global batch (the host model changes only at the
    # update between global batches)
    resident = budget >= (1 << 49) and args.schedule == "atom"
    retain = args.retain or (resident and not args.no_retain)
    # row-sparse embedding transfers (retention keeps group 0 across steps,
    # which needs the whole matrix on the device)
    emb_rows = not args.dense_embedding and not retain
    if emb_rows:
        sess.set_embedding_rows(True)
    if retain:
        sess.set_retention(True)
    if args.warmup:
        losses = run(args.warmup)
        log(f"warmup: losses {[round(l, 5) for l in losses]}")

    if args.copy_calibration:
        n = (args.copy_calibration + 15) // 16 * 16
        src = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty(n, dtype=torch.uint8, device="cuda")
        A.atom_k_copy(src.data_ptr(), dst.data_ptr(), n, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        log(f"calibration copy of {n} bytes done")
        del src, dst

    # dominant kernel: weight-gradient GEMM (A and B not k-contiguous)
    # (bf16 at C = 1 writes bf16 gradients; otherwise micro-batch 0 stores fp32)
    wgrad_epi = A.ATOM_EPI_STORE if (cfg.accum == 1 and cfg.dtype == "bf16") else A.ATOM_EPI_STORE_F32
    A.atom_probe_gemm(sess.ctx, 0, 0, wgrad_epi)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    losses = run(args.steps)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    launches, probe_s, probe_flops, probe_bytes = A.atom_probe_read(sess.ctx)
    A.atom_probe_gemm(sess.ctx, 0, 0, -1)
    st = sess.stats()
    log(f"timed {args.steps} steps: {elapsed / args.steps * 1e3:.1f} ms/step, loss {losses[-1]:.5f}, "
        f"host accumulate {st.host_accum_s * 1e3:.1f} ms")
    if not all(math.isfinite(l) for l in losses):
        raise RuntimeError(f"non-finite loss: {losses}")

    # the schedule model's prediction of this call and of one step alone
    # (measured node costs, measured link sharing; with only the used
    # embedding rows moved, node 0's copy times scaled to the bytes moved)
    pcosts = costs
    if emb_rows:
        src = A.costs_array(costs)
        pcosts = (A.atom_node_cost * len(src))(*src)  # a copy
        row_b = cfg.d_model * (2 if cfg.dtype == "bf16" else 4)
        n0 = pcosts[0].weight_bytes
        moved0 = n0 - (cfg.vocab - np.mean([len(np.unique(tokens[i][..., :-1])) for i in range(args.steps)])) * row_b
        pcosts[0].t_load *= moved0 / n0
        pcosts[0].t_store *= moved0 / n0
    ends, _ = A.atom_plan_predict(c, plan, pcosts, duplex, min(args.steps, A.MAX_STEPS_PER_CALL), retain=retain)
    pred_call = ends[-1] / len(ends)
    pred_one = A.atom_plan_predict(c, plan, pcosts, duplex, 1)[0][0]
    steady = ((ends[-1] - ends[-3]) / 2.0) if len(ends) >= 3 else None
    steady_txt = f"{steady * 1e3:.1f} ms" if steady is not None else "needs 3 steps"
    log(f"predicted {pred_call * 1e3:.1f} ms per step of the call (steady {steady_txt}), "
        f"{pred_one * 1e3:.1f} ms for one step alone")

    # Parity of the timed path: the last timed step's gradients and loss
    # against one atom_step (no cross-step pipelining, nothing resident at its
    # start) on the same tokens, bitwise.
    t0 = time.perf_counter()
    dig_timed = host_digests(sess, A.GRAD_LAST)
    loss_seq = sess.step(tokens[args.steps - 1])
    dig_seq = host_digests(sess, A.GRAD_LAST)
    grad_check = {"kind": "last timed step vs one atom_step on the same tokens, bitwise",
                  "loss_equal": bool(loss_seq == losses[-1]),
                  "grads_equal": dig_timed == dig_seq,
                  "nodes_differing": [i for i, (a, b) in enumerate(zip(dig_timed, dig_seq)) if a != b],
                  "check_s": round(time.perf_counter() - t0, 2)}
    log(f"parity check of the timed path: {grad_check}")
    if not (grad_check["loss_equal"] and grad_check["grads_equal"]):
        raise RuntimeError(f"the timed path differs from a single atom_step: {grad_check}")

    # The survey-literal reading of a step: each step on its own (no weights
    # resident at its start, the next step's loads not overlapping this step's
    # gradient drain).  Timed over a few steps beside the pipelined headline.
    seq_ms = None
    if not args.sequential and args.seq_steps > 0:
        times = []
        for i in range(args.seq_steps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            sess.step(tokens[i % len(tokens)])
            torch.cuda.synchronize()
            times.append(time.perf_counter() - t0)
        seq_ms = sorted(times)[len(times) // 2] * 1e3
        log(f"sequential steps: {[round(t * 1e3, 1) for t in times]} ms (median {seq_ms:.1f})")

    ms_per_step = elapsed / args.steps * 1e3
    n_tok = cfg.accum * cfg.batch * cfg.seq_len
    tokens_per_s = n_tok / (ms_per_step / 1e3)
    peak = MFMA_PEAK_TFLOPS[cfg.dtype]
    achieved = probe_flops / probe_s / 1e12 if probe_s > 0 else 0.0
    alg_bytes = probe_bytes / max(launches, 1)
    traffic = None
    default_workload = args.config == "6.7b" and cfg.accum == 1 and not args.budget_gb
    if default_workload and WGRAD_TRAFFIC["bytes_per_launch"] and \
            WGRAD_TRAFFIC["sources_sha256"] == kernel_sources_sha256():
        traffic = WGRAD_TRAFFIC["bytes_per_launch"]
    fl = step_flops(cfg)
    t_mfma = fl / (peak * 1e12)
    # R0 counts the bytes the configuration forces, whatever the schedule
    # loads: the whole model, less the embedding rows no token of the step
    # uses when only used rows are moved (averaged over the timed steps), or
    # once per call when the weights are retained
    forced_h2d = (A.atom_plan_partition(A.make_config(cfg), budget).forced_h2d_bytes if args.schedule == "paper"
                  else plan.forced_h2d_bytes)
    row_bytes = cfg.d_model * (2 if cfg.dtype == "bf16" else 4)
    rows_used = [len(np.unique(tokens[i][..., :-1])) for i in range(args.steps)]
    unused_bytes = (cfg.vocab - float(np.mean(rows_used))) * row_bytes if emb_rows else 0.0
    forced_h2d = forced_h2d - unused_bytes
    if retain and not args.sequential:
        # weights retained across the steps of a call: one load per call
        forced_h2d *= math.ceil(args.steps / A.MAX_STEPS_PER_CALL) / args.steps
    forced_h2d = int(round(forced_h2d))
    t_h2d_r0 = forced_h2d / (h2d_gbs * 1e9)
    r0 = max(t_mfma, t_h2d_r0)
    # the bytes the timed steps moved each way (the plan's, less the embedding
    # rows they did not need; with retention, the call's loads over its steps)
    # (the stats are the last call's: one step per call with --sequential)
    last_call_steps = 1 if args.sequential else (args.steps - 1) % A.MAX_STEPS_PER_CALL + 1
    h2d_step, d2h_step = st.h2d_bytes / last_call_steps, st.d2h_bytes / last_call_steps
    # R1: R0 with the bytes the schedule moved in
    t_h2d_r1 = h2d_step / (h2d_gbs * 1e9)
    t_link_floor = max(h2d_step / (h2d_gbs * 1e9), d2h_step / (d2h_gbs * 1e9),
                       (h2d_step + d2h_step) / (bidir_gbs * 1e9))

    result = {
        "metric": "training tokens/sec on 1 MI355X (swapped); % of max(MFMA, H2D) roofline",
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded N(0,0.02) weights, uniform tokens)",
        "config": {
            "workload": (("[layer count overridden for profiling] " if args.layers else "")
                         + f"GPT-3 {args.config} swapped training step: {cfg.n_layer} layers, d_model {cfg.d_model}, "
                         f"{cfg.n_head} heads, MLP {cfg.d_mlp}, vocab {cfg.vocab}; batch {cfg.batch} x seq "
                         f"{cfg.seq_len}, accum {cfg.accum}; "
                         + ("one step per call; " if args.sequential else
                            f"{args.steps} steps of one global batch in one pipelined call; ")
                         + (f"device budget {budget / 1e9:.0f} GB" if budget < (1 << 49) else "whole model resident")
                         + ("; paper schedule (one node per group, two weight slots)" if args.schedule == "paper"
                            else "")
                         + ("; weights retained across the steps of the call" if retain else "")
                         + ("; only the embedding rows a step's tokens use cross the host link" if emb_rows
                            else "")
                         + ("; block-input checkpoints in host memory" if cfg.ckpt_host else "")),
            "global_batch": args.steps * cfg.accum * cfg.batch,
            "global_batch_unit": "sequences (timed steps x accum x batch)",
            "micro_batch": cfg.batch,
            "seq_len": cfg.seq_len,
            "accum": cfg.accum,
            "device_budget_gb": round(budget / 1e9, 2) if budget < (1 << 49) else None,
            "parallelism": "single GPU",
        },
        "roofline": {
            "bound": "mfma",
            "kernel": wgrad_kernel_name(cfg, wgrad_epi),
            "achieved": round(achieved, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": traffic,
            "alg_bytes_per_launch": round(alg_bytes),
            "launches": launches,
            "avg_launch_us": round(probe_s / max(launches, 1) * 1e6, 2),
        },
        "step_roofline": {
            "flops_per_step": fl,
            "t_mfma_s": t_mfma,
            "forced_h2d_bytes": forced_h2d,
            "plan_h2d_bytes": plan.h2d_bytes,
            "d2h_bytes": plan.d2h_bytes,
            "moved_h2d_bytes_per_step": round(h2d_step),
            "moved_d2h_bytes_per_step": round(d2h_step),
            "h2d_gbs": round(h2d_gbs, 2),
            "d2h_gbs": round(d2h_gbs, 2),
            "bidir_gbs": round(bidir_gbs, 2),
            "t_h2d_s": t_h2d_r0,
            "bound": "mfma" if t_mfma >= t_h2d_r0 else "h2d",
            "frac_r0": round(r0 / (ms_per_step / 1e3), 4),
            "frac_r1": round(max(t_mfma, t_h2d_r1) / (ms_per_step / 1e3), 4),
            # the host link with both directions counted: weights in, gradients
            # out, each alone and both at once (pipelined steps overlap them)
            "t_link_floor_s": t_link_floor,
            "frac_link_floor": round(t_link_floor / (ms_per_step / 1e3), 4),
            "host_accum_ms": round(st.host_accum_s * 1e3, 2),
        },
        "sequential_step": None if seq_ms is None else {
            "steps": args.seq_steps,
            "ms_per_step": round(seq_ms, 3),
            "tokens_per_s": round(n_tok / (seq_ms / 1e3), 1),
            "frac_r0": round(r0 / (seq_ms / 1e3), 4),
            "note": "each step alone: no weights resident at its start, the next step's loads do not overlap "
                    "its gradient drain",
        },
        "grad_check": grad_check,
        "prediction": {
            "model": "event model of the schedule (compute stream, two DMA engines sharing the host link)",
            "costs": "measured node costs (atom_profile_nodes) and the measured link sharing"
                     + ("; node 0's copies scaled to the embedding rows moved" if emb_rows else "")
                     + ("; weights retained: only the call's first step loads" if retain else ""),
            "duplex": round(duplex, 4),
            "pred_ms_per_step": round(pred_call * 1e3, 1),
            "measured_ms_per_step": round(elapsed / args.steps * 1e3, 1),
            "err": round(pred_call / (elapsed / args.steps) - 1.0, 4),
            "pred_steady_ms": None if steady is None else round(steady * 1e3, 1),
            "pred_one_step_ms": round(pred_one * 1e3, 1),
            "measured_one_step_ms": None if seq_ms is None else round(seq_ms, 1),
            "err_one_step": None if seq_ms is None else round(pred_one / (seq_ms / 1e3) - 1.0, 4),
        },
        "embedding_rows": {"row_sparse": emb_rows, "rows_per_step": round(float(np.mean(rows_used)), 1),
                           "vocab": cfg.vocab, "bytes_not_moved_per_step_each_way": round(unused_bytes)},
        "link_fit": fit,
        "plan": {"groups": plan.n_groups, "slots": plan.n_slots, "slot_mb": round(plan.slot_bytes / 1e6, 1),
                 "arena_gb": round(plan.arena_bytes / 1e9, 3), "pred_step_ms": round(plan.pred_step_s * 1e3, 1),
                 **plan_info},
        "loss": losses[-1],
    }
    if retain:
        # loads amortised over the call; the gradients still leave every step
        t_link = max(h2d_step / (h2d_gbs * 1e9), d2h_step / (d2h_gbs * 1e9))
        result["retention"] = {
            "h2d_bytes_per_step": round(h2d_step),
            "d2h_bytes_per_step": round(d2h_step),
            "t_link_s": t_link,
            "bound": "mfma" if t_mfma >= t_link else "link",
            "frac": round(max(t_mfma, t_link) / (ms_per_step / 1e3), 4),
        }
    if args.optimizer:
        A.atom_probe_gemm(sess.ctx, 0, 0, -1)
        t0 = time.perf_counter()
        A.atom_optimizer_init(sess.ctx)
        t_init = time.perf_counter() - t0
        t0 = time.perf_counter()
        A.atom_optimizer_step(sess.ctx, 1e-4, 1.0 / args.steps, 1)
        t_opt = time.perf_counter() - t0
        n_par = synthetic.param_count(cfg)
        log(f"host AdamW over {n_par / 1e9:.2f} B parameters: {t_opt:.2f} s (init {t_init:.2f} s)")
        # one global batch, then the update (the paper's order) ...
        t0 = time.perf_counter()
        run(args.steps)
        t_mid = time.perf_counter()
        A.atom_optimizer_step(sess.ctx, 1e-4, 1.0 / args.steps, 2)
        t_after = time.perf_counter() - t0
        t_upd = time.perf_counter() - t_mid
        # ... and one with the update armed: each group is updated as soon as
        # its last gradients of the global batch are accumulated
        t0 = time.perf_counter()
        run(args.steps, arm=lambda: A.atom_optimizer_arm(sess.ctx, 1e-4, 1.0 / args.steps, 3))
        t_armed = time.perf_counter() - t0
        st_arm = sess.stats()
        tok_gb = cfg.tokens_per_step * args.steps
        result["optimizer"] = {
            "kind": "host AdamW (fp32 master and moments), once per global batch",
            "state_memory": "pinned" if st_arm.opt_state_pinned else "pageable (the system refused to pin it)",
            "init_s": round(t_init, 3), "step_s": round(t_opt, 3), "params": n_par,
            "host_gbs": round(n_par * 34 / t_opt / 1e9, 1),
            "global_batch_steps": args.steps,
            "global_batch_then_update_s": round(t_after, 3), "update_after_s": round(t_upd, 3),
            "global_batch_armed_update_s": round(t_armed, 3),
            "armed_update_host_s": round(st_arm.host_update_s, 3), "armed_groups": st_arm.updated_groups,
            "tokens_per_s_update_after": round(tok_gb / t_after, 1),
            "tokens_per_s_update_armed": round(tok_gb / t_armed, 1)}
        log(f"global batch + update: {t_after:.2f} s (update {t_upd:.2f} s); armed: {t_armed:.2f} s "
            f"(update work {st_arm.host_update_s:.2f} s over {st_arm.updated_groups} groups)")
    sess.close()
    if not args.no_cpu_baseline:
        log("timing the oracle on the host (cpu_baseline)")
        result["cpu_baseline"] = cpu_baseline(cfg)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
