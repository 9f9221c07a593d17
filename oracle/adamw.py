"""Oracle: the host optimizer step, AdamW, plain NumPy fp64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

The paper trains with AdamW on the host CPUs once the global batch is
complete (Section V-B, convergence experiment: learning rate 1e-4 with a
warm-up of 3K steps, betas 0.9 and 0.999; Section III-E: the peers' updates
happen when the global batch is reached).  AdamW is Adam with the weight decay
decoupled from the gradient (Loshchilov and Hutter, "Decoupled Weight Decay
Regularization"): with step count t starting at 1,

    p <- p - lr * wd * p                       (only for decayed tensors)
    m <- beta1 * m + (1 - beta1) * g
    v <- beta2 * v + (1 - beta2) * g^2
    p <- p - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)

Readings where the paper is silent: the gradient g is the mean over the
global batch (the host accumulators hold the sum over its steps of each
step's mean-loss gradient, so g = accumulator / steps); weight decay applies
to the weight matrices of the linear layers (QKV, output, MLP and LM-head
weights) and not to biases, LayerNorm parameters or the embeddings, the rule
of the minGPT model the paper profiles; the warm-up is linear.
"""
from __future__ import annotations

import numpy as np

DECAYED = ("w_qkv", "w_o", "w_fc", "w_pr", "w_head")


def decayed(name: str) -> bool:
    """Whether weight decay applies to the tensor `name`."""
    return name in DECAYED


def warmup_lr(step: int, base_lr: float, warmup: int) -> float:
    """Linear warm-up to base_lr over `warmup` steps (step counts from 1)."""
    return base_lr * min(1.0, step / warmup) if warmup > 0 else base_lr


def adamw_step(p, g, m, v, t, lr, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0):
    """One AdamW update of one tensor (fp64 arrays).  Returns (p, m, v) new."""
    p = np.asarray(p, np.float64)
    g = np.asarray(g, np.float64)
    if wd:
        p = p - lr * wd * p
    m = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** t)
    vhat = v / (1.0 - beta2 ** t)
    p = p - lr * mhat / (np.sqrt(vhat) + eps)
    return p, m, v


def model_step(params, grads, state, t, lr, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0):
    """AdamW over a whole model: params and grads are lists over nodes of
    {name: array}; state is the same structure of (m, v) pairs (or None at the
    first step).  Returns new params and state."""
    new_p, new_s = [], []
    for node, p in enumerate(params):
        np_, ns = {}, {}
        for name, val in p.items():
            m, v = (np.zeros_like(val, dtype=np.float64),) * 2 if state is None else state[node][name]
            np_[name], mm, vv = adamw_step(val, grads[node][name], m, v, t, lr, beta1, beta2, eps,
                                           wd if decayed(name) else 0.0)
            ns[name] = (mm, vv)
        new_p.append(np_)
        new_s.append(ns)
    return new_p, new_s
