"""Oracle: one GPT training step (forward + backward), plain NumPy fp64.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this
module; only the tests, the package's smoke entry and the CPU-baseline leg of
the benchmark use it.  It shares no code with the GPU path.

What it computes.  Atom swaps sub-models between host and device memory but
leaves the computation unchanged: the sub-models are the same graph cut at
decoder-block boundaries (Section III-B, "Memory swapping vs. network
transmission"; Section III-D, "Model compilation and code generation" states
that user code is not changed).  The result of a swapped step is therefore the
result of the plain GPT-3 training step, which this module writes out from its
definition.  The model is the minGPT GPT used for the paper's profiling
(Section III-B, footnote): a chain of an embedding, identical pre-LayerNorm
decoder blocks, and a final LayerNorm with the "Logits" layer (Section III-B,
layer loading; Section III-C, embedding).  Shapes follow Table II.

Readings where the paper is silent:
GELU in its tanh form; LayerNorm with biased variance and eps 1e-5; no
dropout; attention scale 1/sqrt(d_head) with a strict causal mask; biases on
every block linear, none on the LM head; the LM head is untied from the token
embedding; the loss is the mean next-token cross-entropy over all
accum*batch*seq_len targets.

Layout: linear weights are [out][in] and y = x W^T + b.  The fused QKV weight
holds q, k, v in that order along its output axis, each split into heads of
d_head consecutive features.

Everything is float64.  Memory is bounded by looping over (batch, head) in
attention and over token chunks in the LM head; a loop changes no arithmetic.
"""
from __future__ import annotations

import numpy as np

LN_EPS = 1e-5
GELU_C = np.sqrt(2.0 / np.pi)
GELU_A = 0.044715


# --------------------------------------------------------------------------
# LayerNorm (pre-LN decoder of the minGPT lineage, Section III-B footnote)
# --------------------------------------------------------------------------
def layer_norm(x, g, b, eps=LN_EPS):
    """y = (x - mean) / sqrt(var + eps) * g + b over the last axis (biased var).

    Returns y and the saved (xhat, rstd) needed by the backward.
    """
    x = np.asarray(x, np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mu) * rstd
    return xhat * g + b, (xhat, rstd)


def layer_norm_backward(dy, xhat, rstd, g):
    """Gradient of layer_norm.

    With g' = dy * g:  dx = rstd * (g' - mean(g') - xhat * mean(g' * xhat)),
    dgain = sum over rows of dy * xhat, dshift = sum over rows of dy.
    """
    gp = dy * g
    dx = rstd * (gp - gp.mean(axis=-1, keepdims=True)
                 - xhat * (gp * xhat).mean(axis=-1, keepdims=True))
    rows = tuple(range(dy.ndim - 1))
    return dx, (dy * xhat).sum(axis=rows), dy.sum(axis=rows)


# --------------------------------------------------------------------------
# GELU, tanh form
# --------------------------------------------------------------------------
def gelu(u):
    """GELU(u) = u/2 * (1 + tanh(sqrt(2/pi) * (u + 0.044715 u^3)))."""
    return 0.5 * u * (1.0 + np.tanh(GELU_C * (u + GELU_A * u ** 3)))


def gelu_grad(u):
    """d GELU / du for the tanh form."""
    s = GELU_C * (u + GELU_A * u ** 3)
    t = np.tanh(s)
    return 0.5 * (1.0 + t) + 0.5 * u * (1.0 - t * t) * GELU_C * (1.0 + 3.0 * GELU_A * u * u)


# --------------------------------------------------------------------------
# Causal self-attention, one (sequence, head) at a time
# --------------------------------------------------------------------------
def attention_probs(q, k):
    """P = softmax_row(q k^T / sqrt(dh)) with key j > query i excluded.

    q, k: [T, dh].  Returns P [T, T] (zeros above the diagonal) and the row
    log-sum-exp of the scaled, masked scores.
    """
    T, dh = q.shape
    s = (q @ k.T) / np.sqrt(dh)
    P = np.zeros((T, T))
    lse = np.empty(T)
    for i in range(T):
        row = s[i, : i + 1]
        m = row.max()
        e = np.exp(row - m)
        z = e.sum()
        P[i, : i + 1] = e / z
        lse[i] = m + np.log(z)
    return P, lse


def attention_head(q, k, v):
    """o = P v for one head.  Returns o [T, dh], P, lse."""
    P, lse = attention_probs(q, k)
    return P @ v, P, lse


def attention_head_backward(do, q, k, v, P):
    """Gradient of o = softmax(q k^T / sqrt(dh), causal) v.

    dP = do v^T;  dS = P * (dP - rowsum(dP * P));
    dq = dS k / sqrt(dh);  dk = dS^T q / sqrt(dh);  dv = P^T do.
    """
    dh = q.shape[1]
    dP = do @ v.T
    dS = P * (dP - (dP * P).sum(axis=1, keepdims=True))
    scale = 1.0 / np.sqrt(dh)
    return dS @ k * scale, dS.T @ q * scale, P.T @ do


def split_heads(qkv, n_head):
    """qkv [B, T, 3d] -> q, k, v as [B, n_head, T, dh]."""
    B, T, d3 = qkv.shape
    d = d3 // 3
    dh = d // n_head
    parts = []
    for c in range(3):
        parts.append(qkv[:, :, c * d:(c + 1) * d].reshape(B, T, n_head, dh).transpose(0, 2, 1, 3))
    return parts


def merge_heads(o):
    """[B, n_head, T, dh] -> [B, T, n_head*dh]."""
    B, H, T, dh = o.shape
    return o.transpose(0, 2, 1, 3).reshape(B, T, H * dh)


def causal_attention(qkv, n_head):
    """Multi-head causal attention on a fused qkv [B, T, 3d].  Returns o [B, T, d], lse [B, h, T]."""
    q, k, v = split_heads(qkv, n_head)
    B, H, T, dh = q.shape
    o = np.empty_like(q)
    lse = np.empty((B, H, T))
    for b in range(B):
        for h in range(H):
            o[b, h], _, lse[b, h] = attention_head(q[b, h], k[b, h], v[b, h])
    return merge_heads(o), lse


def causal_attention_backward(do, qkv, n_head):
    """Gradient of causal_attention w.r.t. the fused qkv.  do [B, T, d] -> dqkv [B, T, 3d]."""
    q, k, v = split_heads(qkv, n_head)
    B, H, T, dh = q.shape
    dO = do.reshape(B, T, H, dh).transpose(0, 2, 1, 3)
    dq = np.empty_like(q)
    dk = np.empty_like(k)
    dv = np.empty_like(v)
    for b in range(B):
        for h in range(H):
            P, _ = attention_probs(q[b, h], k[b, h])
            dq[b, h], dk[b, h], dv[b, h] = attention_head_backward(dO[b, h], q[b, h], k[b, h], v[b, h], P)
    return np.concatenate([merge_heads(dq), merge_heads(dk), merge_heads(dv)], axis=-1)


# --------------------------------------------------------------------------
# Linear layers
# --------------------------------------------------------------------------
def linear(x, w, b=None):
    """y = x W^T (+ b), W stored [out][in]."""
    y = x @ w.T
    return y if b is None else y + b


def linear_backward(dy, x, w):
    """dx = dy W, dW = dy^T x (summed over all leading axes), db = sum of dy rows."""
    dx = dy @ w
    dy2 = dy.reshape(-1, dy.shape[-1])
    x2 = x.reshape(-1, x.shape[-1])
    return dx, dy2.T @ x2, dy2.sum(axis=0)


# --------------------------------------------------------------------------
# Decoder block (pre-LN GPT block)
# --------------------------------------------------------------------------
def _p64(p):
    return {k: np.asarray(v, np.float64) for k, v in p.items()}


def block_forward(x, p, n_head):
    """One decoder block on the residual stream x [B, T, d].

    a = LN1(x); qkv = a W_qkv^T + b_qkv; o = causal attention;
    x1 = x + o W_o^T + b_o; c = LN2(x1); u = c W_fc^T + b_fc; g = GELU(u);
    out = x1 + g W_pr^T + b_pr.
    Returns out and the cache the backward needs.
    """
    p = _p64(p)
    a, ln1 = layer_norm(x, p["ln1_g"], p["ln1_b"])
    qkv = linear(a, p["w_qkv"], p["b_qkv"])
    o, lse = causal_attention(qkv, n_head)
    x1 = x + linear(o, p["w_o"], p["b_o"])
    c, ln2 = layer_norm(x1, p["ln2_g"], p["ln2_b"])
    u = linear(c, p["w_fc"], p["b_fc"])
    g = gelu(u)
    out = x1 + linear(g, p["w_pr"], p["b_pr"])
    cache = dict(x=x, a=a, ln1=ln1, qkv=qkv, o=o, lse=lse, x1=x1, c=c, ln2=ln2, u=u, g=g)
    return out, cache


def block_backward(dout, cache, p, n_head):
    """Backward of block_forward.  Returns dx and the parameter gradients."""
    p = _p64(p)
    gr = {}
    dg, gr["w_pr"], gr["b_pr"] = linear_backward(dout, cache["g"], p["w_pr"])
    du = dg * gelu_grad(cache["u"])
    dc, gr["w_fc"], gr["b_fc"] = linear_backward(du, cache["c"], p["w_fc"])
    dx1_ln, gr["ln2_g"], gr["ln2_b"] = layer_norm_backward(dc, *cache["ln2"], p["ln2_g"])
    dx1 = dout + dx1_ln
    do, gr["w_o"], gr["b_o"] = linear_backward(dx1, cache["o"], p["w_o"])
    dqkv = causal_attention_backward(do, cache["qkv"], n_head)
    da, gr["w_qkv"], gr["b_qkv"] = linear_backward(dqkv, cache["a"], p["w_qkv"])
    dx_ln, gr["ln1_g"], gr["ln1_b"] = layer_norm_backward(da, *cache["ln1"], p["ln1_g"])
    return dx1 + dx_ln, gr


# --------------------------------------------------------------------------
# Embedding (node 0) and LM head (node L+1)
# --------------------------------------------------------------------------
def embed_forward(tok, p):
    """x[b, t] = wte[tok[b, t]] + wpe[t].  tok [B, T] int."""
    wte = np.asarray(p["wte"], np.float64)
    wpe = np.asarray(p["wpe"], np.float64)
    T = tok.shape[1]
    return wte[tok] + wpe[None, :T]


def embed_backward(dx, tok, vocab, seq_len):
    """dwte[v] = sum of dx rows whose token is v; dwpe[t] = sum over the batch of dx[:, t]."""
    d = dx.shape[-1]
    dwte = np.zeros((vocab, d))
    np.add.at(dwte, tok.reshape(-1), dx.reshape(-1, d))
    dwpe = np.zeros((seq_len, d))
    dwpe[: dx.shape[1]] = dx.sum(axis=0)
    return {"wte": dwte, "wpe": dwpe}


def cross_entropy_rows(z, y, scale):
    """Per-row next-token cross-entropy and its gradient.

    loss[r] = logsumexp(z[r]) - z[r, y[r]];  dz = (softmax(z) - onehot(y)) * scale.
    """
    m = z.max(axis=1, keepdims=True)
    lse = (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))[:, 0]
    rows = np.arange(z.shape[0])
    loss = lse - z[rows, y]
    dz = np.exp(z - lse[:, None])
    dz[rows, y] -= 1.0
    return loss, dz * scale


def head_forward_backward(x, p, targets, n_total, chunk=4096):
    """Final LN, logits z = LN(x) W_head^T, cross-entropy against `targets`.

    Returns (sum over tokens of [logsumexp(z) - z[y]], dx, grads) where the
    gradients are those of the loss divided by `n_total` (the mean over all
    targets of the step): dz = (softmax(z) - onehot(y)) / n_total.
    Token chunks bound memory only.
    """
    p = _p64(p)
    B, T, d = x.shape
    xf = x.reshape(-1, d)
    yf = targets.reshape(-1)
    yhat, (xhat, rstd) = layer_norm(xf, p["lnf_g"], p["lnf_b"])
    W = p["w_head"]
    loss_sum = 0.0
    dyhat = np.empty_like(yhat)
    dW = np.zeros_like(W)
    for lo in range(0, xf.shape[0], chunk):
        hi = min(xf.shape[0], lo + chunk)
        z = yhat[lo:hi] @ W.T
        loss_rows, dz = cross_entropy_rows(z, yf[lo:hi], 1.0 / n_total)
        loss_sum += float(loss_rows.sum())
        dyhat[lo:hi] = dz @ W
        dW += dz.T @ yhat[lo:hi]
    dx, dg, db = layer_norm_backward(dyhat, xhat, rstd, p["lnf_g"])
    return loss_sum, dx.reshape(B, T, d), {"lnf_g": dg, "lnf_b": db, "w_head": dW}


# --------------------------------------------------------------------------
# Whole step
# --------------------------------------------------------------------------
def _zeros_like_params(p):
    return {k: np.zeros(np.shape(v)) for k, v in p.items()}


def step(cfg, weights, tokens):
    """One training step over `accum` micro-batches.

    weights: list over nodes of {name: array}; tokens: int [accum][B][T+1].
    Returns (mean loss, grads) where grads has the layout of `weights` and
    holds the gradient of the mean loss, summed over the micro-batches.
    """
    L = cfg.n_layer
    C, B, T1 = tokens.shape
    T = T1 - 1
    n_total = C * B * T
    grads = [_zeros_like_params(p) for p in weights]
    loss_sum = 0.0
    for m in range(C):
        inp = tokens[m, :, :T]
        tgt = tokens[m, :, 1:]
        x = embed_forward(inp, weights[0])
        caches = []
        for l in range(L):
            x, cache = block_forward(x, weights[1 + l], cfg.n_head)
            caches.append(cache)
        ls, dx, gh = head_forward_backward(x, weights[L + 1], tgt, n_total)
        loss_sum += ls
        for k, v in gh.items():
            grads[L + 1][k] += v
        for l in reversed(range(L)):
            dx, gb = block_backward(dx, caches[l], weights[1 + l], cfg.n_head)
            for k, v in gb.items():
                grads[1 + l][k] += v
        ge = embed_backward(dx, inp, cfg.vocab, cfg.seq_len)
        for k, v in ge.items():
            grads[0][k] += v
    return loss_sum / n_total, grads


def forward_logits(cfg, weights, inp):
    """Logits of one micro-batch, [B, T, V] (used by invariance tests)."""
    L = cfg.n_layer
    x = embed_forward(inp, weights[0])
    for l in range(L):
        x, _ = block_forward(x, weights[1 + l], cfg.n_head)
    p = _p64(weights[L + 1])
    yhat, _ = layer_norm(x, p["lnf_g"], p["lnf_b"])
    return yhat @ p["w_head"].T
