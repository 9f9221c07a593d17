"""Plant plausible mistakes in the oracle and check that the pins catch them.

Each mutation replaces one oracle function with a subtly wrong copy (a dropped
term, a wrong sign, a wrong scale, a missing mask) and the finite-difference
or library cross-check must then fail.  Mutations are planted on the CPU only.
"""
import numpy as np
import pytest

from oracle import gpt
from tests.test_oracle_gpt import FD_CFG, rand_tokens, rand_weights, torch_reference_step


def fd_max_rel_error(cfg, w, tok, n_pick=3, seed=0):
    _, grads = gpt.step(cfg, w, tok)
    rng = np.random.default_rng(seed)
    worst = 0.0
    h = 1e-6
    for node in range(cfg.n_nodes):
        for name in w[node]:
            flat = w[node][name].reshape(-1)
            for idx in rng.choice(flat.size, size=min(n_pick, flat.size), replace=False):
                old = flat[idx]
                flat[idx] = old + h
                lp, _ = gpt.step(cfg, w, tok)
                flat[idx] = old - h
                lm, _ = gpt.step(cfg, w, tok)
                flat[idx] = old
                an = grads[node][name].reshape(-1)[idx]
                worst = max(worst, abs((lp - lm) / (2 * h) - an) / (abs(an) + 1e-6))
    return worst


def _ln_bwd_dropped_term(dy, xhat, rstd, g):
    gp = dy * g
    dx = rstd * (gp - gp.mean(axis=-1, keepdims=True))
    rows = tuple(range(dy.ndim - 1))
    return dx, (dy * xhat).sum(axis=rows), dy.sum(axis=rows)


def _attn_bwd_wrong_sign(do, q, k, v, P):
    dh = q.shape[1]
    dP = do @ v.T
    dS = P * (dP + (dP * P).sum(axis=1, keepdims=True))
    s = 1.0 / np.sqrt(dh)
    return dS @ k * s, dS.T @ q * s, P.T @ do


def _gelu_grad_dropped_term(u):
    t = np.tanh(gpt.GELU_C * (u + gpt.GELU_A * u ** 3))
    return 0.5 * (1.0 + t)


def _probs_unscaled(q, k):
    T = q.shape[0]
    s = q @ k.T
    P = np.zeros((T, T))
    lse = np.empty(T)
    for i in range(T):
        e = np.exp(s[i, : i + 1] - s[i, : i + 1].max())
        P[i, : i + 1] = e / e.sum()
        lse[i] = 0.0
    return P, lse


def _probs_unmasked(q, k):
    s = (q @ k.T) / np.sqrt(q.shape[1])
    e = np.exp(s - s.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True), np.zeros(q.shape[0])


def _linear_bwd_transposed(dy, x, w):
    dx = dy @ w
    dy2 = dy.reshape(-1, dy.shape[-1])
    x2 = x.reshape(-1, x.shape[-1])
    dw = dy2.T @ x2
    if dw.shape[0] == dw.shape[1]:
        dw = dw.T
    return dx, dw, dy2.sum(axis=0)


def test_unmutated_oracle_passes_fd():
    assert fd_max_rel_error(FD_CFG, rand_weights(FD_CFG), rand_tokens(FD_CFG)) < 1e-5


@pytest.mark.parametrize("name,fn", [
    ("layer_norm_backward", _ln_bwd_dropped_term),
    ("attention_head_backward", _attn_bwd_wrong_sign),
    ("gelu_grad", _gelu_grad_dropped_term),
    ("linear_backward", _linear_bwd_transposed),
])
def test_fd_catches_backward_mutation(monkeypatch, name, fn):
    monkeypatch.setattr(gpt, name, fn)
    assert fd_max_rel_error(FD_CFG, rand_weights(FD_CFG), rand_tokens(FD_CFG)) > 1e-3


@pytest.mark.parametrize("fn", [_probs_unscaled, _probs_unmasked])
def test_library_cross_check_catches_forward_mutation(monkeypatch, fn):
    cfg = FD_CFG
    w = rand_weights(cfg, seed=11)
    tok = rand_tokens(cfg, seed=12)
    tloss, _ = torch_reference_step(cfg, w, tok)
    monkeypatch.setattr(gpt, "attention_probs", fn)
    loss, _ = gpt.step(cfg, w, tok)
    assert abs(loss - tloss) > 1e-6
