"""Pins of the fp64 GPT oracle against things other than itself.

* central finite differences of the loss (every parameter tensor, both
  micro-batches of an accumulated step);
* PyTorch fp64 autograd built from library routines (layer_norm, tanh GELU,
  scaled_dot_product_attention with is_causal, cross_entropy);
* closed forms and special cases: zero LM head gives loss ln V exactly, zero
  block weights give the identity block, T = 1 attention returns v, a
  constant LayerNorm row returns the shift, GELU(0) = 0 and GELU'(0) = 1/2;
* invariants: softmax rows sum to 1, causal invariance (changing later tokens
  leaves earlier outputs bit-identical), LayerNorm input gradients sum to 0
  per row, wpe gradients are batch sums.
"""
import math

import numpy as np
import pytest

from oracle import gpt
from synthetic import Config, gen_tokens, gen_weights, param_specs

FD_CFG = Config("fd", n_layer=2, d_model=8, n_head=2, d_mlp=32, vocab=13, seq_len=5, batch=2, accum=2, dtype="f32")


def rand_weights(cfg, seed=0, std=0.5):
    rng = np.random.default_rng(seed)
    ws = []
    for node in range(cfg.n_nodes):
        p = {}
        for name, shape, init in param_specs(cfg, node):
            if init == "one":
                p[name] = 1.0 + 0.3 * rng.standard_normal(shape)
            else:
                p[name] = std * rng.standard_normal(shape)
        ws.append(p)
    return ws


def rand_tokens(cfg, seed=1):
    rng = np.random.default_rng(seed)
    return rng.integers(0, cfg.vocab, size=(cfg.accum, cfg.batch, cfg.seq_len + 1)).astype(np.int32)


def test_finite_differences_every_tensor():
    cfg = FD_CFG
    w = rand_weights(cfg)
    tok = rand_tokens(cfg)
    loss, grads = gpt.step(cfg, w, tok)
    rng = np.random.default_rng(7)
    h = 1e-6
    for node in range(cfg.n_nodes):
        for name in w[node]:
            arr = w[node][name]
            flat = arr.reshape(-1)
            picks = rng.choice(flat.size, size=min(6, flat.size), replace=False)
            for idx in picks:
                old = flat[idx]
                flat[idx] = old + h
                lp, _ = gpt.step(cfg, w, tok)
                flat[idx] = old - h
                lm, _ = gpt.step(cfg, w, tok)
                flat[idx] = old
                fd = (lp - lm) / (2 * h)
                an = grads[node][name].reshape(-1)[idx]
                assert abs(fd - an) <= 1e-6 * abs(an) + 2e-9, (node, name, idx, fd, an)


def test_fd_wte_rows_of_used_and_unused_tokens():
    cfg = FD_CFG
    w = rand_weights(cfg, seed=3)
    tok = rand_tokens(cfg, seed=4)
    _, grads = gpt.step(cfg, w, tok)
    used = set(tok[:, :, :-1].reshape(-1).tolist())
    unused = [v for v in range(cfg.vocab) if v not in used]
    for v in unused:
        assert np.all(grads[0]["wte"][v] == 0.0)
    v = sorted(used)[0]
    h = 1e-6
    for col in range(cfg.d_model):
        old = w[0]["wte"][v, col]
        w[0]["wte"][v, col] = old + h
        lp, _ = gpt.step(cfg, w, tok)
        w[0]["wte"][v, col] = old - h
        lm, _ = gpt.step(cfg, w, tok)
        w[0]["wte"][v, col] = old
        assert abs((lp - lm) / (2 * h) - grads[0]["wte"][v, col]) < 1e-8


def torch_logits(cfg, P, inp):
    """Logits [B, T, V] of the model from PyTorch library routines (fp64)."""
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    L, d, H = cfg.n_layer, cfg.d_model, cfg.n_head
    dh = d // H
    B, T = inp.shape
    x = P[0]["wte"][inp] + P[0]["wpe"][:T][None]
    for l in range(L):
        p = P[1 + l]
        a = F.layer_norm(x, (d,), p["ln1_g"], p["ln1_b"], eps=1e-5)
        qkv = F.linear(a, p["w_qkv"], p["b_qkv"])
        q, k, v = qkv.split(d, dim=-1)
        q = q.reshape(B, T, H, dh).transpose(1, 2)
        k = k.reshape(B, T, H, dh).transpose(1, 2)
        v = v.reshape(B, T, H, dh).transpose(1, 2)
        o = F.scaled_dot_product_attention(q, k, v, is_causal=True)
        o = o.transpose(1, 2).reshape(B, T, d)
        x = x + F.linear(o, p["w_o"], p["b_o"])
        c = F.layer_norm(x, (d,), p["ln2_g"], p["ln2_b"], eps=1e-5)
        x = x + F.linear(F.gelu(F.linear(c, p["w_fc"], p["b_fc"]), approximate="tanh"), p["w_pr"], p["b_pr"])
    p = P[L + 1]
    return F.linear(F.layer_norm(x, (d,), p["lnf_g"], p["lnf_b"], eps=1e-5), p["w_head"])


def torch_reference_step(cfg, w, tok):
    """The same model from PyTorch library routines, fp64 autograd."""
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    P = [{k: torch.tensor(np.asarray(v, np.float64), requires_grad=True) for k, v in p.items()} for p in w]
    C, B, T1 = tok.shape
    T = T1 - 1
    total = 0.0
    for m in range(C):
        inp = torch.tensor(tok[m, :, :T].astype(np.int64))
        tgt = torch.tensor(tok[m, :, 1:].astype(np.int64))
        z = torch_logits(cfg, P, inp)
        total = total + F.cross_entropy(z.reshape(-1, cfg.vocab), tgt.reshape(-1), reduction="sum")
    loss = total / (C * B * T)
    loss.backward()
    return float(loss.detach()), [{k: t.grad.numpy() for k, t in p.items()} for p in P]


def test_forward_logits_matches_torch_fp64():
    torch = pytest.importorskip("torch")
    cfg = FD_CFG
    w = rand_weights(cfg, seed=21)
    tok = rand_tokens(cfg, seed=22)
    inp = tok[0, :, :cfg.seq_len]
    got = gpt.forward_logits(cfg, w, inp)
    P = [{k: torch.tensor(np.asarray(v, np.float64)) for k, v in p.items()} for p in w]
    ref = torch_logits(cfg, P, torch.tensor(inp.astype(np.int64))).numpy()
    assert got.shape == ref.shape == (cfg.batch, cfg.seq_len, cfg.vocab)
    assert np.max(np.abs(got - ref)) <= 1e-12 * np.max(np.abs(ref))


@pytest.mark.parametrize("cfg", [FD_CFG, FD_CFG.with_(batch=1, accum=1, seq_len=9, n_layer=1, n_head=4, d_model=16, d_mlp=64, vocab=31)])
def test_matches_torch_fp64_autograd(cfg):
    w = rand_weights(cfg, seed=11)
    tok = rand_tokens(cfg, seed=12)
    loss, grads = gpt.step(cfg, w, tok)
    tloss, tgrads = torch_reference_step(cfg, w, tok)
    assert abs(loss - tloss) < 1e-12 * max(1.0, abs(tloss))
    for node in range(cfg.n_nodes):
        for name, g in grads[node].items():
            ref = tgrads[node][name]
            err = np.max(np.abs(g - ref))
            assert err <= 1e-11 * max(1e-3, np.max(np.abs(ref))), (node, name, err)


def test_zero_head_gives_ln_vocab_exactly():
    for V in (1024, 50257, 13):
        cfg = FD_CFG.with_(vocab=V)
        w = rand_weights(cfg, seed=5)
        w[-1]["w_head"][:] = 0.0
        tok = rand_tokens(cfg, seed=6)
        loss, grads = gpt.step(cfg, w, tok)
        assert loss == pytest.approx(math.log(V), rel=0, abs=1e-12)
        # dz rows sum to zero, so the final-LN input gradient is exactly zero with W_head = 0
        assert np.max(np.abs(grads[-1]["lnf_g"])) == 0.0
    assert math.log(1024) == pytest.approx(6.931471805599453, abs=1e-15)
    assert math.log(50257) == pytest.approx(10.82490511970208, abs=1e-13)


def test_loss_at_init_near_ln_vocab():
    cfg = Config("tiny", 2, 256, 4, 1024, 1024, 128, 2, 1, "f32")
    w = gen_weights(cfg)
    tok = gen_tokens(cfg)
    loss, _ = gpt.step(cfg, w, tok)
    # z = LN(x) W_head^T has variance ~ 0.02^2 * d, so E[loss] ~ ln V + var/2
    assert abs(loss - (math.log(1024) + 0.5 * 0.02 ** 2 * 256)) < 0.05


def test_zero_block_is_identity():
    cfg = FD_CFG
    w = rand_weights(cfg, seed=8)
    p = {k: np.zeros_like(v) for k, v in w[1].items()}
    x = np.random.default_rng(0).standard_normal((2, 5, 8))
    out, _ = gpt.block_forward(x, p, cfg.n_head)
    assert np.array_equal(out, x)


def test_single_token_attention_returns_v():
    rng = np.random.default_rng(1)
    q, k, v = rng.standard_normal((3, 1, 16))
    o, P, lse = gpt.attention_head(q, k, v)
    assert np.array_equal(o, v) and P[0, 0] == 1.0
    assert lse[0] == pytest.approx(float(q[0] @ k[0]) / 4.0, abs=1e-15)


def test_softmax_rows_sum_to_one_and_mask():
    rng = np.random.default_rng(2)
    q, k = rng.standard_normal((2, 37, 64)) * 3
    P, _ = gpt.attention_probs(q, k)
    assert np.max(np.abs(P.sum(axis=1) - 1.0)) < 1e-12
    assert np.all(np.triu(P, 1) == 0.0)


def test_constant_layernorm_row_gives_shift():
    b = np.linspace(-1, 1, 10)
    y, _ = gpt.layer_norm(np.full((3, 10), 4.25), np.ones(10) * 2.0, b)
    assert np.allclose(y, b, atol=0, rtol=0)


def test_layernorm_input_grad_rows_sum_to_zero():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((6, 20))
    g = rng.standard_normal(20)
    _, (xhat, rstd) = gpt.layer_norm(x, g, rng.standard_normal(20))
    dx, _, _ = gpt.layer_norm_backward(rng.standard_normal((6, 20)), xhat, rstd, g)
    assert np.max(np.abs(dx.sum(axis=1))) < 1e-13


def test_gelu_special_values_and_derivative():
    assert gpt.gelu(np.float64(0.0)) == 0.0
    assert gpt.gelu_grad(np.float64(0.0)) == 0.5
    u = np.linspace(-6, 6, 101)
    h = 1e-6
    fd = (gpt.gelu(u + h) - gpt.gelu(u - h)) / (2 * h)
    assert np.max(np.abs(fd - gpt.gelu_grad(u))) < 1e-8
    # large |u|: GELU -> relu
    assert gpt.gelu(np.float64(30.0)) == 30.0 and gpt.gelu(np.float64(-30.0)) == 0.0


def test_causal_invariance_bit_identical():
    cfg = FD_CFG.with_(seq_len=8)
    w = rand_weights(cfg, seed=9)
    tok = rand_tokens(cfg, seed=10)[0, :, :8]
    z0 = gpt.forward_logits(cfg, w, tok)
    t0 = 4
    tok2 = tok.copy()
    tok2[:, t0 + 1:] = (tok2[:, t0 + 1:] + 5) % cfg.vocab
    z1 = gpt.forward_logits(cfg, w, tok2)
    assert np.array_equal(z0[:, : t0 + 1], z1[:, : t0 + 1])
    assert not np.array_equal(z0[:, t0 + 1:], z1[:, t0 + 1:])


def test_embedding_backward_sums():
    rng = np.random.default_rng(4)
    tok = np.array([[1, 2, 1], [2, 2, 0]])
    dx = rng.standard_normal((2, 3, 4))
    g = gpt.embed_backward(dx, tok, 5, 6)
    assert np.allclose(g["wpe"][:3], dx.sum(axis=0), rtol=0, atol=1e-15)
    assert np.all(g["wpe"][3:] == 0)
    assert np.allclose(g["wte"][2], dx[0, 1] + dx[1, 0] + dx[1, 1], rtol=0, atol=1e-15)
    assert np.all(g["wte"][3:] == 0)


def test_accumulated_step_is_mean_over_micro_batches():
    cfg = FD_CFG
    w = rand_weights(cfg, seed=13)
    tok = rand_tokens(cfg, seed=14)
    loss, grads = gpt.step(cfg, w, tok)
    one = cfg.with_(accum=1)
    l0, g0 = gpt.step(one, w, tok[:1])
    l1, g1 = gpt.step(one, w, tok[1:])
    assert loss == pytest.approx((l0 + l1) / 2, abs=1e-14)
    for node in range(cfg.n_nodes):
        for k in grads[node]:
            assert np.allclose(grads[node][k], (g0[node][k] + g1[node][k]) / 2, rtol=1e-12, atol=1e-15)
