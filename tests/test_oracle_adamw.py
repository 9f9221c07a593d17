"""Pins of the AdamW oracle: torch's AdamW (fp64, CPU) on the same tensors,
the closed form of the first step, pure decoupled decay at zero gradient, and
the linear warm-up."""
import numpy as np
import pytest

from oracle import adamw as O


def torch_adamw(p0, grads, lr, wd, betas=(0.9, 0.999), eps=1e-8):
    import torch

    p = torch.tensor(p0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([p], lr=lr, betas=betas, eps=eps, weight_decay=wd)
    for g in grads:
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
    return p.detach().numpy()


@pytest.mark.parametrize("wd", [0.0, 0.1])
def test_matches_torch_adamw_over_several_steps(wd):
    r = np.random.default_rng(4)
    p0 = r.standard_normal(257)
    grads = [r.standard_normal(257) * s for s in (1.0, 0.1, 3.0, 1e-3, 0.5)]
    lrs = 1e-3
    p, m, v = p0.copy(), np.zeros(257), np.zeros(257)
    for t, g in enumerate(grads, start=1):
        p, m, v = O.adamw_step(p, g, m, v, t, lrs, wd=wd)
    ref = torch_adamw(p0, grads, lrs, wd)
    np.testing.assert_allclose(p, ref, rtol=0, atol=1e-13)


def test_first_step_closed_form():
    # t = 1: mhat = g, vhat = g^2, so the update is lr * g / (|g| + eps)
    g = np.array([2.0, -3.0, 1e-9, 0.0, -1e-3])
    p, m, v = O.adamw_step(np.ones(5), g, np.zeros(5), np.zeros(5), 1, lr=0.01, eps=1e-8)
    np.testing.assert_allclose(p, 1.0 - 0.01 * g / (np.abs(g) + 1e-8), rtol=1e-15, atol=0)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-12)
    np.testing.assert_allclose(v, 0.001 * g * g, rtol=1e-12)  # 1 - 0.999 is not exactly 0.001


def test_zero_gradient_is_pure_decoupled_decay():
    p0 = np.array([1.0, -2.0, 0.5])
    p, m, v = O.adamw_step(p0, np.zeros(3), np.zeros(3), np.zeros(3), 7, lr=0.01, wd=0.1)
    np.testing.assert_allclose(p, p0 * (1 - 0.01 * 0.1), rtol=1e-15)
    assert not m.any() and not v.any()


def test_decay_rule_and_warmup():
    assert O.decayed("w_qkv") and O.decayed("w_head")
    assert not any(O.decayed(n) for n in ("b_qkv", "ln1_g", "lnf_b", "wte", "wpe"))
    assert O.warmup_lr(1, 1e-4, 3000) == pytest.approx(1e-4 / 3000)
    assert O.warmup_lr(3000, 1e-4, 3000) == 1e-4 and O.warmup_lr(5000, 1e-4, 3000) == 1e-4


def test_model_step_applies_decay_per_tensor():
    params = [{"w_o": np.ones((2, 2)), "b_o": np.ones(2)}]
    grads = [{"w_o": np.zeros((2, 2)), "b_o": np.zeros(2)}]
    new, state = O.model_step(params, grads, None, 1, lr=0.1, wd=0.5)
    np.testing.assert_allclose(new[0]["w_o"], 0.95)
    np.testing.assert_allclose(new[0]["b_o"], 1.0)
