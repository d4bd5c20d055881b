"""Pins of the memory-bound-operator oracle (oracle/memops_oracle.py) against
facts that do not come from the oracle: hand-worked values, closed forms,
invariants, central finite differences of the forward, torch's float64
layer_norm / gelu / cross_entropy with autograd, the erf form of GELU within
the tanh form's approximation error, and planted mistakes that each trip at
least one of these checks."""

import math

import numpy as np
import pytest
import torch

import oracle.memops_oracle as mo


def _rand(shape, seed, sigma=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * sigma


# ---------------------------------------------------------------------------
# LayerNorm
# ---------------------------------------------------------------------------
def test_layernorm_two_columns_closed_form():
    # C = 2: mean (a+b)/2, biased variance ((a-b)/2)^2, so xhat = +-d / sqrt(d^2 + eps), d = (a-b)/2
    a, b, eps = 3.0, 1.0, 1e-5
    y, mu, rstd = mo.layernorm_fwd([[a, b]], [1.0, 1.0], [0.0, 0.0], eps)
    d = (a - b) / 2
    assert mu[0] == 2.0
    assert abs(rstd[0] - 1 / math.sqrt(d * d + eps)) <= 1e-15
    assert np.allclose(y, [[d / math.sqrt(d * d + eps), -d / math.sqrt(d * d + eps)]], rtol=0, atol=1e-15)


def test_layernorm_row_moments():
    x = _rand((6, 48), 1, 3.0) + 5.0
    y, mu, rstd = mo.layernorm_fwd(x, np.ones(48), np.zeros(48), 1e-5)
    var = x.var(axis=1)
    assert np.allclose(y.mean(axis=1), 0, atol=1e-14)
    assert np.allclose(y.var(axis=1), var / (var + 1e-5), rtol=1e-13)
    # affine part: y = xhat * gamma + beta column by column
    g, be = _rand(48, 2), _rand(48, 3)
    y2, _, _ = mo.layernorm_fwd(x, g, be, 1e-5)
    assert np.allclose(y2, y * g + be, rtol=0, atol=1e-13)


def test_layernorm_matches_torch_float64():
    x, g, be, dy = _rand((7, 40), 4, 2.0), _rand(40, 5), _rand(40, 6), _rand((7, 40), 7)
    xt = torch.tensor(x, requires_grad=True)
    gt = torch.tensor(g, requires_grad=True)
    bt = torch.tensor(be, requires_grad=True)
    yt = torch.nn.functional.layer_norm(xt, (40,), gt, bt, eps=1e-5)
    yt.backward(torch.tensor(dy))
    y, mu, rstd = mo.layernorm_fwd(x, g, be, 1e-5)
    dx, dg, db = mo.layernorm_bwd(x, g, dy, 1e-5)
    assert np.allclose(y, yt.detach().numpy(), rtol=0, atol=1e-12)
    assert np.allclose(dx, xt.grad.numpy(), rtol=0, atol=1e-12)
    assert np.allclose(dg, gt.grad.numpy(), rtol=0, atol=1e-12)
    assert np.allclose(db, bt.grad.numpy(), rtol=0, atol=1e-12)


def test_layernorm_finite_differences():
    x, g, be, dy = _rand((3, 6), 8), _rand(6, 9), _rand(6, 10), _rand((3, 6), 11)
    h = 1e-6

    def f(x_, g_, b_):
        return float((mo.layernorm_fwd(x_, g_, b_, 1e-5)[0] * dy).sum())

    dx, dg, db = mo.layernorm_bwd(x, g, dy, 1e-5)
    for arr, grad, which in ((x, dx, 0), (g, dg, 1), (be, db, 2)):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            p, m = arr.copy(), arr.copy()
            p[idx] += h
            m[idx] -= h
            args_p = [x, g, be]
            args_m = [x, g, be]
            args_p[which], args_m[which] = p, m
            num[idx] = (f(*args_p) - f(*args_m)) / (2 * h)
        assert np.allclose(grad, num, rtol=1e-6, atol=1e-7), which


def test_layernorm_dx_rows_sum_to_zero():
    # y is invariant to adding a constant to a row, so every row of dx sums to 0
    x, g, dy = _rand((5, 64), 12), _rand(64, 13), _rand((5, 64), 14)
    dx, _, db = mo.layernorm_bwd(x, g, dy, 1e-5)
    assert np.allclose(dx.sum(axis=1), 0, atol=1e-12)
    assert np.allclose(db, dy.sum(axis=0), rtol=0, atol=0)


# ---------------------------------------------------------------------------
# GELU
# ---------------------------------------------------------------------------
def test_gelu_special_values():
    assert mo.gelu_fwd(np.array([0.0]))[0] == 0.0
    assert abs(mo.gelu_bwd(np.array([0.0]), np.array([1.0]))[0] - 0.5) <= 1e-16
    big = np.array([30.0, -30.0])
    assert np.allclose(mo.gelu_fwd(big), [30.0, 0.0], rtol=0, atol=1e-300)
    assert np.allclose(mo.gelu_bwd(big, np.ones(2)), [1.0, 0.0], rtol=0, atol=1e-300)


def test_gelu_odd_part_is_x():
    # 0.5 (1 + tanh u) + 0.5 (1 + tanh(-u)) = 1, so gelu(x) - gelu(-x) = x
    x = _rand(1000, 15, 3.0)
    assert np.allclose(mo.gelu_fwd(x) - mo.gelu_fwd(-x), x, rtol=0, atol=1e-14)


def test_gelu_matches_torch_tanh_form():
    x, dy = _rand(2000, 16, 2.5), _rand(2000, 17)
    xt = torch.tensor(x, requires_grad=True)
    yt = torch.nn.functional.gelu(xt, approximate="tanh")
    yt.backward(torch.tensor(dy))
    assert np.allclose(mo.gelu_fwd(x), yt.detach().numpy(), rtol=0, atol=1e-14)
    assert np.allclose(mo.gelu_bwd(x, dy), xt.grad.numpy(), rtol=0, atol=1e-13)


def test_gelu_within_tanh_approximation_error_of_erf_form():
    from scipy.special import erf
    x = np.linspace(-8, 8, 20001)
    exact = 0.5 * x * (1 + erf(x / math.sqrt(2)))
    assert np.max(np.abs(mo.gelu_fwd(x) - exact)) < 1e-3


def test_gelu_finite_differences():
    x, h = _rand(200, 18, 2.0), 1e-6
    num = (mo.gelu_fwd(x + h) - mo.gelu_fwd(x - h)) / (2 * h)
    assert np.allclose(mo.gelu_bwd(x, np.ones_like(x)), num, rtol=1e-7, atol=1e-8)


# ---------------------------------------------------------------------------
# Softmax cross entropy
# ---------------------------------------------------------------------------
def test_sce_two_classes_is_softplus():
    # V = 2: loss of target 0 = log(1 + exp(z1 - z0))
    z = np.array([[0.3, 1.7], [-2.0, 5.0]])
    lse, rl, loss = mo.sce_fwd(z, [0, 1])
    assert abs(rl[0] - math.log1p(math.exp(1.7 - 0.3))) <= 1e-15
    assert abs(rl[1] - math.log1p(math.exp(-2.0 - 5.0))) <= 1e-15
    assert abs(loss - (rl[0] + rl[1]) / 2) <= 1e-15


def test_sce_uniform_logits_give_log_vocab():
    z = np.full((4, 50304), 1.25)
    lse, rl, loss = mo.sce_fwd(z, [0, 7, 50257, 50303])
    assert np.allclose(lse, 1.25 + math.log(50304), rtol=0, atol=1e-12)
    assert np.allclose(rl, math.log(50304), rtol=0, atol=1e-12)
    dz = mo.sce_bwd(z, [0, 7, 50257, 50303], 1.0)
    assert abs(dz[0, 1] - 1 / 50304) <= 1e-18 and abs(dz[0, 0] - (1 / 50304 - 1)) <= 1e-15


def test_sce_shift_invariance_and_gradient_rows():
    z, t = _rand((6, 300), 19, 4.0), np.random.default_rng(20).integers(0, 300, 6)
    lse, rl, _ = mo.sce_fwd(z, t)
    lse2, rl2, _ = mo.sce_fwd(z + 123.0, t)
    assert np.allclose(rl, rl2, rtol=0, atol=1e-11) and np.allclose(lse2, lse + 123.0, rtol=0, atol=1e-11)
    dz = mo.sce_bwd(z, t, 0.5)
    assert np.allclose(dz.sum(axis=1), 0, atol=1e-15)
    assert np.all(dz[np.arange(6), t] < 0) and np.all(np.delete(dz, t + 300 * np.arange(6)) >= 0)


def test_sce_matches_torch_cross_entropy():
    z, t = _rand((9, 500), 21, 3.0), np.random.default_rng(22).integers(0, 500, 9)
    zt = torch.tensor(z, requires_grad=True)
    loss_t = torch.nn.functional.cross_entropy(zt, torch.tensor(t), reduction="mean")
    loss_t.backward()
    lse, rl, loss = mo.sce_fwd(z, t)
    assert np.allclose(lse, torch.logsumexp(torch.tensor(z), 1).numpy(), rtol=0, atol=1e-12)
    assert abs(loss - loss_t.item()) <= 1e-12
    assert np.allclose(mo.sce_bwd(z, t, 1.0 / 9), zt.grad.numpy(), rtol=0, atol=1e-15)


def test_sce_finite_differences():
    z, t, h = _rand((2, 7), 23), np.array([3, 6]), 1e-6
    num = np.zeros_like(z)
    for idx in np.ndindex(z.shape):
        p, m = z.copy(), z.copy()
        p[idx] += h
        m[idx] -= h
        num[idx] = (mo.sce_fwd(p, t)[2] - mo.sce_fwd(m, t)[2]) / (2 * h)
    assert np.allclose(mo.sce_bwd(z, t, 0.5), num, rtol=1e-7, atol=1e-9)


def test_sce_invalid_target_is_nan_for_that_row_only():
    z = _rand((3, 10), 24)
    _, rl, loss = mo.sce_fwd(z, [1, 10, -1])
    assert np.isfinite(rl[0]) and np.isnan(rl[1]) and np.isnan(rl[2]) and np.isnan(loss)
    dz = mo.sce_bwd(z, [1, 10, 2], 1.0)
    assert np.all(np.isfinite(dz[[0, 2]])) and np.all(np.isnan(dz[1]))


# ---------------------------------------------------------------------------
# Planted mistakes: each plausible slip trips a pin above
# ---------------------------------------------------------------------------
def _ln_unbiased(x, g, b, eps=1e-5):
    x = np.asarray(x, float)
    mu = x.mean(1)
    rstd = 1 / np.sqrt(x.var(1, ddof=1) + eps)
    return (x - mu[:, None]) * rstd[:, None] * g + b


def _ln_bwd_no_xhat_term(x, g, dy, eps=1e-5):
    mu, rstd = mo.layernorm_stats(x, eps)
    gg = dy * g
    return rstd[:, None] * (gg - gg.mean(1, keepdims=True))


def _gelu_bwd_no_tanh_derivative(x, dy):
    t = np.tanh(mo.GELU_C * (x + mo.GELU_A * x ** 3))
    return dy * 0.5 * (1 + t)


def _gelu_sign(x):
    return 0.5 * x * (1 - np.tanh(mo.GELU_C * (x + mo.GELU_A * x ** 3)))


def _sce_bwd_no_onehot(z, t, s):
    return s * np.exp(z - mo.sce_lse(z)[:, None])


@pytest.mark.parametrize("kind", ["ln_unbiased", "ln_bwd_no_xhat", "gelu_bwd_no_tanh", "gelu_sign",
                                  "sce_no_onehot"])
def test_planted_mistakes_are_caught(kind):
    if kind == "ln_unbiased":
        x = _rand((4, 32), 30)
        ref = torch.nn.functional.layer_norm(torch.tensor(x), (32,), eps=1e-5).numpy()
        assert not np.allclose(_ln_unbiased(x, np.ones(32), np.zeros(32)), ref, rtol=0, atol=1e-6)
    elif kind == "ln_bwd_no_xhat":
        x, g, dy = _rand((3, 16), 31), _rand(16, 32), _rand((3, 16), 33)
        assert not np.allclose(_ln_bwd_no_xhat_term(x, g, dy), mo.layernorm_bwd(x, g, dy)[0], rtol=0, atol=1e-6)
        xt = torch.tensor(x, requires_grad=True)
        torch.nn.functional.layer_norm(xt, (16,), torch.tensor(g), None, eps=1e-5).backward(torch.tensor(dy))
        assert not np.allclose(_ln_bwd_no_xhat_term(x, g, dy), xt.grad.numpy(), rtol=0, atol=1e-6)
    elif kind == "gelu_bwd_no_tanh":
        x, h = _rand(50, 34, 2.0), 1e-6
        num = (mo.gelu_fwd(x + h) - mo.gelu_fwd(x - h)) / (2 * h)
        assert not np.allclose(_gelu_bwd_no_tanh_derivative(x, np.ones(50)), num, rtol=1e-7, atol=1e-8)
    elif kind == "gelu_sign":
        # the odd-part identity holds for this slip too; the large-x limit does not
        assert not np.allclose(_gelu_sign(np.array([30.0, -30.0])), [30.0, 0.0], rtol=0, atol=1e-300)
    else:
        z, t = _rand((3, 20), 36), np.array([0, 5, 19])
        assert not np.allclose(_sce_bwd_no_onehot(z, t, 1.0).sum(1), 0, atol=1e-15)
