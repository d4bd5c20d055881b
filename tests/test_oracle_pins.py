"""Pins of the CPU float64 oracle against facts that do not come from the oracle.

Each check compares the oracle with something fixed independently of its code:
a hand-worked example (tests/golden), closed forms, invariants of softmax
attention, central finite differences of the scalar sum(dO * O), and torch's
own float64 scaled-dot-product attention with autograd.  A final test plants
plausible mistakes in copies of the oracle's functions and shows that every
one of them trips at least one check.
"""

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle.attn_oracle as orc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_worked_s3.json")


def _val(s: str) -> float:
    if s.startswith("log:"):
        return math.log(float(Fraction(s[4:])))
    if s.endswith("*ln2"):
        return float(Fraction(s[:-4])) * math.log(2.0)
    return float(Fraction(s))


def _vec(lst):
    return np.array([_val(x) for x in lst])


def _rand(shape, seed, sigma=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * sigma


# --------------------------------------------------------------------------------------
# Checks, written as plain functions so that the planted-mistake test can re-run them
# against a mutated oracle.  Each takes the forward and backward callables to check.
# --------------------------------------------------------------------------------------

def check_golden(fwd, bwd):
    g = json.load(open(GOLDEN))
    inp = g["inputs"]
    q, k, v, do = (_vec(inp[n]).reshape(1, 1, 3, 1) for n in ("q", "k", "v", "do"))
    for causal, key in ((True, "causal"), (False, "noncausal")):
        exp = g[key]
        o, lse = fwd(q, k, v, inp["scale"], causal)
        dq, dk, dv = bwd(q, k, v, do, inp["scale"], causal)
        for name, got in (("o", o), ("lse", lse), ("dq", dq), ("dk", dk), ("dv", dv)):
            np.testing.assert_allclose(got.reshape(-1), _vec(exp[name]), rtol=0, atol=1e-13,
                                       err_msg=f"{key} {name}")


def check_zero_query_prefix_mean(fwd, bwd):
    """Q = 0 makes every visible score 0: O_i is the mean of V_0..V_i, LSE_i = ln(i+1).
    The same holds for K = 0."""
    B, H, S, D = 2, 3, 17, 5
    v = _rand((B, H, S, D), 1)
    x = _rand((B, H, S, D), 2)
    zero = np.zeros((B, H, S, D))
    prefix = np.cumsum(v, axis=2) / np.arange(1, S + 1)[None, None, :, None]
    for q, k in ((zero, x), (x, zero)):
        o, lse = fwd(q, k, v, 0.37, True)
        np.testing.assert_allclose(o, prefix, rtol=0, atol=1e-13)
        np.testing.assert_allclose(lse, np.broadcast_to(np.log(np.arange(1, S + 1)), lse.shape),
                                   rtol=0, atol=1e-13)


def check_first_row(fwd, bwd):
    """Query 0 sees only key 0: O_0 = V_0 and LSE_0 = scale * q_0 . k_0."""
    B, H, S, D = 2, 2, 9, 4
    q, k, v = _rand((B, H, S, D), 3), _rand((B, H, S, D), 4), _rand((B, H, S, D), 5)
    o, lse = fwd(q, k, v, 0.5, True)
    np.testing.assert_allclose(o[:, :, 0], v[:, :, 0], rtol=0, atol=1e-14)
    np.testing.assert_allclose(lse[:, :, 0], 0.5 * np.sum(q[:, :, 0] * k[:, :, 0], axis=-1),
                               rtol=0, atol=1e-13)


def check_single_token(fwd, bwd):
    """S = 1: O = V, dV = dO, dQ = dK = 0 (softmax of one entry is constant 1)."""
    q, k, v, do = (_rand((2, 3, 1, 8), s) for s in range(10, 14))
    for causal in (True, False):
        o, lse = fwd(q, k, v, 0.3, causal)
        dq, dk, dv = bwd(q, k, v, do, 0.3, causal)
        np.testing.assert_allclose(o, v, rtol=0, atol=1e-15)
        np.testing.assert_allclose(dv, do, rtol=0, atol=1e-15)
        np.testing.assert_allclose(dq, 0.0, rtol=0, atol=1e-15)
        np.testing.assert_allclose(dk, 0.0, rtol=0, atol=1e-15)


def check_gradient_invariants(fwd, bwd):
    """Sum_j dK_j = 0 (scores are invariant to a common shift of the keys),
    sum_j dV_j = sum_i dO_i (rows of P sum to 1), <Q, dQ> = <K, dK> per head
    (both equal sum_ij dS_ij S_ij)."""
    B, H, S, D = 2, 2, 13, 6
    q, k, v, do = (_rand((B, H, S, D), s) for s in range(20, 24))
    for causal in (True, False):
        dq, dk, dv = bwd(q, k, v, do, 0.41, causal)
        np.testing.assert_allclose(dk.sum(axis=2), 0.0, rtol=0, atol=1e-12)
        np.testing.assert_allclose(dv.sum(axis=2), do.sum(axis=2), rtol=0, atol=1e-12)
        np.testing.assert_allclose((q * dq).sum(axis=(2, 3)), (k * dk).sum(axis=(2, 3)),
                                   rtol=0, atol=1e-12)


def check_value_affine(fwd, bwd):
    """O(Q, K, a V + 1 b^T) = a O + 1 b^T (rows of P sum to 1)."""
    B, H, S, D = 1, 2, 11, 4
    q, k, v = _rand((B, H, S, D), 30), _rand((B, H, S, D), 31), _rand((B, H, S, D), 32)
    b = _rand((D,), 33)
    for causal in (True, False):
        o1, _ = fwd(q, k, v, 0.7, causal)
        o2, _ = fwd(q, k, 2.5 * v + b, 0.7, causal)
        np.testing.assert_allclose(o2, 2.5 * o1 + b, rtol=0, atol=1e-12)


def check_finite_differences(fwd, bwd):
    """Central differences of f = sum(dO * O) with respect to every entry of Q, K, V."""
    B, H, S, D = 1, 2, 6, 3
    q, k, v, do = (_rand((B, H, S, D), s) for s in range(40, 44))
    scale, h = 0.8, 1e-6
    for causal in (True, False):
        dq, dk, dv = bwd(q, k, v, do, scale, causal)

        def f(qq, kk, vv):
            return float(np.sum(do * fwd(qq, kk, vv, scale, causal)[0]))

        for which, grad in ((0, dq), (1, dk), (2, dv)):
            num = np.zeros_like(grad)
            for idx in np.ndindex(*grad.shape):
                args_p = [q.copy(), k.copy(), v.copy()]
                args_m = [q.copy(), k.copy(), v.copy()]
                args_p[which][idx] += h
                args_m[which][idx] -= h
                num[idx] = (f(*args_p) - f(*args_m)) / (2 * h)
            np.testing.assert_allclose(grad, num, rtol=0, atol=2e-8,
                                       err_msg=f"causal={causal} operand={'QKV'[which]}")


def check_torch_sdpa(fwd, bwd):
    """torch's own float64 scaled_dot_product_attention (an independent
    implementation) with autograd, and torch.logsumexp of the masked scores."""
    B, H, S, D = 2, 3, 37, 16
    q, k, v, do = (_rand((B, H, S, D), s, 1.5) for s in range(50, 54))
    scale = 1.0 / math.sqrt(D)
    for causal in (True, False):
        tq, tk, tv = (torch.tensor(x, requires_grad=True) for x in (q, k, v))
        to = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=causal,
                                                              scale=scale)
        to.backward(torch.tensor(do))
        s = (tq.detach() @ tk.detach().transpose(-1, -2)) * scale
        if causal:
            s = s.masked_fill(torch.ones(S, S, dtype=torch.bool).triu(1), float("-inf"))
        tlse = torch.logsumexp(s, dim=-1)
        o, lse = fwd(q, k, v, scale, causal)
        dq, dk, dv = bwd(q, k, v, do, scale, causal)
        np.testing.assert_allclose(o, to.detach().numpy(), rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse, tlse.numpy(), rtol=0, atol=1e-12)
        np.testing.assert_allclose(dq, tq.grad.numpy(), rtol=0, atol=1e-12)
        np.testing.assert_allclose(dk, tk.grad.numpy(), rtol=0, atol=1e-12)
        np.testing.assert_allclose(dv, tv.grad.numpy(), rtol=0, atol=1e-12)


ALL_CHECKS = [check_golden, check_zero_query_prefix_mean, check_first_row, check_single_token,
              check_gradient_invariants, check_value_affine, check_finite_differences,
              check_torch_sdpa]


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda c: c.__name__)
def test_oracle_pin(check):
    check(orc.attn_fwd, orc.attn_bwd)


def test_probabilities_row_stochastic():
    """P >= 0, every row sums to 1, and P_ij = 0 exactly for j > i."""
    q, k = _rand((2, 2, 19, 7), 60, 3.0), _rand((2, 2, 19, 7), 61, 3.0)
    p = orc.attn_probabilities(q, k, 0.9, True)
    assert np.all(p >= 0)
    np.testing.assert_allclose(p.sum(axis=-1), 1.0, rtol=0, atol=1e-13)
    assert np.all(p[..., np.triu_indices(19, 1)[0], np.triu_indices(19, 1)[1]] == 0.0)


def test_bwd_given_own_o_and_lse_matches_bwd():
    q, k, v, do = (_rand((1, 2, 23, 8), s) for s in range(70, 74))
    o, lse = orc.attn_fwd(q, k, v, 0.35, True)
    a = orc.attn_bwd(q, k, v, do, 0.35, True)
    b = orc.attn_bwd_given_o(q, k, v, o, do, lse, 0.35, True)
    for x, y in zip(a, b):
        np.testing.assert_allclose(x, y, rtol=0, atol=1e-13)


def test_peaked_softmax_is_finite():
    """Scores of magnitude ~1e3 (far beyond exp's float64 range unshifted)."""
    q, k, v, do = _rand((1, 1, 64, 16), 80, 30.0), _rand((1, 1, 64, 16), 81, 30.0), \
        _rand((1, 1, 64, 16), 82), _rand((1, 1, 64, 16), 83)
    o, lse = orc.attn_fwd(q, k, v, 1.0, True)
    grads = orc.attn_bwd(q, k, v, do, 1.0, True)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    assert all(np.all(np.isfinite(g)) for g in grads)


# --------------------------------------------------------------------------------------
# Planted mistakes: each mutant is a copy of the oracle's per-head code with one
# plausible error; at least one check above must fail on it.
# --------------------------------------------------------------------------------------

def _mutant(head_fwd=None, head_bwd=None):
    def fwd(q, k, v, scale, causal=True):
        q, k, v = (np.asarray(x, dtype=np.float64) for x in (q, k, v))
        B, H, S, D = q.shape
        o, lse = np.empty((B, H, S, D)), np.empty((B, H, S))
        for b in range(B):
            for h in range(H):
                o[b, h], lse[b, h] = (head_fwd or orc.head_forward)(q[b, h], k[b, h], v[b, h],
                                                                     scale, causal)
        return o, lse

    def bwd(q, k, v, do, scale, causal=True):
        q, k, v, do = (np.asarray(x, dtype=np.float64) for x in (q, k, v, do))
        out = [np.empty(q.shape) for _ in range(3)]
        for b in range(q.shape[0]):
            for h in range(q.shape[1]):
                r = (head_bwd or orc.head_backward)(q[b, h], k[b, h], v[b, h], do[b, h], scale,
                                                    causal)
                for o_, r_ in zip(out, r):
                    o_[b, h] = r_
        return tuple(out)
    return fwd, bwd


def _scores_mask_diag_too(q, k, scale, causal):
    s = scale * (q @ k.T)
    if causal:
        s = np.where(np.triu(np.ones(s.shape, dtype=bool), k=0), -np.inf, s)
    return s


def _scores_mask_lower(q, k, scale, causal):
    s = scale * (q @ k.T)
    if causal:
        s = np.where(np.tril(np.ones(s.shape, dtype=bool), k=-1), -np.inf, s)
    return s


def _fwd_with_scores(scores):
    def f(q, k, v, scale, causal):
        s = scores(q, k, scale, causal)
        lse = orc.row_logsumexp(s)
        return orc.probabilities(s, lse) @ v, lse
    return f


def _fwd_lse_without_max(q, k, v, scale, causal):
    s = orc.masked_scores(q, k, scale, causal)
    m = np.max(s, axis=1)
    lse = np.log(np.sum(np.exp(s - m[:, None]), axis=1))  # dropped + m
    return orc.probabilities(s, lse) @ v, lse


def _fwd_scale_twice(q, k, v, scale, causal):
    s = orc.masked_scores(q, k, scale, causal) * scale
    lse = orc.row_logsumexp(s)
    return orc.probabilities(s, lse) @ v, lse


def _bwd_variant(kind):
    def g(q, k, v, do, scale, causal):
        s = orc.masked_scores(q, k, scale, causal)
        lse = orc.row_logsumexp(s)
        p = orc.probabilities(s, lse)
        o = p @ v
        dv = p.T @ do
        dp = do @ v.T
        d = np.sum(do * o, axis=1)
        if kind == "d_without_o":
            d = np.sum(do, axis=1)
        if kind == "d_from_columns":
            d = np.sum(p * dp, axis=0)
        ds = p * (dp - d[:, None])
        if kind == "no_p_factor":
            ds = dp - d[:, None]
        dq = scale * (ds @ k)
        dk = scale * (ds.T @ q)
        if kind == "dq_no_scale":
            dq = ds @ k
        if kind == "dk_untransposed":
            dk = scale * (ds @ q)
        if kind == "dv_untransposed":
            dv = p @ do
        if kind == "dq_uses_v":
            dq = scale * (ds @ v)
        return dq, dk, dv
    return g


MUTANTS = {
    "mask_includes_diagonal": _mutant(head_fwd=_fwd_with_scores(_scores_mask_diag_too)),
    "mask_below_diagonal": _mutant(head_fwd=_fwd_with_scores(_scores_mask_lower)),
    "lse_without_max": _mutant(head_fwd=_fwd_lse_without_max),
    "scale_applied_twice": _mutant(head_fwd=_fwd_scale_twice),
    **{k: _mutant(head_bwd=_bwd_variant(k)) for k in
       ("d_without_o", "d_from_columns", "no_p_factor", "dq_no_scale", "dk_untransposed",
        "dv_untransposed", "dq_uses_v")},
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    fwd, bwd = MUTANTS[name]
    caught = []
    with np.errstate(all="ignore"):
        for check in ALL_CHECKS:
            try:
                check(fwd, bwd)
            except (AssertionError, ValueError, FloatingPointError):
                caught.append(check.__name__)
    assert caught, f"mutant {name} passed every check"


# --------------------------------------------------------------------------------------
# The term magnitudes the GPU parity tests derive their per-element error bounds from.
# --------------------------------------------------------------------------------------

def test_term_magnitudes_hand_worked():
    """Every magnitude of the S=3 hand-worked example (derived by hand, golden file)."""
    g = json.load(open(GOLDEN))
    inp = g["inputs"]
    q, k, v, do = (_vec(inp[n]).reshape(1, 1, 3, 1) for n in ("q", "k", "v", "do"))
    m = orc.attn_term_magnitudes(q, k, v, do, inp["scale"], True)
    for name, exp in g["causal_magnitudes"].items():
        np.testing.assert_allclose(m[name].reshape(-1), _vec(exp), rtol=0, atol=1e-13, err_msg=name)


def test_term_magnitudes_bound_the_outputs():
    """Triangle inequality: each output element is at most its terms' absolute sum,
    with equality when every term is nonnegative (V >= 0 for O, dO >= 0 for dV)."""
    q, k, v, do = (_rand((2, 2, 37, 8), s, 2.0) for s in range(90, 94))
    for causal in (True, False):
        m = orc.attn_term_magnitudes(q, k, v, do, 0.3, causal)
        o, _ = orc.attn_fwd(q, k, v, 0.3, causal)
        dq, dk, dv = orc.attn_bwd(q, k, v, do, 0.3, causal)
        tol = 1e-12
        assert np.all(np.abs(o) <= m["m_o"] * (1 + tol) + tol)
        assert np.all(np.abs(dv) <= m["m_dv"] * (1 + tol) + tol)
        assert np.all(np.abs(dq) <= 0.3 * m["g_dq"] * (1 + tol) + tol)
        assert np.all(np.abs(dk) <= 0.3 * m["g_dk"] * (1 + tol) + tol)
        # a_i bounds |D_i| = |rowsum(dO * O)|
        d = np.sum(do * o, axis=-1)
        assert np.all(np.abs(d) <= m["a"] * (1 + tol) + tol)
        vp, dop = np.abs(v), np.abs(do)
        mp = orc.attn_term_magnitudes(q, k, vp, dop, 0.3, causal)
        op, _ = orc.attn_fwd(q, k, vp, 0.3, causal)
        _, _, dvp = orc.attn_bwd(q, k, vp, dop, 0.3, causal)
        np.testing.assert_allclose(mp["m_o"], op, rtol=1e-13, atol=0)
        np.testing.assert_allclose(mp["m_dv"], dvp, rtol=1e-13, atol=0)
        # h = (a * P)|X|: with a = 1 it is P|X|, which for X >= 0 is the forward itself
        np.testing.assert_allclose(mp["h_dq"] / mp["a"][..., None],
                                   orc.attn_fwd(q, k, np.abs(k), 0.3, causal)[0], rtol=1e-12, atol=0)
