"""Pins of the loss-head oracle (oracle/lmhead_oracle.py) against facts that do
not come from the oracle: a hand-worked case with exact answers, closed forms,
torch's float64 logsumexp and cross entropy, the tile-merge identity for
every tile width, and planted mistakes that each trip at least one check."""

import math

import numpy as np
import pytest
import torch

import oracle.lmhead_oracle as lm


def _rand(shape, seed, sigma=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * sigma


def test_hand_worked_two_rows():
    # X = [[1, 2], [0, 1]], W rows [1, 0], [0, 1], [1, 1]: Z = [[1, 2, 3], [0, 1, 1]]
    x = np.array([[1.0, 2.0], [0.0, 1.0]])
    w = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0]])
    z, lse, rl, loss = lm.lmhead_fwd(x, w, targets=[2, 0])
    assert np.array_equal(z, [[1, 2, 3], [0, 1, 1]])
    e = math.e
    lse_ref = [math.log(e + e ** 2 + e ** 3), math.log(1 + 2 * e)]
    assert np.allclose(lse, lse_ref, rtol=0, atol=1e-15)
    assert np.allclose(rl, [lse_ref[0] - 3, lse_ref[1] - 0], rtol=0, atol=1e-15)
    assert abs(loss - (rl[0] + rl[1]) / 2) <= 1e-15


def test_zero_weight_gives_log_vocab():
    x, w = _rand((5, 16), 1), np.zeros((37, 16))
    z, lse, rl, loss = lm.lmhead_fwd(x, w, targets=np.arange(5))
    assert np.all(z == 0)
    assert np.allclose(lse, math.log(37), rtol=0, atol=1e-14)
    assert abs(loss - math.log(37)) <= 1e-14


def test_constant_row_closed_form():
    z = np.full((3, 11), 2.5)
    assert np.allclose(lm.row_logsumexp(z), 2.5 + math.log(11), rtol=0, atol=1e-14)


def test_lse_and_loss_match_torch():
    x, w = _rand((64, 48), 2), _rand((300, 48), 3, 0.3)
    y = np.random.default_rng(4).integers(0, 300, 64)
    z, lse, rl, loss = lm.lmhead_fwd(x, w, targets=y)
    zt = torch.tensor(x) @ torch.tensor(w).T
    assert np.allclose(z, zt.numpy(), rtol=0, atol=1e-12)
    assert np.allclose(lse, torch.logsumexp(zt, dim=1).numpy(), rtol=0, atol=1e-12)
    ce = torch.nn.functional.cross_entropy(zt, torch.tensor(y), reduction="none")
    assert np.allclose(rl, ce.numpy(), rtol=0, atol=1e-12)
    assert abs(loss - float(ce.mean())) <= 1e-12


@pytest.mark.parametrize("tile", [1, 7, 64, 128, 300, 305])
def test_tile_merge_equals_plain_logsumexp(tile):
    # peaked rows (large logits) so that an unrescaled merge would be far off
    z = _rand((40, 300), 5, 8.0)
    pm, ps = lm.tile_partials(z, tile)
    assert pm.shape[1] == (300 + tile - 1) // tile
    assert np.allclose(lm.merge_partials(pm, ps), lm.row_logsumexp(z), rtol=0, atol=1e-12)


def test_single_tile_partial_is_the_row():
    z = _rand((6, 50), 6)
    pm, ps = lm.tile_partials(z, 50)
    assert np.array_equal(pm[:, 0], z.max(axis=1))
    assert np.allclose(np.log(ps[:, 0]) + pm[:, 0], lm.row_logsumexp(z), rtol=0, atol=1e-13)


def test_error_bound_holds_for_float32_accumulation():
    # bf16-representable inputs, float32 accumulation in numpy: inside the bound
    x = torch.tensor(_rand((32, 768), 7)).to(torch.bfloat16).double().numpy()
    w = torch.tensor(_rand((64, 768), 8, 0.02)).to(torch.bfloat16).double().numpy()
    z32 = (x.astype(np.float32) @ w.astype(np.float32).T).astype(np.float64)
    err = np.abs(z32 - lm.logits(x, w))
    assert np.all(err <= lm.dot_error_bound(x, w))


def test_error_bound_is_reached_by_a_worst_case_sum():
    """The bound is not loose in the worst case: with products 1, t, t, ... and
    t = 2^-24 (1 + 2^-7) (a bf16 value just above half an ulp of the running
    sum), every float32 addition of a left-to-right sum rounds up by almost
    u = 2^-24 of the sum, so the error reaches 99% of gamma_K sum|p|."""
    K = 768
    t = 2.0 ** -24 * (1 + 2.0 ** -7)
    x = np.ones((1, K))
    w = np.full((1, K), t)
    w[0, 0] = 1.0
    assert np.array_equal(torch.tensor(w).to(torch.bfloat16).double().numpy(), w)  # bf16 values
    z32 = np.cumsum((x[0] * w[0]).astype(np.float32), dtype=np.float32)[-1]
    assert z32 == np.float32(1 + (K - 1) * 2.0 ** -23)  # every addition rounded up
    err = abs(float(z32) - float(lm.logits(x, w)[0, 0]))
    bound = float(lm.dot_error_bound(x, w)[0, 0])
    assert 0.98 * bound < err <= bound


def test_logit_tolerance_catches_plausible_mistakes():
    """The GPU test holds logits to twice the bound.  On inputs shaped like the
    loss head's (hidden states N(0, 1), weights N(0, 0.02^2), K = 768), that
    tolerance still fails logits rounded to bf16 and logits missing one
    16-wide contraction step, the kind of mistake a kernel could make."""
    x = torch.tensor(_rand((16, 768), 21)).to(torch.bfloat16).double().numpy()
    w = torch.tensor(_rand((256, 768), 22, 0.02)).to(torch.bfloat16).double().numpy()
    z = lm.logits(x, w)
    tol = 2 * lm.dot_error_bound(x, w)
    z_bf16 = torch.tensor(z).to(torch.bfloat16).double().numpy()
    assert np.mean(np.abs(z_bf16 - z) > tol) > 0.05
    z_short = lm.logits(x[:, 16:], w[:, 16:])
    assert np.mean(np.abs(z_short - z) > tol) > 0.9


def _planted(kind):
    """Copies of oracle steps with one plausible mistake each."""
    def merge_no_rescale(pm, ps):
        return np.log(ps.sum(axis=1)) + pm.max(axis=1)

    def lse_no_max(z):
        with np.errstate(over="ignore"):
            return np.log(np.exp(z).sum(axis=1))

    def loss_wrong_sign(z, lse, y):
        return z[np.arange(z.shape[0]), y] - lse

    def loss_off_by_one(z, lse, y):
        return lse - z[np.arange(z.shape[0]), (np.asarray(y) + 1) % z.shape[1]]

    def logits_untransposed(x, w):  # W taken as [K, N] instead of [N, K]
        return x @ w

    return {"merge_no_rescale": merge_no_rescale, "lse_no_max": lse_no_max, "loss_wrong_sign": loss_wrong_sign,
            "loss_off_by_one": loss_off_by_one, "logits_untransposed": logits_untransposed}[kind]


@pytest.mark.parametrize("kind", ["merge_no_rescale", "lse_no_max", "loss_wrong_sign", "loss_off_by_one",
                                  "logits_untransposed"])
def test_planted_mistakes_are_caught(kind):
    bad = _planted(kind)
    z = _rand((8, 96), 9, 400.0)  # large logits: exp overflows without the max shift
    x, w = _rand((8, 16), 10), _rand((96, 16), 11)
    y = np.random.default_rng(12).integers(0, 96, 8)
    zt = torch.tensor(z)
    ref_lse = torch.logsumexp(zt, dim=1).numpy()
    if kind == "merge_no_rescale":
        pm, ps = lm.tile_partials(z, 32)
        assert not np.allclose(bad(pm, ps), ref_lse, rtol=0, atol=1e-6)
    elif kind == "lse_no_max":
        got = bad(z)
        assert not (np.all(np.isfinite(got)) and np.allclose(got, ref_lse, rtol=0, atol=1e-6))
    elif kind in ("loss_wrong_sign", "loss_off_by_one"):
        ref = torch.nn.functional.cross_entropy(zt, torch.tensor(y), reduction="none").numpy()
        assert not np.allclose(bad(z, ref_lse, y), ref, rtol=0, atol=1e-6)
    else:
        ws = _rand((16, 16), 13)  # square, so the untransposed product is defined
        assert not np.allclose(bad(x, ws), lm.logits(x, ws), rtol=0, atol=1e-6)
        assert np.allclose((torch.tensor(x) @ torch.tensor(ws).T).numpy(), lm.logits(x, ws), rtol=0, atol=1e-12)
