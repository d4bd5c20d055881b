"""GPU parity of the memory-bound operators (LayerNorm, GELU, softmax cross
entropy; forward and backward) against the float64 oracle, through the C ABI.

Tolerances, derived from the float32 arithmetic of the kernels:

* LayerNorm y, dx: per row, max abs error <= 1e-5 (1 + |mean|) max(1, rstd).
  Each output is a handful of roundings of O(1) values after sums of C terms
  (relative error <= ~20 * 2^-24 of sum |terms|); the mean's error scales with
  |mean| and enters xhat multiplied by rstd, and dx itself scales with rstd.
  mean: |err| <= 1e-5 (|mean| + 1/rstd); rstd: relative 1e-5.  dgamma,
  dbeta: each is a sum over every row, accumulated in chains of at most ~100
  float additions (a wave's rows, the four waves of a group, then the partial
  rows in 128 strided streams, a butterfly and 16 wave sums), so the error is
  bounded by
  100 * 2^-24 * sum_r |term| < 1e-5 * sum_r |term|, which is the test.
* GELU y: |err| <= 1e-6 (1 + |x|): y = x (1 - r) with r = 1 / (1 + 2^t) from
  one hardware exp2 and one reciprocal (1 ulp each) and t from three
  roundings; the propagated error is below 4 * 2^-24 |x|.  dx: |err| <=
  2e-6 |dy| (1 + |x|) for the few more roundings of the derivative.
* Cross entropy lse, row loss: per row |err| <= e = 1e-5 + 6e-7 max|z|.  The
  sum of V exponentials is kept per lane in chains of V / 1024 additions of
  4-term sums and merged in a 256-leaf tree (relative error < 1e-5); the
  scaling of z by log2(e) and the final conversion each round at the
  magnitude of max|z| * 1.44 (<= 2^-24 of it per rounding, three of them).
  Mean loss: the largest row e.  dz: |err| <= |scale| (p (2e + 1e-6) + 2e-7),
  p the softmax probability: the exponent carries lse's error plus two
  roundings, and the target entry's p - 1 adds one rounding of 1.

Small cases compare every element and cover ragged shapes (columns that do not
fill a wave, vocabulary chunks with a ragged tail, element counts that are not
a multiple of 4).  The paper's shapes (LayerNorm 16x1024x768, GELU
16x1024x3072, cross entropy 16x1024x50304) run at full size in the launch
configuration the benchmark times: LayerNorm and GELU compared element by
element, cross entropy on sampled rows the oracle computes exactly plus
properties that hold on every row.
"""

import numpy as np
import pytest
import torch

import oracle.memops_oracle as mo
from paper_2608_00029_amd import binding as b
from paper_2608_00029_amd.workloads import (GPT2_VOCAB, MEMOPS_WORKLOADS, make_gelu_inputs, make_layernorm_inputs,
                                            make_sce_inputs)

pytestmark = pytest.mark.gpu

WL = {w.op: w for w in MEMOPS_WORKLOADS}


def _np(t):
    return t.detach().cpu().double().numpy()


def _check_layernorm(x, g, be, dy, dev, eps=1e-5):
    xd, gd, bd, dyd = (t.to(dev) for t in (x, g, be, dy))
    y, mean, rstd = b.layernorm_fwd(xd, gd, bd, eps)
    dx, dg, db = b.layernorm_bwd(xd, gd, mean, rstd, dyd)
    torch.cuda.synchronize()
    ry, rm, rr = mo.layernorm_fwd(x, g, be, eps)
    rdx, rdg, rdb = mo.layernorm_bwd(x, g, dy, eps)
    tol = (1e-5 * (1 + np.abs(rm)) * np.maximum(1.0, rr))[:, None]
    assert np.all(np.abs(_np(y) - ry) <= tol)
    assert np.all(np.abs(_np(mean) - rm) <= 1e-5 * (np.abs(rm) + 1 / rr))
    assert np.max(np.abs(_np(rstd) - rr) / rr) <= 1e-5
    assert np.all(np.abs(_np(dx) - rdx) <= tol)
    xn, dyn = x.double().numpy(), dy.double().numpy()
    xhat = (xn - rm[:, None]) * rr[:, None]
    assert np.all(np.abs(_np(dg) - rdg) <= 1e-5 * np.abs(dyn * xhat).sum(axis=0) + 1e-30)
    assert np.all(np.abs(_np(db) - rdb) <= 1e-5 * np.abs(dyn).sum(axis=0) + 1e-30)


@pytest.mark.parametrize("rows,C", [(1, 4), (5, 64), (3, 256), (7, 768), (300, 1000), (33, 3072), (9, 4096),
                                    (2000, 768)])
def test_layernorm_small(cuda, rows, C):
    x, g, be, dy = make_layernorm_inputs(rows, C, seed=rows * 7 + C)
    _check_layernorm(x, g, be, dy, cuda)


def test_layernorm_constant_row_and_offset(cuda):
    # a constant row has variance 0: xhat = 0, y = beta exactly, rstd = 1/sqrt(eps); an offset of
    # 8 standard deviations exercises the two-pass variance
    x, g, be, dy = make_layernorm_inputs(6, 768, seed=99)
    x[0] = 2.5
    x[1:] += 8.0
    _check_layernorm(x, g, be, dy, cuda)
    y, _, _ = b.layernorm_fwd(x.to(cuda), g.to(cuda), be.to(cuda))
    assert torch.equal(y[0].cpu(), be)


def test_layernorm_full_size(cuda):
    w = WL["layernorm"]
    x, g, be, dy = make_layernorm_inputs(w.rows, w.C, w.seed)
    _check_layernorm(x, g, be, dy, cuda)


def _check_gelu(x, dy, dev):
    y = b.gelu_fwd(x.to(dev))
    dx = b.gelu_bwd(x.to(dev), dy.to(dev))
    torch.cuda.synchronize()
    xn, dyn = x.double().numpy(), dy.double().numpy()
    assert np.all(np.abs(_np(y) - mo.gelu_fwd(xn)) <= 1e-6 * (1 + np.abs(xn)))
    assert np.all(np.abs(_np(dx) - mo.gelu_bwd(xn, dyn)) <= 2e-6 * np.abs(dyn) * (1 + np.abs(xn)))


@pytest.mark.parametrize("n", [1, 3, 4, 7, 1023, 4096 + 3, 1 << 20, 3 * (1 << 20) + 5])
def test_gelu_small(cuda, n):
    x, dy = make_gelu_inputs(n, seed=n)
    _check_gelu(x, dy, cuda)


def test_gelu_extremes(cuda):
    x = torch.tensor([0.0, -0.0, 1e-30, -1e-30, 1e-6, 20.0, -20.0, 60.0, -60.0, 1e4, -1e4, 3.0], dtype=torch.float32)
    _check_gelu(x, torch.ones_like(x), cuda)


def test_gelu_full_size(cuda):
    w = WL["gelu"]
    x, dy = make_gelu_inputs(w.rows * w.C, w.seed)
    _check_gelu(x, dy, cuda)


def _check_sce_rows(z, t, lse, rl, dz, rows, scale):
    zs = z[rows].double().numpy()
    ts = t[rows].numpy()
    rlse, rrl, _ = mo.sce_fwd(zs, ts)
    e = 1e-5 + 6e-7 * np.abs(zs).max(axis=1)
    assert np.all(np.abs(_np(lse)[rows] - rlse) <= e)
    assert np.all(np.abs(_np(rl)[rows] - rrl) <= e)
    rdz = mo.sce_bwd(zs, ts, scale)
    p = np.exp(zs - rlse[:, None])
    assert np.all(np.abs(_np(dz[rows]) - rdz) <= abs(scale) * (p * (2 * e[:, None] + 1e-6) + 2e-7))
    return e.max()


@pytest.mark.parametrize("rows,V,sigma", [(1, 4, 1.0), (3, 100, 2.0), (5, 1028, 2.0), (4, 4100, 4.0),
                                          (8, 50304, 2.0), (2, 8192, 30.0)])
def test_sce_small(cuda, rows, V, sigma):
    z, t = make_sce_inputs(rows, V, seed=rows * 13 + V, sigma=sigma)
    zd, td = z.to(cuda), t.to(cuda)
    lse, rl, loss = b.sce_fwd(zd, td)
    scale = 1.0 / rows
    dz = b.sce_bwd(zd, td, lse, scale)
    torch.cuda.synchronize()
    e = _check_sce_rows(z, t, lse, rl, dz, np.arange(rows), scale)
    assert abs(loss.item() - mo.sce_fwd(z, t)[2]) <= e


def test_sce_without_targets_writes_lse_only(cuda):
    z, _ = make_sce_inputs(4, 256, seed=5)
    lse, rl, loss = b.sce_fwd(z.to(cuda))
    torch.cuda.synchronize()
    assert rl is None and loss is None
    assert np.max(np.abs(_np(lse) - mo.sce_lse(z))) <= 1e-5


def test_sce_invalid_target_gives_nan_for_that_row_only(cuda):
    z, t = make_sce_inputs(4, 512, seed=6)
    t[1] = 512
    t[2] = -3
    zd, td = z.to(cuda), t.to(cuda)
    lse, rl, loss = b.sce_fwd(zd, td)
    dz = b.sce_bwd(zd, td, lse, 0.25)
    torch.cuda.synchronize()
    rl, dz = _np(rl), _np(dz)
    assert np.isfinite(rl[[0, 3]]).all() and np.isnan(rl[[1, 2]]).all() and np.isnan(loss.item())
    assert np.isfinite(dz[[0, 3]]).all() and np.isnan(dz[[1, 2]]).all()


def test_sce_full_size_sampled_rows(cuda):
    w = WL["sce"]
    z, t = make_sce_inputs(w.rows, w.C, w.seed, n_real=GPT2_VOCAB)
    zd, td = z.to(cuda), t.to(cuda)
    lse, rl, loss = b.sce_fwd(zd, td)
    scale = 1.0 / w.rows
    dz = b.sce_bwd(zd, td, lse, scale)
    torch.cuda.synchronize()
    rows = np.random.default_rng(7).choice(w.rows, 48, replace=False)
    rows = np.concatenate([[0, w.rows - 1], rows])
    e = _check_sce_rows(z, t, lse, rl, dz, rows, scale)
    # every row: lse >= row max, the loss is the mean of the row losses, the gradient rows sum to ~0
    zmax = zd.max(dim=1).values
    assert bool((lse >= zmax - 1e-5).all())
    rln = _np(rl)
    assert abs(loss.item() - rln.mean()) <= e
    rs = dz.double().sum(dim=1).abs().max().item()
    assert rs <= abs(scale) * 1e-4


def test_memops_deterministic(cuda):
    x, g, be, dy = (t.to(cuda) for t in make_layernorm_inputs(3000, 768, seed=1))
    z, t = (a.to(cuda) for a in make_sce_inputs(64, 50304, seed=2))
    outs = []
    for _ in range(2):
        y, m, r = b.layernorm_fwd(x, g, be)
        dx, dg, db = b.layernorm_bwd(x, g, m, r, dy)
        lse, rl, loss = b.sce_fwd(z, t)
        outs.append([a.clone() for a in (y, dx, dg, db, lse, loss, b.gelu_bwd(x, dy))])
    torch.cuda.synchronize()
    for a, c in zip(*outs):
        assert torch.equal(a, c)
