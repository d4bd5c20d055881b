"""Parity of the fused loss head (through the C ABI) with the float64 oracle.

Tolerances (the acceptance bar states none for this operation, so they are
derived from the arithmetic):
  * logits: products of bf16 values are exact in float32, so a float32
    accumulation of K of them in any order is within
    gamma_K * sum_k |x_ik w_jk| of the exact dot product (gamma_K = K u /
    (1 - K u), u = 2^-24; the oracle's `dot_error_bound`).  The matrix cores'
    internal order and rounding are not specified, so the test allows twice
    that bound.
  * LSE: the exact log-sum-exp moves by at most max_j |dZ_ij| when the
    logits move by dZ; the float32 exponentials, the 64-entry tile sums and
    the merge over N/64 partials add a relative error of at most about
    (64 + N/64 + 8) u to the sum of exponentials, i.e. that much absolute
    error in LSE.  Tolerance: 2 max_j bound_ij + 1e-5 + (64 + N/64 + 8) u.
  * row loss LSE - Z[y]: the LSE tolerance plus the logit tolerance of Z[y].
  * mean: the float64 mean of the GPU's own row losses within 1e-6 relative
    (a fixed-order float32 sum of M terms).
  * the partials: each tile maximum equals, bit for bit, the maximum of the
    GPU's own logits over the tile's 64 columns; each tile sum matches the
    float64 sum of exp(z - maximum) over those logits within 1e-5 relative.

Small cases compare every element; they span several 256 x 256 output tiles,
ragged last tiles in either direction (half-width tiles whose idle waves skip
their copies), vocabulary-tile counts that leave some chiplets without work
and some with an extra tile, work groups of the persistent grid that walk
several tiles, and logit scales where the per-tile maxima differ widely (so
the merge's rescale matters).  The GPT-2 head (M 8192, N 50304, K 768) runs at
full size in the configuration the benchmark times and is compared on sampled
rows, which the oracle computes exactly.
"""

import math

import numpy as np
import pytest
import torch

import oracle.lmhead_oracle as lm
from paper_2608_00029_amd import lmhead_fwd, lmhead_workspace_bytes
from paper_2608_00029_amd.workloads import LMHEAD_WORKLOADS, make_lmhead_inputs
from parity_util import say

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
U = 2.0 ** -24
PART_W = 64


def _lse_tol(bound_rows, N):
    return 2.0 * bound_rows + 1e-5 + (64 + N / PART_W + 8) * U


def check_rows(rows, x, w, y, z_gpu, lse_gpu, rl_gpu, part_gpu, N):
    """Compare the given rows of every output with the oracle."""
    xs = x[rows]
    z_ref = lm.logits(xs, w)
    bound = lm.dot_error_bound(xs, w)
    z64 = z_gpu.double().numpy()
    assert np.all(np.isfinite(z64)), "non-finite logits"
    err = np.abs(z64 - z_ref)
    assert np.all(err <= 2.0 * bound), f"logits: worst err/bound {np.max(err / np.maximum(bound, 1e-300)):.3f} > 2"
    lse_ref = lm.row_logsumexp(z_ref)
    brow = bound.max(axis=1)
    lerr = np.abs(lse_gpu.double().numpy() - lse_ref)
    ltol = _lse_tol(brow, N)
    assert np.all(lerr <= ltol), f"lse: max err {lerr.max():.3e}, tol {ltol.min():.3e}"
    rep = f"z max err {err.max():.2e} (bound {bound.max():.2e})  lse max err {lerr.max():.2e}"
    if rl_gpu is not None:
        yr = np.asarray(y)[rows]
        rl_ref = lm.row_losses(z_ref, lse_ref, yr)
        rerr = np.abs(rl_gpu.double().numpy() - rl_ref)
        rtol_ = ltol + 2.0 * bound[np.arange(len(rows)), yr]
        assert np.all(rerr <= rtol_), f"row loss: max err {rerr.max():.3e}"
        rep += f"  row loss max err {rerr.max():.2e}"
    # partials against the GPU's own logits: maximum bit for bit, sum within 1e-5 relative
    zt = z_gpu.float().numpy().reshape(len(rows), N // PART_W, PART_W)
    pm, ps = part_gpu[..., 0].numpy(), part_gpu[..., 1].numpy()
    assert np.array_equal(pm, zt.max(axis=2)), "tile maxima differ from the maxima of the logits"
    ps_ref = np.exp(zt.astype(np.float64) - pm[..., None].astype(np.float64)).sum(axis=2)
    perr = np.abs(ps.astype(np.float64) - ps_ref) / ps_ref
    assert perr.max() <= 1e-5, f"tile sums: max rel err {perr.max():.3e}"
    # and the merge of the GPU's partials, in float64, gives the GPU's LSE
    merged = lm.merge_partials(pm, ps)
    merr = np.abs(merged - lse_gpu.double().numpy())
    assert merr.max() <= 2e-5, f"merge of partials vs LSE: {merr.max():.3e}"
    return rep


def run(x, w, y):
    xd, wd = x.to(DEV), w.to(DEV)
    yd = y.to(DEV) if y is not None else None
    M, N = x.shape[0], w.shape[0]
    ws = torch.full((lmhead_workspace_bytes(M, N, x.shape[1]) // 4,), float("nan"), device=DEV)
    z, lse, rl, loss = lmhead_fwd(xd, wd, yd, workspace=ws)
    torch.cuda.synchronize()
    part = ws.view(M, N // PART_W, 2)
    return z, lse, rl, loss, part


SMALL = [
    # M, N, K, w_sigma, with targets
    (128, 128, 64, 0.02, True),
    (256, 384, 192, 0.02, True),
    (128, 256, 128, 1.0, True),      # two vocabulary tiles: six chiplets get no work
    (384, 1152, 128, 0.5, True),     # nine vocabulary tiles: chiplet 0 gets two
    (256, 2304, 320, 3.0, False),    # wide logits (sigma ~ 50): the merge rescale dominates; no targets
    (512, 1280, 768, 0.02, True),    # GPT-2's hidden size
    (4096, 8320, 128, 0.3, True),    # 33 x 16 tiles: every work group walks two or three tiles
]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: "-".join(map(str, c)))
def test_small_full(case):
    M, N, K, sig, with_y = case
    x, w, y = make_lmhead_inputs(M, N, K, sig, seed=4321 + M + N + K)
    say(f"lmhead small M{M} N{N} K{K} sigma{sig} targets={with_y}")
    z, lse, rl, loss, part = run(x, w, y if with_y else None)
    rows = np.arange(M)
    rep = check_rows(rows, x, w, y, z.cpu(), lse.cpu(), rl.cpu() if with_y else None, part.cpu(), N)
    if with_y:
        l64 = rl.cpu().double().mean().item()
        assert abs(loss.item() - l64) <= 1e-6 * abs(l64) + 1e-7
        _, _, _, loss_ref = lm.lmhead_fwd(x, w, y)
        assert abs(loss.item() - loss_ref) <= float(_lse_tol(lm.dot_error_bound(x, w).max(), N) * 3)
    else:
        assert rl is None and loss is None
    print("  " + rep, flush=True)


def test_out_of_range_target_gives_nan_for_that_row_only():
    M, N, K = 128, 256, 64
    x, w, y = make_lmhead_inputs(M, N, K, 0.02, seed=99)
    y = y.clone()
    y[3], y[77] = N, -1
    say("lmhead out-of-range targets")
    z, lse, rl, loss, _ = run(x, w, y)
    rl = rl.cpu()
    assert math.isnan(rl[3].item()) and math.isnan(rl[77].item())
    ok = torch.ones(M, dtype=torch.bool)
    ok[3] = ok[77] = False
    assert torch.isfinite(rl[ok]).all()
    assert math.isnan(loss.item())


def test_deterministic():
    M, N, K = 256, 1280, 256
    x, w, y = make_lmhead_inputs(M, N, K, 0.3, seed=7)
    say("lmhead determinism")
    a = run(x, w, y)
    b = run(x, w, y)
    for t, u in zip(a, b):
        assert torch.equal(t.cpu().view(-1).view(torch.int32), u.cpu().view(-1).view(torch.int32))


@pytest.mark.parametrize("wl", LMHEAD_WORKLOADS, ids=lambda w: w.name)
def test_gpt2_head_full_size_sampled_rows(wl):
    x, w, y = make_lmhead_inputs(wl.M, wl.N, wl.K, wl.w_sigma, wl.seed)
    say(f"lmhead full size {wl.name}")
    z, lse, rl, loss, part = run(x, w, y)
    g = np.random.default_rng(5)
    # first and last rows of the first and last token tiles, plus random rows
    rows = np.unique(np.concatenate([[0, 1, 127, 128, wl.M - 129, wl.M - 1], g.choice(wl.M, 26, replace=False)]))
    ri = torch.as_tensor(rows)
    rep = check_rows(rows, x, w, y, z[ri.to(DEV)].cpu(), lse.cpu()[ri], rl.cpu()[ri], part[ri.to(DEV)].cpu(), wl.N)
    rl_all = rl.cpu().double()
    assert torch.isfinite(rl_all).all()
    l64 = rl_all.mean().item()
    assert abs(loss.item() - l64) <= 1e-6 * abs(l64)
    # every row's LSE is the float64 merge of its GPU partials
    merged = lm.merge_partials(part[..., 0].cpu().numpy(), part[..., 1].cpu().numpy())
    assert np.abs(merged - lse.cpu().double().numpy()).max() <= 2e-5
    print("  " + rep + f"  loss {loss.item():.6f}", flush=True)
