"""CPU reference ("oracle") for the fused language-model loss head, forward.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import this module.  The product path (the
HIP library and its Python binding) never imports, calls or links it, and this
module imports nothing from the product package.

What it computes (paper section 4.1, case study "Fusing a Reduction into a
Contraction Epilogue", and the fused loss-head evaluation of section 6): the
language-model head projects the final hidden states onto the vocabulary and
feeds a softmax cross-entropy loss.  For hidden states X [M, K], the head's
weight W [N, K] (one row per vocabulary entry, no bias) and target ids
y [M]:

    Z    = X W^T                                  logits [M, N]
    LSE  = log sum_j exp(Z[i, j])                 per row, natural log
    l_i  = LSE_i - Z[i, y_i]                      per-row loss
    loss = (1/M) sum_i l_i                        mean over rows

The fused method accumulates the row maximum and the row sum of exponentials
per N tile inside the contraction's epilogue, and merges the per-tile
partials afterwards.  The merge is not the fold itself: two partial sums are
added only after one is rescaled by the exponential of the difference of their
maxima.  `tile_partials` and `merge_partials` write exactly that split out;
the definition above (`row_logsumexp`) is the plain one, and the tests pin
that the two agree for every tile width.

Every input is upcast exactly to float64 first (bf16 and fp32 values are
exactly representable in float64).
"""

from __future__ import annotations

import numpy as np


def _as_f64(x) -> np.ndarray:
    """Exact upcast of a numpy array or a CPU torch tensor to float64."""
    if hasattr(x, "detach"):  # torch tensor (bf16 has no numpy dtype)
        x = x.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def logits(x, w) -> np.ndarray:
    """Z = X W^T (section 4.1: the loss head's projection onto the vocabulary)."""
    return _as_f64(x) @ _as_f64(w).T


def row_logsumexp(z) -> np.ndarray:
    """log sum_j exp(z[i, j]) per row, shifted by the row maximum for range."""
    z = _as_f64(z)
    m = z.max(axis=1)
    return m + np.log(np.exp(z - m[:, None]).sum(axis=1))


def tile_partials(z, tile: int):
    """Per-(row, N-tile) statistics the epilogue keeps: the tile's row maximum
    and the sum of exp(z - that maximum) over the tile's columns (section 4.1).
    The last tile may be narrower.  Returns (max [M, T], sum [M, T])."""
    z = _as_f64(z)
    M, N = z.shape
    nt = (N + tile - 1) // tile
    pm = np.empty((M, nt))
    ps = np.empty((M, nt))
    for t in range(nt):
        blk = z[:, t * tile:(t + 1) * tile]
        pm[:, t] = blk.max(axis=1)
        ps[:, t] = np.exp(blk - pm[:, t:t + 1]).sum(axis=1)
    return pm, ps


def merge_partials(pm, ps) -> np.ndarray:
    """Combine per-tile (max, sum) into the row log-sum-exp: the running sums are
    added only after rescaling each by exp(its maximum - the overall maximum)
    (section 4.1: the merge region that is not the fold)."""
    pm, ps = _as_f64(pm), _as_f64(ps)
    m = pm.max(axis=1)
    s = (ps * np.exp(pm - m[:, None])).sum(axis=1)
    return m + np.log(s)


def row_losses(z, lse, targets) -> np.ndarray:
    """l_i = LSE_i - Z[i, y_i] (softmax cross entropy of row i)."""
    z = _as_f64(z)
    y = np.asarray(targets, dtype=np.int64)
    return _as_f64(lse) - z[np.arange(z.shape[0]), y]


def lmhead_fwd(x, w, targets=None):
    """(Z, LSE, per-row losses, mean loss) of the loss head; losses None without targets."""
    z = logits(x, w)
    lse = row_logsumexp(z)
    if targets is None:
        return z, lse, None, None
    rl = row_losses(z, lse, targets)
    return z, lse, rl, float(rl.mean())


def dot_error_bound(x, w) -> np.ndarray:
    """Bound on |fl32(Z) - Z| for a float32 accumulation of the K products of
    each logit in any order (products of bf16 values are exact in float32):
    gamma_K * sum_k |x_ik w_jk|, gamma_K = K u / (1 - K u), u = 2^-24."""
    xa, wa = np.abs(_as_f64(x)), np.abs(_as_f64(w))
    K = xa.shape[1]
    u = 2.0 ** -24
    gamma = K * u / (1.0 - K * u)
    return gamma * (xa @ wa.T)
