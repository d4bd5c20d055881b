"""CPU reference ("oracle") for the memory-bound neighbours of attention in the
GPT-2 training step: LayerNorm, GELU and softmax cross entropy, forward and
backward.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import this module.  The product path (the
HIP library and its Python binding) never imports, calls or links it, and this
module imports nothing from the product package.

The paper measures these three operators on their own (section 6,
"Memory-Bound Operators": LayerNorm at 16 x 1024 x 768, GELU at
16 x 1024 x 3072, fused softmax cross entropy at 16 x 1024 x 50304, forward and
backward, float32 tensors) and names GELU, softmax cross entropy and their
backward ops in its dialect (section 3, the language-model-head IR example).
Each is a plain definition; the oracle writes it out in float64:

LayerNorm over the last axis of x [R, C], per row r:
    mu_r   = (1/C) sum_c x[r, c]
    var_r  = (1/C) sum_c (x[r, c] - mu_r)^2          (biased variance)
    rstd_r = 1 / sqrt(var_r + eps)
    xhat   = (x - mu_r) * rstd_r
    y      = xhat * gamma + beta
  backward, for dy:
    g      = dy * gamma
    dx     = rstd_r * (g - mean_c(g) - xhat * mean_c(g * xhat))
    dgamma = sum_r dy * xhat,   dbeta = sum_r dy

GELU, the tanh form GPT-2 uses:
    u    = sqrt(2/pi) * (x + 0.044715 x^3)
    y    = 0.5 x (1 + tanh u)
    dy/dx = 0.5 (1 + tanh u) + 0.5 x (1 - tanh^2 u) sqrt(2/pi) (1 + 3 * 0.044715 x^2)

Softmax cross entropy of logits z [R, V] with target ids t [R]:
    lse_r  = log sum_j exp(z[r, j])
    l_r    = lse_r - z[r, t_r]
    loss   = (1/R) sum_r l_r
  backward, for an upstream factor s on every row loss (s = dloss / R for the
  mean):
    dz[r, j] = s * (exp(z[r, j] - lse_r) - [j == t_r])

Readings of the paper (it states none of these):
  * GELU is the tanh approximation (GPT-2's activation); the exact erf form
    differs from it by less than 1e-3 everywhere (pinned in the tests).
  * LayerNorm uses the biased variance and eps inside the square root, the
    convention of GPT-2 and of the common framework layer; eps defaults to
    1e-5.
  * The cross-entropy backward recomputes the softmax from the logits and the
    saved lse instead of reading a stored softmax tensor, which is the same
    value; a target outside [0, V) makes that row's loss and gradient NaN.

Every input is upcast exactly to float64 first.
"""

from __future__ import annotations

import math

import numpy as np

GELU_C = math.sqrt(2.0 / math.pi)
GELU_A = 0.044715


def _as_f64(x) -> np.ndarray:
    """Exact upcast of a numpy array or a CPU torch tensor to float64."""
    if hasattr(x, "detach"):
        x = x.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


# ---------------------------------------------------------------------------
# LayerNorm
# ---------------------------------------------------------------------------
def layernorm_stats(x, eps: float = 1e-5):
    """(mean [R], rstd [R]) of the rows of x [R, C]: biased variance, eps inside the root."""
    x = _as_f64(x)
    mu = x.mean(axis=1)
    var = ((x - mu[:, None]) ** 2).mean(axis=1)
    return mu, 1.0 / np.sqrt(var + eps)


def layernorm_fwd(x, gamma, beta, eps: float = 1e-5):
    """y = (x - mean) * rstd * gamma + beta per row; returns (y, mean, rstd)."""
    x, gamma, beta = _as_f64(x), _as_f64(gamma), _as_f64(beta)
    mu, rstd = layernorm_stats(x, eps)
    xhat = (x - mu[:, None]) * rstd[:, None]
    return xhat * gamma[None, :] + beta[None, :], mu, rstd


def layernorm_bwd(x, gamma, dy, eps: float = 1e-5):
    """(dx, dgamma, dbeta) of LayerNorm for upstream dy, statistics recomputed from x."""
    x, gamma, dy = _as_f64(x), _as_f64(gamma), _as_f64(dy)
    mu, rstd = layernorm_stats(x, eps)
    xhat = (x - mu[:, None]) * rstd[:, None]
    g = dy * gamma[None, :]
    dx = rstd[:, None] * (g - g.mean(axis=1, keepdims=True) - xhat * (g * xhat).mean(axis=1, keepdims=True))
    return dx, (dy * xhat).sum(axis=0), dy.sum(axis=0)


# ---------------------------------------------------------------------------
# GELU (tanh form)
# ---------------------------------------------------------------------------
def gelu_fwd(x) -> np.ndarray:
    x = _as_f64(x)
    return 0.5 * x * (1.0 + np.tanh(GELU_C * (x + GELU_A * x ** 3)))


def gelu_bwd(x, dy) -> np.ndarray:
    """dx = dy * GELU'(x)."""
    x, dy = _as_f64(x), _as_f64(dy)
    t = np.tanh(GELU_C * (x + GELU_A * x ** 3))
    d = 0.5 * (1.0 + t) + 0.5 * x * (1.0 - t * t) * GELU_C * (1.0 + 3.0 * GELU_A * x * x)
    return dy * d


# ---------------------------------------------------------------------------
# Softmax cross entropy
# ---------------------------------------------------------------------------
def sce_lse(z) -> np.ndarray:
    """log sum_j exp(z[r, j]) per row, shifted by the row maximum for range."""
    z = _as_f64(z)
    m = z.max(axis=1)
    return m + np.log(np.exp(z - m[:, None]).sum(axis=1))


def _target_values(z: np.ndarray, targets) -> np.ndarray:
    t = np.asarray(targets.detach().cpu().numpy() if hasattr(targets, "detach") else targets).astype(np.int64)
    ok = (t >= 0) & (t < z.shape[1])
    vals = np.full(z.shape[0], np.nan)
    vals[ok] = z[np.nonzero(ok)[0], t[ok]]
    return vals


def sce_fwd(z, targets):
    """(lse [R], row losses [R], mean loss) of logits z [R, V] against target ids."""
    z = _as_f64(z)
    lse = sce_lse(z)
    rl = lse - _target_values(z, targets)
    return lse, rl, rl.mean()


def sce_bwd(z, targets, scale: float) -> np.ndarray:
    """dz = scale * (softmax(z) - onehot(targets)), rows with an invalid target all NaN."""
    z = _as_f64(z)
    t = np.asarray(targets.detach().cpu().numpy() if hasattr(targets, "detach") else targets).astype(np.int64)
    p = np.exp(z - sce_lse(z)[:, None])
    ok = (t >= 0) & (t < z.shape[1])
    rows = np.nonzero(ok)[0]
    p[rows, t[ok]] -= 1.0
    p[~ok, :] = np.nan
    return scale * p
