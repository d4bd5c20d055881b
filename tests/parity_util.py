"""Shared helpers of the GPU parity tests: error metrics and the tolerances.

Tolerances of the attention hot path (fixed before any kernel ran, from its
acceptance bar):
  * float32 mode: max |GPU - oracle| <= 1e-5 on O, LSE, dQ, dK, dV;
  * bfloat16 mode: relative L2 error ||GPU - oracle|| / ||oracle|| <= 1e-2 on
    O, dQ, dK, dV, and max |LSE_GPU - LSE_oracle| <= 1e-3.

bfloat16 mode is also held to a per-element bound, so that an error confined
to a few rows (a diagonal or ragged tile, one head) cannot hide under the
global relative L2.  It is derived from the arithmetic of the kernels:

  Every output element is a float sum of terms, each a softmax-derived factor
  (P, or dS = P (dP - D)) times an input element.  The factor is rounded to
  bf16 before its contraction (relative error <= u = 2^-8, bf16 keeping 8
  significant bits), the float sum of
  n <= S terms of D-long dot products adds at most (S + D) 2^-24 relative to
  the terms' absolute sum, and the result is rounded to bf16 (<= u of the
  element, itself <= the terms' absolute sum).  P carries a relative error
  eps_P from the score contraction (|delta s| <= scale D 2^-24 max|q| max|k|)
  and, in the backward, from the LSE it is recomputed with (the measured LSE
  error).  So, with M the terms' absolute sum from
  oracle.attn_term_magnitudes,

      |O - O_ref|   <= tau_O M_o,        tau_O = 2u + (S + D) 2^-24 + 2 eps_s
      |dV - dV_ref| <= tau_B M_dv,       tau_B = 2u + (S + D) 2^-24 + eps_s + err_LSE
      |dQ - dQ_ref| <= scale (tau_B G_dq + tau_D H_dq),  tau_D = tau_O + D 2^-24
      |dK - dK_ref| <= scale (tau_B G_dk + tau_D H_dk)

  where the H terms carry the error of D = rowsum(dO * O) formed from the
  forward's rounded O.  Values below the smallest normal float, 2^-126, are
  flushed to zero (probabilities, dS and the outputs): each flushed factor
  drops a term of at most 2^-126 max|x| (x the other operand), so every bound
  also carries (S max|x| + 1) 2^-126 (times scale for dQ and dK), which only
  matters where the exact values themselves are that small.  The tests check
  every element against its bound and every row's L2 error against the L2
  norm of its row of bounds.
"""

import sys

import numpy as np
import torch

F32_MAX_ABS = 1e-5
BF16_REL_L2 = 1e-2
LSE_MAX_ABS = 1e-3
U_BF16 = 2.0 ** -8  # bf16 keeps 8 significant bits: unit roundoff 2^-8
U_F32 = 2.0 ** -24


def say(msg: str) -> None:
    """Name the case before a GPU step (flushed, so a fault still shows it)."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def to64(t) -> np.ndarray:
    if isinstance(t, torch.Tensor):
        return t.detach().to("cpu").double().numpy()
    return np.asarray(t, dtype=np.float64)


def rel_l2(got, ref) -> float:
    got, ref = to64(got), to64(ref)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def max_abs(got, ref) -> float:
    got, ref = to64(got), to64(ref)
    return float(np.max(np.abs(got - ref))) if got.size else 0.0


def check_tensor(name: str, dtype: str, got, ref) -> str:
    """Assert the global tolerance for one output; return a one-line report."""
    got64, ref64 = to64(got), to64(ref)
    assert np.all(np.isfinite(got64)), f"{name}: non-finite values"
    if name == "lse":
        err = max_abs(got64, ref64)
        tol = F32_MAX_ABS if dtype == "f32" else LSE_MAX_ABS
        assert err <= tol, f"{name}: max abs {err:.3e} > {tol:.1e}"
        return f"{name} maxabs={err:.2e}"
    if dtype == "f32":
        err = max_abs(got64, ref64)
        assert err <= F32_MAX_ABS, f"{name}: max abs {err:.3e} > {F32_MAX_ABS:.1e}"
        return f"{name} maxabs={err:.2e}"
    err = rel_l2(got64, ref64)
    assert err <= BF16_REL_L2, f"{name}: rel L2 {err:.3e} > {BF16_REL_L2:.1e}"
    return f"{name} relL2={err:.2e}"


def bf16_bounds(q, k, v, do, mags, scale: float, lse_err: float):
    """Per-element error bounds of O, dQ, dK, dV in bf16 mode ([B, H, S, D]
    each), from the term magnitudes of the oracle and the measured LSE error."""
    q64, k64 = to64(q), to64(k)
    S, D = q64.shape[2], q64.shape[3]
    qn = np.linalg.norm(q64, axis=-1).max(axis=-1)  # [B, H]
    kn = np.linalg.norm(k64, axis=-1).max(axis=-1)
    eps_s = (scale * D * U_F32 * qn * kn)[..., None, None]
    acc = (S + D) * U_F32
    tau_o = 2 * U_BF16 + acc + 2 * eps_s
    tau_b = 2 * U_BF16 + acc + eps_s + lse_err
    tau_d = tau_o + D * U_F32
    tiny = 2.0 ** -126
    flush = lambda x: (S * np.abs(to64(x)).max() + 1) * tiny  # noqa: E731
    return {"o": tau_o * mags["m_o"] + flush(v), "dv": tau_b * mags["m_dv"] + flush(do),
            "dq": scale * (tau_b * mags["g_dq"] + tau_d * mags["h_dq"] + flush(k)),
            "dk": scale * (tau_b * mags["g_dk"] + tau_d * mags["h_dk"] + flush(q))}


def check_bounded(name: str, got, ref, bound) -> str:
    """Assert |got - ref| <= bound element by element and, per row, the L2
    error <= the L2 norm of the row's bounds; report the largest ratios."""
    err = np.abs(to64(got) - to64(ref))
    bound = np.asarray(bound)
    assert np.all(bound > 0) or np.all(err[bound == 0] == 0), f"{name}: zero bound with nonzero error"
    with np.errstate(divide="ignore", invalid="ignore"):
        elem = np.where(bound > 0, err / bound, 0.0)
        rows = np.linalg.norm(err, axis=-1) / np.maximum(np.linalg.norm(bound, axis=-1), 1e-300)
    e_max, r_max = float(elem.max()), float(rows.max())
    if e_max > 1.0:
        idx = np.unravel_index(int(np.argmax(elem)), elem.shape)
        raise AssertionError(f"{name}: element {idx} error {err[idx]:.3e} > bound {bound[idx]:.3e}")
    assert r_max <= 1.0, f"{name}: a row's L2 error exceeds its bound (ratio {r_max:.3f})"
    return f"{name} elem/bound={e_max:.2f} row/bound={r_max:.2f}"
