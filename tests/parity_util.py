"""Shared helpers of the GPU parity tests: error metrics and the tolerances.

Tolerances (fixed before any kernel ran, from the acceptance bar of the
attention hot path):
  * float32 mode: max |GPU - oracle| <= 1e-5 on O, LSE, dQ, dK, dV;
  * bfloat16 mode: relative L2 error ||GPU - oracle|| / ||oracle|| <= 1e-2 on
    O, dQ, dK, dV, and max |LSE_GPU - LSE_oracle| <= 1e-3.
"""

import sys

import numpy as np
import torch

F32_MAX_ABS = 1e-5
BF16_REL_L2 = 1e-2
LSE_MAX_ABS = 1e-3


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
    """Assert the tolerance for one output; return a one-line report."""
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
