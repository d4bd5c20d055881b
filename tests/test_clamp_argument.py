"""Why the causal loop clamping is exact (section 4.2): a score masked with the
finite sentinel -1e30 contributes exactly 0 in each kernel's float32 arithmetic,
for every scale the library accepts and any realistic softmax offset or LSE.

The kernels form, for a masked score (c = scale * log2 e):
  forward  p = exp2(fma(-1e30, c, -m c))   m: the running offset (a real score)
  dQ       p = exp2(fma(-1e30, c, -LSE log2 e))
  dK/dV    p = exp2(-1e30 c)
An exponent at or below -150 has no float32 value but 0, so p = 0, the
probability sum gains 0 (the lazy offset never moves on it: 0 is inside the
bound) and every contraction adds exact zero products.  The GPU test
test_gpu_noclamp.py checks the whole kernels end to end."""

import numpy as np

MASKED = np.float32(-1.0e30)
LOG2E = np.float32(1.4426950408889634)


def fma32(a, b, c):
    """float32 fused multiply-add: exact product and sum in float64, one rounding."""
    return np.float32(np.float64(a) * np.float64(b) + np.float64(c))


def test_masked_probability_is_exactly_zero():
    scales = [1e-20, 1e-12, 1e-6, 1e-3, 0.125, 128 ** -0.5, 1.0, 10.0, 1e3, 1e6]
    offsets = [-1e25, -1e10, -1e3, -30.0, -1.0, 0.0, 1.0, 30.0, 1e3, 1e10, 1e25]
    lses = [-1e6, -100.0, 0.0, 1.0, 100.0, 1e6]
    for s in scales:
        c = np.float32(s) * LOG2E
        assert np.isfinite(MASKED * c)
        for m in offsets:
            mc = np.float32(m) * c
            if not np.isfinite(mc):
                continue
            x = fma32(MASKED, c, -mc)
            assert x <= -150 and np.exp2(x) == 0.0, (s, m)
        for lse in lses:
            x = fma32(MASKED, c, -np.float32(lse) * LOG2E)
            assert np.exp2(x) == 0.0, (s, lse)
        assert np.exp2(MASKED * c) == 0.0, s


def test_outside_the_range_the_sentinel_fails():
    """Below the accepted scale range the sentinel no longer vanishes, which is
    why the library rejects such scales."""
    c = np.float32(1e-29) * LOG2E
    assert np.exp2(MASKED * c) > 0.0
