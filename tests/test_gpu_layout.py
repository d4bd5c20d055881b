"""The [B, S, H, D] storage order (CATTN_BSHD) through the C ABI.

The kernels read and write sequence-major tensors in place; the arithmetic is
the same as for [B, H, S, D], so every output must equal the heads-major run
bit for bit, and the heads-major view of it must meet the float64 oracle's
tolerance.  Cases span both dtypes and head dimensions, causal and not, ragged
lengths, several heads (so a row stride differs from D) and the GPT-2 small
workload at full size.
"""

import math

import pytest
import torch

import oracle.attn_oracle as orc
from paper_2608_00029_amd import attn_bwd, attn_fwd
from paper_2608_00029_amd.workloads import BY_NAME, make_inputs, workload_inputs
from parity_util import check_tensor, say

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def to_bshd(t):
    return t.transpose(1, 2).contiguous()


def to_bhsd(t):
    return t.transpose(1, 2).contiguous()


def run(q, k, v, do, scale, causal, layout):
    o, lse = attn_fwd(q, k, v, scale, causal, layout=layout)
    dq, dk, dv = attn_bwd(q, k, v, o, do, lse, scale, causal, layout=layout)
    torch.cuda.synchronize()
    return o, lse, dq, dk, dv


CASES = [
    # dtype, B, H, S, D, causal
    ("bf16", 2, 3, 300, 64, True),
    ("bf16", 1, 4, 257, 128, True),
    ("bf16", 2, 2, 200, 64, False),
    ("f32", 1, 3, 200, 64, True),
    ("f32", 2, 2, 129, 128, False),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "-".join(map(str, c)))
def test_bshd_matches_bhsd_and_oracle(cuda, case):
    dtype, B, H, S, D, causal = case
    scale = 1.0 / math.sqrt(D)
    q, k, v, do = make_inputs(B, H, S, D, dtype, seed=4242 + S + H)
    say(f"layout bshd {case}")
    dev = [t.to(DEV) for t in (q, k, v, do)]
    ref = run(*dev, scale, causal, "bhsd")
    got = run(*[to_bshd(t) for t in dev], scale, causal, "bshd")
    names = ("o", "lse", "dq", "dk", "dv")
    for n, g, r in zip(names, got, ref):
        g = g if n == "lse" else to_bhsd(g)
        assert torch.equal(g, r), f"{n}: [B,S,H,D] result differs from [B,H,S,D]"
    ro, rlse = orc.attn_fwd(q, k, v, scale, causal)
    rdq, rdk, rdv = orc.attn_bwd(q, k, v, do, scale, causal)
    for n, g, r in zip(names, got, (ro, rlse, rdq, rdk, rdv)):
        g = g if n == "lse" else to_bhsd(g)
        check_tensor(n, dtype, g.cpu(), r)


@pytest.mark.parametrize("name", ["gpt2_small_B8_H12_S1024_D64", "long_ctx_B2_H16_S4096_D128"])
def test_bshd_full_size(cuda, name):
    """Full-size workloads (D = 64 and D = 128, whose kernels address their
    LDS fragments differently) in both storage orders: bit for bit equal."""
    w = BY_NAME[name]
    say(f"layout bshd full {w.name}")
    dev = [t.to(DEV) for t in workload_inputs(w)]
    ref = run(*dev, w.scale, w.causal, "bhsd")
    got = run(*[to_bshd(t) for t in dev], w.scale, w.causal, "bshd")
    for n, g, r in zip(("o", "lse", "dq", "dk", "dv"), got, ref):
        g = g if n == "lse" else to_bhsd(g)
        assert torch.equal(g, r), f"{n}: [B,S,H,D] result differs from [B,H,S,D] at full size"


@pytest.mark.parametrize("causal", [True, False])
def test_bshd_unsplit_ragged_grid(cuda, causal):
    """A grid that takes the unsplit D = 64 kernels, with a ragged sequence end,
    in both storage orders: bit for bit the same results."""
    B, H, S, D = 4, 32, 1000, 64
    q, k, v, do = make_inputs(B, H, S, D, "bf16", seed=777 + int(causal))
    say(f"layout bshd unsplit B{B} H{H} S{S} causal={causal}")
    dev = [t.to(DEV) for t in (q, k, v, do)]
    ref = run(*dev, 0.125, causal, "bhsd")
    got = run(*[to_bshd(t) for t in dev], 0.125, causal, "bshd")
    for n, g, r in zip(("o", "lse", "dq", "dk", "dv"), got, ref):
        g = g if n == "lse" else to_bhsd(g)
        assert torch.equal(g, r), f"{n}: [B,S,H,D] result differs from [B,H,S,D]"


def test_layout_argument_checked(cuda):
    q = torch.zeros((1, 2, 64, 64), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(ValueError):
        attn_fwd(q, q, q, 0.125, True, layout="sbhd")
