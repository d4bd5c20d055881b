"""Causal loop clamping changes no result (section 4.2, exploiting causality in
the loop bounds).  libcattn_noclamp.so is the same library with the bf16
attention loops visiting every tile -- the forward and dQ loops running past
the diagonal, the dK/dV loop starting at query tile 0 -- and masking the tiles
past the diagonal entirely.  Its O, LSE, dQ, dK and dV equal the product
library's value for value on grids that run the unsplit kernels in both
(+0 and -0 compare equal: an added zero product may flip the sign of an exact
zero)."""

import ctypes
import os

import pytest
import torch

from paper_2608_00029_amd import binding
from paper_2608_00029_amd.build import NOCLAMP_LIB
from paper_2608_00029_amd.workloads import make_inputs
from parity_util import say

pytestmark = pytest.mark.gpu

DEV = "cuda:0"

# grids that take the unsplit kernels in the product library too: head
# dimension 128 always, head dimension 64 from 768 work groups of 128 queries
CASES = [
    # B, H, S, D, sigma
    (8, 12, 1024, 64, 1.0),   # GPT-2 small
    (4, 24, 1000, 64, 1.0),   # ragged end
    (4, 32, 1000, 64, 1.0),   # 1024 work groups: the dQ kernel's streamed four-wave form
    (1, 2, 300, 128, 1.0),    # small grid, ragged end
    (1, 2, 384, 128, 3.0),    # peaked softmax
]


def _load(path):
    L = ctypes.CDLL(path)
    vp, i, f = ctypes.c_void_p, ctypes.c_int, ctypes.c_float
    L.cattn_attn_fwd.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, f, i, i, vp]
    L.cattn_attn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, f, i, i, vp]
    L.cattn_bwd_workspace_bytes.argtypes = [i, i, i, i]
    L.cattn_bwd_workspace_bytes.restype = ctypes.c_size_t
    return L


def _run(L, q, k, v, do, scale):
    B, H, S, D = q.shape
    o, dq, dk, dv = (torch.empty_like(q) for _ in range(4))
    lse = torch.empty((B, H, S), dtype=torch.float32, device=DEV)
    ws = torch.empty((L.cattn_bwd_workspace_bytes(B, H, S, D) // 4,), dtype=torch.float32, device=DEV)
    sp = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    p = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    assert L.cattn_attn_fwd(p(q), p(k), p(v), p(o), p(lse), B, H, S, D, scale, 1, binding.CATTN_BF16, sp) == 0
    assert L.cattn_attn_bwd(p(q), p(k), p(v), p(o), p(do), p(lse), p(dq), p(dk), p(dv), p(ws), B, H, S, D, scale,
                            1, binding.CATTN_BF16, sp) == 0
    torch.cuda.synchronize()
    return o, lse, dq, dk, dv


@pytest.fixture(scope="module")
def noclamp():
    if not os.path.exists(NOCLAMP_LIB):
        pytest.fail(f"{NOCLAMP_LIB} is not built (run __graft_entry__.build())")
    return _load(NOCLAMP_LIB)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "-".join(map(str, c)))
def test_clamped_equals_unclamped(cuda, noclamp, case):
    B, H, S, D, sigma = case
    say(f"no-clamp B={B} H={H} S={S} D={D} sigma={sigma}")
    q, k, v, do = (t.to(DEV) for t in make_inputs(B, H, S, D, "bf16", seed=7300 + S, qk_sigma=sigma))
    scale = D ** -0.5
    ref = _run(_load(binding.library_path()), q, k, v, do, scale)
    got = _run(noclamp, q, k, v, do, scale)
    for name, g, r in zip(("o", "lse", "dq", "dk", "dv"), got, ref):
        assert torch.equal(g, r), f"{name}: the unclamped loops give a different result"
