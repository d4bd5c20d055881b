"""The C-ABI library loads on a host without a GPU, exports every symbol that
include/cattn.h declares, and rejects bad arguments on the host before any
HIP call (no kernel is launched by these tests)."""

import ctypes
import os
import re

import pytest

from paper_2608_00029_amd import binding as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cattn.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cattn_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(b.library_path()):
        pytest.fail("libcattn.so is not built (run __graft_entry__.build())")
    return b.lib()


def test_header_declares_expected_entry_points():
    assert declared_functions() == sorted(b.EXPORTED)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert ctypes.cast(getattr(lib, name), ctypes.c_void_p).value


def test_status_strings(lib):
    assert b.status_string(0) == "CATTN_OK"
    assert b.status_string(1) == "CATTN_ERR_INVALID_ARG"
    assert b.status_string(2) == "CATTN_ERR_UNSUPPORTED"
    assert b.status_string(3) == "CATTN_ERR_HIP"
    assert b.status_string(77) == "unknown status"


def test_workspace_bytes(lib):
    assert b.workspace_bytes(8, 12, 1024, 64) == 2 * 8 * 12 * 1024 * 4
    assert b.workspace_bytes(1, 2, 33, 64) == 2 * 1 * 2 * 64 * 4  # rows padded to a multiple of 32
    assert b.workspace_bytes(0, 12, 1024, 64) == 0
    assert b.workspace_bytes(-1, 12, 1024, 64) == 0


# Fake, non-NULL "device" addresses: every case below is rejected on the host
# before anything is enqueued, so they are never dereferenced.
P = [0x10000000 * (i + 1) for i in range(10)]


@pytest.mark.parametrize("args,status", [
    ((1, 1, 16, 64, 0.125, 1, 1), b.CATTN_OK),              # valid shape, but NULL pointers below
    ((-1, 1, 16, 64, 0.125, 1, 1), b.CATTN_ERR_INVALID_ARG),
    ((1, 1, 16, 0, 0.125, 1, 1), b.CATTN_ERR_INVALID_ARG),
    ((1, 1, 16, 64, 0.125, 1, 7), b.CATTN_ERR_INVALID_ARG),   # bad dtype
    ((1, 1, 16, 64, 0.0, 1, 1), b.CATTN_ERR_INVALID_ARG),     # scale must be > 0
    ((1, 1, 16, 64, float("nan"), 1, 1), b.CATTN_ERR_INVALID_ARG),
    ((1, 1, 16, 64, float("inf"), 1, 1), b.CATTN_ERR_INVALID_ARG),
    ((1, 1, 16, 64, 1e-25, 1, 1), b.CATTN_ERR_INVALID_ARG),   # below the masked-sentinel range
    ((1, 1, 16, 64, 1e7, 1, 1), b.CATTN_ERR_INVALID_ARG),     # above it
    ((1, 1, 16, 96, 0.125, 1, 1), b.CATTN_ERR_UNSUPPORTED),   # D not in {64, 128}
    ((1, 1, 16, 32, 0.125, 1, 0), b.CATTN_ERR_UNSUPPORTED),
    ((1, 1, 1 << 24, 128, 0.125, 1, 1), b.CATTN_ERR_UNSUPPORTED),  # S*D > 2^30
])
def test_fwd_argument_errors(lib, args, status):
    st = b.raw_fwd(0, 0, 0, 0, 0, *args)
    expected = b.CATTN_ERR_INVALID_ARG if status == b.CATTN_OK else status  # NULL pointers
    assert st == expected, b.last_error_string()
    assert b.last_error_string() != ""


def test_empty_problem_is_a_noop(lib):
    for B, H, S in ((0, 4, 16), (2, 0, 16), (2, 4, 0)):
        assert b.raw_fwd(0, 0, 0, 0, 0, B, H, S, 64, 0.125, 1, 1) == b.CATTN_OK
        assert b.raw_bwd(0, 0, 0, 0, 0, 0, 0, 0, 0, 0, B, H, S, 64, 0.125, 1, 1) == b.CATTN_OK


def test_fwd_rejects_overlapping_output(lib):
    B, H, S, D = 1, 2, 64, 64
    n = B * H * S * D * 2
    # o aliases q
    assert b.raw_fwd(P[0], P[1], P[2], P[0], P[3], B, H, S, D, 0.125, 1, 1) == b.CATTN_ERR_INVALID_ARG
    # lse starts inside v
    assert b.raw_fwd(P[0], P[1], P[2], P[3], P[2] + n - 4, B, H, S, D, 0.125, 1, 1) == b.CATTN_ERR_INVALID_ARG
    # o overlaps lse
    assert b.raw_fwd(P[0], P[1], P[2], P[3], P[3] + 16, B, H, S, D, 0.125, 1, 1) == b.CATTN_ERR_INVALID_ARG


def test_bwd_argument_errors(lib):
    B, H, S, D = 1, 2, 64, 64
    ok = dict(q=P[0], k=P[1], v=P[2], o=P[3], do=P[4], lse=P[5], dq=P[6], dk=P[7], dv=P[8], ws=P[9])

    def call(**kw):
        a = dict(ok, **kw)
        return b.raw_bwd(a["q"], a["k"], a["v"], a["o"], a["do"], a["lse"], a["dq"], a["dk"], a["dv"], a["ws"],
                         B, H, S, D, 0.125, 1, 1)

    assert call(ws=0) == b.CATTN_ERR_INVALID_ARG
    assert call(dq=P[0]) == b.CATTN_ERR_INVALID_ARG        # dq aliases q
    assert call(dk=P[6]) == b.CATTN_ERR_INVALID_ARG        # dk aliases dq
    assert call(ws=P[8] + 8) == b.CATTN_ERR_INVALID_ARG    # workspace inside dv
    assert call(ws=P[9] + 2) == b.CATTN_ERR_INVALID_ARG    # misaligned workspace
    assert b.raw_bwd(*[ok[k] for k in ("q", "k", "v", "o", "do", "lse", "dq", "dk", "dv", "ws")],
                     B, H, S, 80, 0.125, 1, 1) == b.CATTN_ERR_UNSUPPORTED


def test_binding_refuses_cpu_tensors(lib):
    import torch
    q = torch.zeros(1, 1, 8, 64)
    with pytest.raises(ValueError):
        b.attn_fwd(q, q, q, 0.125)


def test_unknown_layout_is_rejected_before_any_launch(lib):
    vp = __import__("ctypes").c_void_p
    fake = [vp(4096 * (i + 1)) for i in range(10)]  # never dereferenced: the layout check comes first
    for layout in (-1, 2, 7):
        st = lib.cattn_attn_fwd_ex(*fake[:5], 1, 2, 64, 64, 0.125, 1, 1, layout, vp(0))
        assert st == b.CATTN_ERR_INVALID_ARG
        assert "layout" in b.last_error_string()
        st = lib.cattn_attn_bwd_ex(*fake, 1, 2, 64, 64, 0.125, 1, 1, layout, vp(0))
        assert st == b.CATTN_ERR_INVALID_ARG


def test_empty_problem_in_either_layout_is_a_noop(lib):
    vp = __import__("ctypes").c_void_p
    for layout in (b.CATTN_BHSD, b.CATTN_BSHD):
        assert lib.cattn_attn_fwd_ex(*[vp(0)] * 5, 0, 2, 64, 64, 0.125, 1, 1, layout, vp(0)) == b.CATTN_OK


def test_lmhead_workspace_bytes(lib):
    assert b.lmhead_workspace_bytes(8192, 50304, 768) == 8192 * (50304 // 64) * 2 * 4
    assert b.lmhead_workspace_bytes(128, 128, 64) == 128 * 2 * 2 * 4
    assert b.lmhead_workspace_bytes(0, 128, 64) == 0
    assert b.lmhead_workspace_bytes(100, 128, 64) == 0  # unsupported shape


def test_lmhead_argument_errors(lib):
    vp = ctypes.c_void_p
    x, w, y, z, lse, rl, loss, ws = (vp(p) for p in P[:8])
    M, N, K = 128, 256, 64

    def call(*a, M=M, N=N, K=K):
        return lib.cattn_lmhead_fwd(*a, M, N, K, vp(0))

    assert call(x, w, y, z, lse, rl, loss, ws, M=-1) == b.CATTN_ERR_INVALID_ARG
    assert call(x, w, y, z, lse, rl, loss, ws, M=0) == b.CATTN_OK          # empty problem: nothing touched
    assert call(x, w, y, z, lse, rl, loss, ws, K=0) == b.CATTN_OK
    assert call(x, w, y, z, lse, rl, loss, ws, M=100) == b.CATTN_ERR_UNSUPPORTED
    assert call(x, w, y, z, lse, rl, loss, ws, N=200) == b.CATTN_ERR_UNSUPPORTED
    assert call(x, w, y, z, lse, rl, loss, ws, K=96) == b.CATTN_ERR_UNSUPPORTED
    assert call(vp(0), w, y, z, lse, rl, loss, ws) == b.CATTN_ERR_INVALID_ARG
    assert call(x, w, y, z, lse, vp(0), loss, ws) == b.CATTN_ERR_INVALID_ARG  # targets need row_loss
    assert call(x, w, y, z, lse, rl, loss, vp(0)) == b.CATTN_ERR_INVALID_ARG
    assert call(x, w, y, z, lse, rl, loss, vp(P[7] + 2)) == b.CATTN_ERR_INVALID_ARG  # misaligned workspace
    assert call(x, w, y, vp(P[0]), lse, rl, loss, ws) == b.CATTN_ERR_INVALID_ARG     # logits alias x
    assert call(x, w, y, z, vp(P[3] + 64), rl, loss, ws) == b.CATTN_ERR_INVALID_ARG  # lse inside logits
    assert call(x, w, y, z, lse, rl, loss, vp(P[1] + 4)) == b.CATTN_ERR_INVALID_ARG  # workspace inside w
    assert "overlap" in b.last_error_string()


def test_memops_argument_errors(lib):
    vp, ll = ctypes.c_void_p, ctypes.c_longlong
    p = [vp(a) for a in P]
    s0 = vp(0)
    # LayerNorm forward
    assert lib.cattn_layernorm_fwd(*p[:6], -1, 768, 1e-5, s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_layernorm_fwd(*p[:6], 16, 768, -1.0, s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_layernorm_fwd(*p[:6], 16, 768, float("nan"), s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_layernorm_fwd(*[vp(0)] * 6, 0, 768, 1e-5, s0) == b.CATTN_OK  # empty
    assert lib.cattn_layernorm_fwd(*p[:6], 16, 770, 1e-5, s0) == b.CATTN_ERR_UNSUPPORTED
    assert lib.cattn_layernorm_fwd(*p[:6], 16, 4100, 1e-5, s0) == b.CATTN_ERR_UNSUPPORTED
    assert lib.cattn_layernorm_fwd(vp(0), *p[1:6], 16, 768, 1e-5, s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_layernorm_fwd(vp(P[0] + 4), *p[1:6], 16, 768, 1e-5, s0) == b.CATTN_ERR_INVALID_ARG  # alignment
    assert lib.cattn_layernorm_fwd(p[0], p[1], p[2], p[0], p[4], p[5], 16, 768, 1e-5, s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_layernorm_fwd(*p[:4], vp(P[3] + 16), p[5], 16, 768, 1e-5, s0) == b.CATTN_ERR_INVALID_ARG
    # LayerNorm backward
    assert lib.cattn_layernorm_bwd(*p[:8], vp(0), 16, 768, s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_layernorm_bwd(*p[:8], vp(P[4] + 32), 16, 768, s0) == b.CATTN_ERR_INVALID_ARG  # ws inside dy
    assert lib.cattn_layernorm_bwd(*p[:9], 16, 6, s0) == b.CATTN_ERR_UNSUPPORTED
    assert lib.cattn_layernorm_bwd(*[vp(0)] * 9, 16, 0, s0) == b.CATTN_OK
    assert b.layernorm_bwd_workspace_bytes(16384, 768) == 512 * 2 * 768 * 4
    assert b.layernorm_bwd_workspace_bytes(20, 768) == 2 * 2 * 768 * 4
    assert b.layernorm_bwd_workspace_bytes(0, 768) == 0
    # GELU
    assert lib.cattn_gelu_fwd(p[0], p[1], ll(-1), s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_gelu_fwd(vp(0), vp(0), ll(0), s0) == b.CATTN_OK
    assert lib.cattn_gelu_fwd(p[0], p[0], ll(1024), s0) == b.CATTN_ERR_INVALID_ARG      # in place
    assert lib.cattn_gelu_bwd(p[0], p[1], vp(P[1] + 64), ll(1024), s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_gelu_bwd(p[0], vp(0), p[2], ll(1024), s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_gelu_fwd(vp(P[0] + 8), p[1], ll(1024), s0) == b.CATTN_ERR_INVALID_ARG
    # softmax cross entropy
    assert lib.cattn_sce_fwd(*p[:5], 16, 50302, s0) == b.CATTN_ERR_UNSUPPORTED
    assert lib.cattn_sce_fwd(*p[:5], -2, 50304, s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_sce_fwd(p[0], p[1], p[2], vp(0), p[4], 16, 50304, s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_sce_fwd(p[0], p[1], vp(P[0] + 64), p[3], p[4], 16, 50304, s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_sce_fwd(*[vp(0)] * 5, 0, 50304, s0) == b.CATTN_OK
    assert lib.cattn_sce_bwd(*p[:3], ctypes.c_float(float("inf")), p[3], 16, 50304, s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_sce_bwd(p[0], vp(0), p[2], ctypes.c_float(1.0), p[3], 16, 50304, s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_sce_bwd(*p[:3], ctypes.c_float(1.0), p[0], 16, 50304, s0) == b.CATTN_ERR_INVALID_ARG
    assert lib.cattn_sce_bwd(*p[:3], ctypes.c_float(1.0), p[3], 16, 10, s0) == b.CATTN_ERR_UNSUPPORTED


def test_memops_binding_refuses_cpu_tensors(lib):
    import torch
    x = torch.zeros(4, 8)
    with pytest.raises(ValueError):
        b.gelu_fwd(x)
    with pytest.raises(ValueError):
        b.layernorm_fwd(x, torch.ones(8), torch.zeros(8))
    with pytest.raises(ValueError):
        b.sce_fwd(x)


def test_fwd_rejects_misaligned_pointers(lib):
    """Q, K, V, O must start on 16 bytes (rows move in 16-byte pieces), LSE on 4."""
    B, H, S, D = 1, 2, 64, 64
    good = [P[0], P[1], P[2], P[3], P[4]]  # never passed as is: that call would launch
    for i, off in ((0, 2), (1, 8), (2, 4), (3, 2), (4, 2)):
        a = list(good)
        a[i] += off
        assert b.raw_fwd(*a, B, H, S, D, 0.125, 1, 1) == b.CATTN_ERR_INVALID_ARG, (i, off)
        assert "aligned" in b.last_error_string()


def test_bwd_rejects_misaligned_pointers(lib):
    B, H, S, D = 1, 2, 64, 64
    names = ("q", "k", "v", "o", "do", "lse", "dq", "dk", "dv", "ws")
    for i, name in enumerate(names):
        a = list(P)
        a[i] += 2 if name == "lse" else 8
        assert b.raw_bwd(*a, B, H, S, D, 0.125, 1, 1) == b.CATTN_ERR_INVALID_ARG, name
        assert "aligned" in b.last_error_string(), name


def test_scale_range_boundaries_accepted(lib):
    """The ends of the supported scale range pass the argument checks (the call
    then fails only on its NULL pointers)."""
    for scale in (1e-20, 1e6):
        assert b.raw_fwd(0, 0, 0, 0, 0, 1, 1, 16, 64, scale, 1, 1) == b.CATTN_ERR_INVALID_ARG
        assert "NULL" in b.last_error_string()


def test_noalloc_rejects_shapes_beyond_its_static_scratch(lib):
    """8 MiB of static workspace holds 2 * B * H * Sp floats up to 2^21; larger
    shapes are refused on the host before any HIP call."""
    vp = ctypes.c_void_p
    args = [vp(p) for p in P[:9]]
    st = lib.cattn_attn_bwd_noalloc(*args, 16, 32, 4096, 64, ctypes.c_float(0.125), 1, 1, 0, vp(0))
    assert st == b.CATTN_ERR_UNSUPPORTED
    assert "static scratch" in b.last_error_string()
    assert b.workspace_bytes(16, 32, 4096, 64) > 8 << 20 >= b.workspace_bytes(16, 32, 2048, 64)
