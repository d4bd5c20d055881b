"""Thin ctypes binding over the C ABI of libcattn.so (include/cattn.h).

Argument marshalling only: tensors are checked for device, dtype, layout and
shape, outputs are allocated with torch when the caller does not pass them,
and the raw device pointers plus torch's current HIP stream are handed to the
library.  Every step of attention runs in the library's HIP kernels; if the
library is not built this module raises instead of computing anything.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcattn.so")
_lib: Optional[ctypes.CDLL] = None

CATTN_OK, CATTN_ERR_INVALID_ARG, CATTN_ERR_UNSUPPORTED, CATTN_ERR_HIP = 0, 1, 2, 3
CATTN_F32, CATTN_BF16 = 0, 1

CATTN_BHSD, CATTN_BSHD = 0, 1
_LAYOUTS = {"bhsd": CATTN_BHSD, "bshd": CATTN_BSHD}

EXPORTED = ("cattn_attn_fwd", "cattn_attn_bwd", "cattn_attn_fwd_ex", "cattn_attn_bwd_ex", "cattn_attn_bwd_dq",
            "cattn_attn_bwd_dkdv", "cattn_lmhead_fwd", "cattn_lmhead_workspace_bytes",
            "cattn_bwd_workspace_bytes", "cattn_status_string", "cattn_last_error_string",
            "cattn_layernorm_fwd", "cattn_layernorm_bwd", "cattn_layernorm_bwd_workspace_bytes", "cattn_gelu_fwd",
            "cattn_gelu_bwd", "cattn_sce_fwd", "cattn_sce_bwd", "cattn_attn_bwd_noalloc")


class CattnError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)}: {detail}")


def library_path() -> str:
    return _LIB_PATH


def lib() -> ctypes.CDLL:
    """Load libcattn.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"HIP attention library not built: {_LIB_PATH} is missing "
                               "(run __graft_entry__.build() or python -m paper_2608_00029_amd.build)")
        L = ctypes.CDLL(_LIB_PATH)
        vp, i, f = ctypes.c_void_p, ctypes.c_int, ctypes.c_float
        L.cattn_attn_fwd.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, f, i, i, vp]
        L.cattn_attn_fwd.restype = i
        L.cattn_attn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, f, i, i, vp]
        L.cattn_attn_bwd.restype = i
        L.cattn_attn_fwd_ex.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, f, i, i, i, vp]
        L.cattn_attn_fwd_ex.restype = i
        L.cattn_attn_bwd_ex.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, f, i, i, i, vp]
        L.cattn_attn_bwd_ex.restype = i
        L.cattn_attn_bwd_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, f, i, i, i, vp]
        L.cattn_attn_bwd_noalloc.restype = i
        L.cattn_attn_bwd_dq.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, f, i, i, vp]
        L.cattn_attn_bwd_dq.restype = i
        L.cattn_attn_bwd_dkdv.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, f, i, i, vp]
        L.cattn_attn_bwd_dkdv.restype = i
        L.cattn_lmhead_fwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, vp]
        L.cattn_lmhead_fwd.restype = i
        L.cattn_lmhead_workspace_bytes.argtypes = [i, i, i]
        L.cattn_lmhead_workspace_bytes.restype = ctypes.c_size_t
        L.cattn_bwd_workspace_bytes.argtypes = [i, i, i, i]
        L.cattn_bwd_workspace_bytes.restype = ctypes.c_size_t
        ll = ctypes.c_longlong
        L.cattn_layernorm_fwd.argtypes = [vp] * 6 + [i, i, f, vp]
        L.cattn_layernorm_fwd.restype = i
        L.cattn_layernorm_bwd.argtypes = [vp] * 9 + [i, i, vp]
        L.cattn_layernorm_bwd.restype = i
        L.cattn_layernorm_bwd_workspace_bytes.argtypes = [i, i]
        L.cattn_layernorm_bwd_workspace_bytes.restype = ctypes.c_size_t
        L.cattn_gelu_fwd.argtypes = [vp, vp, ll, vp]
        L.cattn_gelu_fwd.restype = i
        L.cattn_gelu_bwd.argtypes = [vp, vp, vp, ll, vp]
        L.cattn_gelu_bwd.restype = i
        L.cattn_sce_fwd.argtypes = [vp] * 5 + [i, i, vp]
        L.cattn_sce_fwd.restype = i
        L.cattn_sce_bwd.argtypes = [vp, vp, vp, f, vp, i, i, vp]
        L.cattn_sce_bwd.restype = i
        L.cattn_status_string.argtypes = [i]
        L.cattn_status_string.restype = ctypes.c_char_p
        L.cattn_last_error_string.argtypes = []
        L.cattn_last_error_string.restype = ctypes.c_char_p
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().cattn_status_string(int(status)).decode()


def last_error_string() -> str:
    return lib().cattn_last_error_string().decode()


def workspace_bytes(B: int, H: int, S: int, D: int) -> int:
    return int(lib().cattn_bwd_workspace_bytes(B, H, S, D))


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return CATTN_F32
    if t.dtype == torch.bfloat16:
        return CATTN_BF16
    raise TypeError(f"unsupported dtype {t.dtype}: use float32 or bfloat16")


def _check(name: str, t: torch.Tensor, shape, dtype, device):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if t.numel() and not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous [B, H, S, D]")


def _ptr(t: Optional[torch.Tensor]):
    return ctypes.c_void_p(t.data_ptr() if t is not None and t.numel() else 0)


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _shape(q, layout: str):
    """(B, H, S, D) of a contiguous 4-d tensor stored in `layout` ("bhsd" or "bshd")."""
    if layout not in _LAYOUTS:
        raise ValueError(f"layout must be 'bhsd' or 'bshd', not {layout!r}")
    if q.dim() != 4:
        raise ValueError(f"q must be 4-d ({layout.upper()})")
    if layout == "bhsd":
        B, H, S, D = q.shape
    else:
        B, S, H, D = q.shape
    return B, H, S, D


def attn_fwd(q, k, v, scale: float, causal: bool = True, o=None, lse=None, layout: str = "bhsd"):
    """O, LSE = attention forward of contiguous tensors on a HIP device.

    Q, K, V (and O) are [B, H, S, D] for layout "bhsd", [B, S, H, D] for
    "bshd" (read and written in place, no transposes).  LSE is float32
    [B, H, S] in natural-log units in both.  `o` / `lse` may be passed to
    write into existing buffers.  Enqueued on torch's current stream.
    """
    B, H, S, D = _shape(q, layout)
    if q.device.type != "cuda":
        raise ValueError("tensors must live on a HIP device")
    for n, t in (("q", q), ("k", k), ("v", v)):
        _check(n, t, q.shape, q.dtype, q.device)
    if o is None:
        o = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((B, H, S), dtype=torch.float32, device=q.device)
    _check("o", o, q.shape, q.dtype, q.device)
    _check("lse", lse, (B, H, S), torch.float32, q.device)
    st = lib().cattn_attn_fwd_ex(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, H, S, D, float(scale),
                                 int(bool(causal)), _dtype_code(q), _LAYOUTS[layout], _stream(q.device))
    if st != CATTN_OK:
        raise CattnError(st, "cattn_attn_fwd_ex", last_error_string())
    return o, lse


def attn_bwd(q, k, v, o, do, lse, scale: float, causal: bool = True, dq=None, dk=None, dv=None,
             workspace=None, layout: str = "bhsd"):
    """dQ, dK, dV of attention for upstream gradient `do`, given the forward's O and LSE.

    Tensors are stored as for attn_fwd with the same `layout`.  `workspace` (float32,
    >= workspace_bytes(B, H, S, D) / 4 elements) receives D = rowsum(dO * O) and
    -LSE / scale, each [B*H, S rounded up to 32] with zero padding rows.
    """
    B, H, S, D = _shape(q, layout)
    if q.device.type != "cuda":
        raise ValueError("tensors must live on a HIP device")
    for n, t in (("q", q), ("k", k), ("v", v), ("o", o), ("do", do)):
        _check(n, t, q.shape, q.dtype, q.device)
    _check("lse", lse, (B, H, S), torch.float32, q.device)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    for n, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        _check(n, t, q.shape, q.dtype, q.device)
    nws = workspace_bytes(B, H, S, D) // 4
    if workspace is None:
        workspace = torch.empty((nws,), dtype=torch.float32, device=q.device)
    _check_workspace(workspace, nws, q.device)
    st = lib().cattn_attn_bwd_ex(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(do), _ptr(lse), _ptr(dq), _ptr(dk),
                                 _ptr(dv), _ptr(workspace), B, H, S, D, float(scale), int(bool(causal)),
                                 _dtype_code(q), _LAYOUTS[layout], _stream(q.device))
    if st != CATTN_OK:
        raise CattnError(st, "cattn_attn_bwd_ex", last_error_string())
    return dq, dk, dv


def attn_bwd_noalloc(q, k, v, o, do, lse, dq, dk, dv, scale: float, causal: bool = True, layout: str = "bhsd"):
    """attn_bwd into caller-provided dq, dk, dv through cattn_attn_bwd_noalloc:
    nothing is allocated (the workspace is the library's static device array)."""
    B, H, S, D = _shape(q, layout)
    if q.device.type != "cuda":
        raise ValueError("tensors must live on a HIP device")
    for n, t in (("q", q), ("k", k), ("v", v), ("o", o), ("do", do), ("dq", dq), ("dk", dk), ("dv", dv)):
        _check(n, t, q.shape, q.dtype, q.device)
    _check("lse", lse, (B, H, S), torch.float32, q.device)
    st = lib().cattn_attn_bwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(do), _ptr(lse), _ptr(dq), _ptr(dk),
                                      _ptr(dv), B, H, S, D, float(scale), int(bool(causal)), _dtype_code(q),
                                      _LAYOUTS[layout], _stream(q.device))
    if st != CATTN_OK:
        raise CattnError(st, "cattn_attn_bwd_noalloc", last_error_string())
    return dq, dk, dv


def attn_bwd_dq(q, k, v, o, do, lse, scale: float, causal: bool = True, dq=None, workspace=None):
    """First backward phase: dQ, and D = rowsum(dO * O) into `workspace` (returned)."""
    B, H, S, D = q.shape
    for n, t in (("q", q), ("k", k), ("v", v), ("o", o), ("do", do)):
        _check(n, t, q.shape, q.dtype, q.device)
    _check("lse", lse, (B, H, S), torch.float32, q.device)
    dq = torch.empty_like(q) if dq is None else dq
    _check("dq", dq, q.shape, q.dtype, q.device)
    nws = workspace_bytes(B, H, S, D) // 4
    if workspace is None:
        workspace = torch.empty((nws,), dtype=torch.float32, device=q.device)
    _check_workspace(workspace, nws, q.device)
    st = lib().cattn_attn_bwd_dq(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(do), _ptr(lse), _ptr(dq),
                                 _ptr(workspace), B, H, S, D, float(scale), int(bool(causal)), _dtype_code(q),
                                 _stream(q.device))
    if st != CATTN_OK:
        raise CattnError(st, "cattn_attn_bwd_dq", last_error_string())
    return dq, workspace


def attn_bwd_dkdv(q, k, v, do, lse, workspace, scale: float, causal: bool = True, dk=None, dv=None):
    """Second backward phase: dK, dV, reading D from `workspace` (written by attn_bwd_dq)."""
    B, H, S, D = q.shape
    for n, t in (("q", q), ("k", k), ("v", v), ("do", do)):
        _check(n, t, q.shape, q.dtype, q.device)
    _check("lse", lse, (B, H, S), torch.float32, q.device)
    _check_workspace(workspace, workspace_bytes(B, H, S, D) // 4, q.device)
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    for n, t in (("dk", dk), ("dv", dv)):
        _check(n, t, q.shape, q.dtype, q.device)
    st = lib().cattn_attn_bwd_dkdv(_ptr(q), _ptr(k), _ptr(v), _ptr(do), _ptr(lse), _ptr(workspace), _ptr(dk),
                                   _ptr(dv), B, H, S, D, float(scale), int(bool(causal)), _dtype_code(q),
                                   _stream(q.device))
    if st != CATTN_OK:
        raise CattnError(st, "cattn_attn_bwd_dkdv", last_error_string())
    return dk, dv


def _check_workspace(ws, n, device):
    if not isinstance(ws, torch.Tensor) or ws.dtype != torch.float32 or ws.device != device \
            or not ws.is_contiguous() or ws.numel() < n:
        raise ValueError("workspace must be a contiguous float32 tensor of >= cattn_bwd_workspace_bytes / 4 "
                         "elements on q's device")


def raw_fwd(q_ptr: int, k_ptr: int, v_ptr: int, o_ptr: int, lse_ptr: int, B: int, H: int, S: int, D: int,
            scale: float, causal: int, dtype: int, stream: int = 0) -> int:
    """Direct C-ABI call with integer pointers (returns the status code)."""
    vp = ctypes.c_void_p
    return lib().cattn_attn_fwd(vp(q_ptr), vp(k_ptr), vp(v_ptr), vp(o_ptr), vp(lse_ptr), B, H, S, D,
                                float(scale), int(causal), int(dtype), vp(stream))


def raw_bwd(q_ptr, k_ptr, v_ptr, o_ptr, do_ptr, lse_ptr, dq_ptr, dk_ptr, dv_ptr, ws_ptr, B, H, S, D,
            scale: float, causal: int, dtype: int, stream: int = 0) -> int:
    vp = ctypes.c_void_p
    return lib().cattn_attn_bwd(vp(q_ptr), vp(k_ptr), vp(v_ptr), vp(o_ptr), vp(do_ptr), vp(lse_ptr),
                                vp(dq_ptr), vp(dk_ptr), vp(dv_ptr), vp(ws_ptr), B, H, S, D, float(scale),
                                int(causal), int(dtype), vp(stream))


def lmhead_workspace_bytes(M: int, N: int, K: int) -> int:
    return int(lib().cattn_lmhead_workspace_bytes(M, N, K))


def lmhead_fwd(x, w, targets=None, workspace=None):
    """Fused loss head: (logits [M, N] float32, lse [M], row_loss [M] or None, loss [1] or None).

    x: [M, K] bfloat16 hidden states; w: [N, K] bfloat16 head weight (one row per
    vocabulary entry); targets: [M] int32 ids or None.  Enqueued on torch's
    current stream; the partial statistics land in `workspace` (float32).
    """
    if x.dim() != 2 or w.dim() != 2:
        raise ValueError("x must be [M, K] and w [N, K]")
    M, K = x.shape
    N = w.shape[0]
    if x.device.type != "cuda":
        raise ValueError("tensors must live on a HIP device")
    _check("x", x, (M, K), torch.bfloat16, x.device)
    _check("w", w, (N, K), torch.bfloat16, x.device)
    if targets is not None:
        _check("targets", targets, (M,), torch.int32, x.device)
    logits = torch.empty((M, N), dtype=torch.float32, device=x.device)
    lse = torch.empty((M,), dtype=torch.float32, device=x.device)
    row_loss = torch.empty((M,), dtype=torch.float32, device=x.device) if targets is not None else None
    loss = torch.empty((1,), dtype=torch.float32, device=x.device) if targets is not None else None
    nws = lmhead_workspace_bytes(M, N, K) // 4
    if workspace is None:
        workspace = torch.empty((max(nws, 1),), dtype=torch.float32, device=x.device)
    _check_workspace(workspace, nws, x.device)
    st = lib().cattn_lmhead_fwd(_ptr(x), _ptr(w), _ptr(targets), _ptr(logits), _ptr(lse), _ptr(row_loss),
                                _ptr(loss), _ptr(workspace), M, N, K, _stream(x.device))
    if st != CATTN_OK:
        raise CattnError(st, "cattn_lmhead_fwd", last_error_string())
    return logits, lse, row_loss, loss



# ---------------------------------------------------------------------------
# Memory-bound operators (float32): LayerNorm, GELU, softmax cross entropy
# ---------------------------------------------------------------------------
def _f32_on_device(name, t, shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must live on a HIP device")
    if t.dtype != torch.float32:
        raise TypeError(f"{name} must be float32, not {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _rows_cols(x):
    if x.dim() < 1:
        raise ValueError("x needs at least one dimension")
    C = x.shape[-1]
    return (x.numel() // C if C else 0), C


def layernorm_fwd(x, gamma, beta, eps: float = 1e-5):
    """(y, mean, rstd): LayerNorm over the last axis of float32 x; mean / rstd are [rows]."""
    _f32_on_device("x", x)
    R, C = _rows_cols(x)
    _f32_on_device("gamma", gamma, (C,))
    _f32_on_device("beta", beta, (C,))
    y = torch.empty_like(x)
    mean = torch.empty((R,), dtype=torch.float32, device=x.device)
    rstd = torch.empty((R,), dtype=torch.float32, device=x.device)
    st = lib().cattn_layernorm_fwd(_ptr(x), _ptr(gamma), _ptr(beta), _ptr(y), _ptr(mean), _ptr(rstd), R, C,
                                   float(eps), _stream(x.device))
    if st != CATTN_OK:
        raise CattnError(st, "cattn_layernorm_fwd", last_error_string())
    return y, mean, rstd


def layernorm_bwd_workspace_bytes(rows: int, C: int) -> int:
    return int(lib().cattn_layernorm_bwd_workspace_bytes(rows, C))


def layernorm_bwd(x, gamma, mean, rstd, dy, workspace=None):
    """(dx, dgamma, dbeta) of LayerNorm for upstream dy, given the forward's mean and rstd."""
    _f32_on_device("x", x)
    R, C = _rows_cols(x)
    _f32_on_device("gamma", gamma, (C,))
    _f32_on_device("mean", mean, (R,))
    _f32_on_device("rstd", rstd, (R,))
    _f32_on_device("dy", dy, tuple(x.shape))
    dx = torch.empty_like(x)
    dgamma = torch.empty((C,), dtype=torch.float32, device=x.device)
    dbeta = torch.empty((C,), dtype=torch.float32, device=x.device)
    nws = layernorm_bwd_workspace_bytes(R, C) // 4
    if workspace is None:
        workspace = torch.empty((max(nws, 4),), dtype=torch.float32, device=x.device)
    _check_workspace(workspace, nws, x.device)
    st = lib().cattn_layernorm_bwd(_ptr(x), _ptr(gamma), _ptr(mean), _ptr(rstd), _ptr(dy), _ptr(dx), _ptr(dgamma),
                                   _ptr(dbeta), _ptr(workspace), R, C, _stream(x.device))
    if st != CATTN_OK:
        raise CattnError(st, "cattn_layernorm_bwd", last_error_string())
    return dx, dgamma, dbeta


def gelu_fwd(x):
    """y = GELU(x), tanh form, elementwise over a float32 tensor."""
    _f32_on_device("x", x)
    y = torch.empty_like(x)
    st = lib().cattn_gelu_fwd(_ptr(x), _ptr(y), x.numel(), _stream(x.device))
    if st != CATTN_OK:
        raise CattnError(st, "cattn_gelu_fwd", last_error_string())
    return y


def gelu_bwd(x, dy):
    """dx = dy * GELU'(x)."""
    _f32_on_device("x", x)
    _f32_on_device("dy", dy, tuple(x.shape))
    dx = torch.empty_like(x)
    st = lib().cattn_gelu_bwd(_ptr(x), _ptr(dy), _ptr(dx), x.numel(), _stream(x.device))
    if st != CATTN_OK:
        raise CattnError(st, "cattn_gelu_bwd", last_error_string())
    return dx


def _targets(targets, R, device):
    if targets is None:
        return None
    if not isinstance(targets, torch.Tensor) or targets.dtype != torch.int32 or targets.device != device \
            or tuple(targets.shape) != (R,) or not targets.is_contiguous():
        raise ValueError(f"targets must be a contiguous int32 tensor of shape ({R},) on {device}")
    return targets


def sce_fwd(logits, targets=None):
    """(lse [rows], row_loss [rows] or None, loss [1] or None) of softmax cross entropy over the last axis."""
    _f32_on_device("logits", logits)
    R, V = _rows_cols(logits)
    targets = _targets(targets, R, logits.device)
    lse = torch.empty((R,), dtype=torch.float32, device=logits.device)
    row_loss = torch.empty((R,), dtype=torch.float32, device=logits.device) if targets is not None else None
    loss = torch.empty((1,), dtype=torch.float32, device=logits.device) if targets is not None else None
    st = lib().cattn_sce_fwd(_ptr(logits), _ptr(targets), _ptr(lse), _ptr(row_loss), _ptr(loss), R, V,
                             _stream(logits.device))
    if st != CATTN_OK:
        raise CattnError(st, "cattn_sce_fwd", last_error_string())
    return lse, row_loss, loss


def sce_bwd(logits, targets, lse, scale: float):
    """dlogits = scale * (softmax(logits) - onehot(targets)), softmax recomputed from the saved lse."""
    _f32_on_device("logits", logits)
    R, V = _rows_cols(logits)
    targets = _targets(targets, R, logits.device)
    if targets is None:
        raise ValueError("sce_bwd needs targets")
    _f32_on_device("lse", lse, (R,))
    dz = torch.empty_like(logits)
    st = lib().cattn_sce_bwd(_ptr(logits), _ptr(targets), _ptr(lse), float(scale), _ptr(dz), R, V,
                             _stream(logits.device))
    if st != CATTN_OK:
        raise CattnError(st, "cattn_sce_bwd", last_error_string())
    return dz
