"""CPU reference ("oracle") for fused causal multi-head self-attention, fwd + bwd.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import this module.  The product path (the
HIP library and its Python binding) never imports, calls or links it, and this
module imports nothing from the product package.

What it computes (paper section 4.2, "Attention as a First-Class Lowering"):
the fused kernel the paper generates is an exact reformulation of plain
masked-softmax attention -- the online softmax of the forward loop reaches the
same O as softmax-then-matmul (up to rounding order), and the two backward
kernels recompute P from the saved log-sum-exp instead of storing it, which is
again exact.  So the oracle is the plain definition, written out in float64
over the full S x S score matrix of every (batch, head):

    S   = scale * Q K^T                         (scaled score contraction)
    S[i, j] = -inf  for j > i  when causal      (a query never sees a later
                                                 key; the diagonal is kept)
    LSE = log sum_j exp(S[i, j])                (natural log, saved per row)
    P   = exp(S - LSE)                          (masked entries are exactly 0)
    O   = P V                                   (probability-value contraction)

and the analytic gradients of O with respect to Q, K and V for an upstream
gradient dO:

    dV  = P^T dO
    dP  = dO V^T
    D   = rowsum(dO * O)        (equals rowsum(P * dP); the paper is silent on
                                 how D is formed -- it is the standard softmax
                                 Jacobian-vector identity)
    dS  = P * (dP - D[:, None])
    dQ  = scale * dS K
    dK  = scale * dS^T Q

Readings of the paper that this file takes:
  * LSE is exported in natural-log units.  The paper computes the softmax in
    base 2 and converts back to base e once at the end (section 4.2, "Base-2
    softmax"); the oracle works in base e throughout, which is the same value.
  * The paper masks with a finite -1e30 sentinel under fast-math; here the
    masked scores are -inf in float64, which exp() maps to exactly 0, the same
    value the sentinel underflows to.
  * Causal means key j is visible to query i iff j <= i (queries and keys
    share one sequence axis); no row is ever fully masked.

Every input is upcast exactly to float64 before any arithmetic (bf16 and fp32
values are exactly representable in float64).  Arrays are [B, H, S, D]
contiguous, the layout of the library's boundary.
"""

from __future__ import annotations

import numpy as np


def _as_f64(x) -> np.ndarray:
    """Exact upcast of a numpy array or a CPU torch tensor to float64."""
    if hasattr(x, "detach"):  # torch tensor (bf16 has no numpy dtype)
        x = x.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def masked_scores(q: np.ndarray, k: np.ndarray, scale: float, causal: bool) -> np.ndarray:
    """S = scale * Q K^T for one (batch, head), with the causal mask applied.

    Section 4.2: the score contraction carries the softmax scale, and under
    causal masking a key later than the query is excluded.  q, k: [S, D]
    float64.
    Returns [S, S] float64 with -inf above the diagonal when causal.
    """
    s = scale * (q @ k.T)
    if causal:
        n = s.shape[0]
        above = np.triu(np.ones((n, n), dtype=bool), k=1)  # j > i
        s = np.where(above, -np.inf, s)
    return s


def row_logsumexp(s: np.ndarray) -> np.ndarray:
    """LSE_i = log sum_j exp(S_ij), computed stably as m_i + log sum exp(S_ij - m_i).

    Section 4.2: the forward saves the log-sum-exp of every row for the
    backward.  Rows always hold at least one finite entry (the diagonal).
    """
    m = np.max(s, axis=1)
    return m + np.log(np.sum(np.exp(s - m[:, None]), axis=1))


def probabilities(s: np.ndarray, lse: np.ndarray) -> np.ndarray:
    """P = exp(S - LSE) -- the softmax rows recomputed from the saved LSE
    (section 4.2, "The Backward Pass").  Masked entries come out exactly 0."""
    return np.exp(s - lse[:, None])


def head_forward(q, k, v, scale, causal):
    """Forward for one (batch, head).  q, k, v: [S, D] float64.
    Returns (O [S, D], LSE [S])."""
    s = masked_scores(q, k, scale, causal)
    lse = row_logsumexp(s)
    p = probabilities(s, lse)
    return p @ v, lse


def head_backward(q, k, v, do, scale, causal):
    """Analytic gradients for one (batch, head); P recomputed from LSE as the
    paper's two backward kernels do (section 4.2).  Returns (dQ, dK, dV)."""
    s = masked_scores(q, k, scale, causal)
    lse = row_logsumexp(s)
    p = probabilities(s, lse)
    o = p @ v
    dv = p.T @ do
    dp = do @ v.T
    d = np.sum(do * o, axis=1)
    ds = p * (dp - d[:, None])
    dq = scale * (ds @ k)
    dk = scale * (ds.T @ q)
    return dq, dk, dv


def attn_fwd(q, k, v, scale: float, causal: bool = True):
    """O, LSE for [B, H, S, D] inputs (any float dtype, upcast to float64).

    Returns O [B, H, S, D] float64 and LSE [B, H, S] float64 (natural log).
    """
    q, k, v = _as_f64(q), _as_f64(k), _as_f64(v)
    b, h, n, d = q.shape
    o = np.empty((b, h, n, d))
    lse = np.empty((b, h, n))
    for bi in range(b):
        for hi in range(h):
            o[bi, hi], lse[bi, hi] = head_forward(q[bi, hi], k[bi, hi], v[bi, hi], scale, causal)
    return o, lse


def attn_bwd(q, k, v, do, scale: float, causal: bool = True):
    """dQ, dK, dV for [B, H, S, D] inputs and upstream gradient dO.

    The forward is recomputed internally (the oracle's own float64 O feeds D),
    so the result is the exact gradient of sum(dO * O) at these inputs.
    """
    q, k, v, do = _as_f64(q), _as_f64(k), _as_f64(v), _as_f64(do)
    b, h, n, d = q.shape
    dq = np.empty((b, h, n, d))
    dk = np.empty((b, h, n, d))
    dv = np.empty((b, h, n, d))
    for bi in range(b):
        for hi in range(h):
            dq[bi, hi], dk[bi, hi], dv[bi, hi] = head_backward(
                q[bi, hi], k[bi, hi], v[bi, hi], do[bi, hi], scale, causal)
    return dq, dk, dv


def attn_bwd_given_o(q, k, v, o, do, lse, scale: float, causal: bool = True):
    """Backward that takes O and LSE as given (as the library's backward does)
    instead of recomputing them: P = exp(S - LSE), D = rowsum(dO * O).

    Used to localise errors: fed the oracle's own O and LSE it equals
    attn_bwd; fed a rounded O it shows what rounding O alone costs.
    """
    q, k, v, o, do, lse = (_as_f64(x) for x in (q, k, v, o, do, lse))
    b, h, n, d = q.shape
    dq = np.empty((b, h, n, d))
    dk = np.empty((b, h, n, d))
    dv = np.empty((b, h, n, d))
    for bi in range(b):
        for hi in range(h):
            s = masked_scores(q[bi, hi], k[bi, hi], scale, causal)
            p = probabilities(s, lse[bi, hi])
            dv[bi, hi] = p.T @ do[bi, hi]
            dp = do[bi, hi] @ v[bi, hi].T
            dd = np.sum(do[bi, hi] * o[bi, hi], axis=1)
            ds = p * (dp - dd[:, None])
            dq[bi, hi] = scale * (ds @ k[bi, hi])
            dk[bi, hi] = scale * (ds.T @ q[bi, hi])
    return dq, dk, dv


def attn_probabilities(q, k, scale: float, causal: bool = True):
    """The full probability matrix P [B, H, S, S] (float64).  Test helper for
    the row-stochasticity pin; never used by the fwd/bwd functions above."""
    q, k = _as_f64(q), _as_f64(k)
    b, h, n, _ = q.shape
    out = np.empty((b, h, n, n))
    for bi in range(b):
        for hi in range(h):
            s = masked_scores(q[bi, hi], k[bi, hi], scale, causal)
            out[bi, hi] = probabilities(s, row_logsumexp(s))
    return out


def head_term_magnitudes(q, k, v, do, scale, causal):
    """Sizes of the terms each output element of one (batch, head) sums, for
    error bounds in tests (float64; q, k, v, do: [S, D]).

    Every output of section 4.2's forward and backward is a contraction whose
    terms are products of a softmax-derived factor and an input row:
    O_i = sum_j P_ij V_j, dV_j = sum_i P_ij dO_i, dQ_i = scale sum_j dS_ij K_j,
    dK_j = scale sum_i dS_ij Q_i.  A rounding of relative size u in each term
    (P or dS rounded to bf16, a float sum of n terms) moves an output element
    by at most u times the sum of its terms' absolute values, which is what
    this returns:

        m_o  = P |V|           m_dv = P^T |dO|
        g_dq = |dS| |K|        g_dk = |dS|^T |Q|

    D = rowsum(dO * O) enters every dS_ij of row i through P_ij; an error in O
    of at most t * m_o moves D_i by at most t * a_i, a_i = sum_d |dO_id| m_o_id,
    and therefore dQ and dK by at most t times

        h_dq = (a * P) |K|     h_dk = (a * P)^T |Q|     (a scales row i of P).

    Returns a dict of these arrays ([S, D] each; a: [S]).
    """
    s = masked_scores(q, k, scale, causal)
    p = probabilities(s, row_logsumexp(s))
    o = p @ v
    dp = do @ v.T
    d = np.sum(do * o, axis=1)
    ads = np.abs(p * (dp - d[:, None]))
    m_o = p @ np.abs(v)
    a = np.sum(np.abs(do) * m_o, axis=1)
    ap = a[:, None] * p
    return {"m_o": m_o, "m_dv": p.T @ np.abs(do), "g_dq": ads @ np.abs(k), "g_dk": ads.T @ np.abs(q),
            "a": a, "h_dq": ap @ np.abs(k), "h_dk": ap.T @ np.abs(q)}


def attn_term_magnitudes(q, k, v, do, scale: float, causal: bool = True):
    """head_term_magnitudes for every (batch, head) of [B, H, S, D] inputs:
    a dict of [B, H, S, D] arrays (a: [B, H, S])."""
    q, k, v, do = _as_f64(q), _as_f64(k), _as_f64(v), _as_f64(do)
    b, h, n, d = q.shape
    out = None
    for bi in range(b):
        for hi in range(h):
            m = head_term_magnitudes(q[bi, hi], k[bi, hi], v[bi, hi], do[bi, hi], scale, causal)
            if out is None:
                out = {key: np.empty((b, h) + val.shape) for key, val in m.items()}
            for key, val in m.items():
                out[key][bi, hi] = val
    return out
