"""CPU float64 references for fused causal attention and the fused loss head -- test infrastructure only.

Only the tests, the smoke check and the CPU-baseline leg of the benchmark use
this package; the HIP library and its binding never import it.
"""
from .attn_oracle import (  # noqa: F401
    attn_fwd, attn_bwd, attn_bwd_given_o, attn_probabilities,
    head_forward, head_backward, masked_scores, row_logsumexp, probabilities,
)
