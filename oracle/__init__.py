"""fp64 CPU oracle of the MoE layer (test infrastructure only; see moe_oracle and,
for the MXFP8 expert GEMMs, mxfp8)."""
from .moe_oracle import (route, permute, swiglu_ffn, ffn_rows, combine, layer,  # noqa: F401
                         dense_swiglu, token_outputs, router_logits, router_topk)
