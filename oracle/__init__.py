"""CPU oracle for Sparse Feature Attention -- test infrastructure only.

Only `tests/`, `__graft_entry__.smoke()` and `bench.py`'s `cpu_baseline` leg
may import this package.  It shares no code with the HIP library.
"""
from .sfa_oracle import (  # noqa: F401
    widen, topk_select, topk_encode, bf16_rne, topk_encode_bf16, densify,
    softmax_attention, attn_fwd, attn_fwd_rows, attn_decode, overlap_count,
    csr_bytes, softmax_attention_grad, attn_bwd, attn_bwd_rows, attn_bwd_cols,
    cache_location, cache_capacity, kv_append, cache_gather, attn_decode_paged,
    f16_rne, widen_f16, topk_encode_f16, csr_densify, csr_to_fixed, token_mask,
    quant_q8, dequant_q8, kv_append_q8, stored_output,
)
