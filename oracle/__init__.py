"""fp64 CPU oracle for response-replay attention (test infrastructure only).

Imported by the tests, the smoke check and the benchmark's CPU-baseline leg;
never by the library or its binding.
"""
from .attention import (attn_bwd, attn_fwd, bf16_round, cyclic_owned_positions,  # noqa: F401
                        decode, dsa_index_scores, gather, lse_merge, lse_merge_bf16_numerator,
                        sparse_bwd, sparse_fwd, topk_select)
