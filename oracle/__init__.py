"""fp64 CPU oracle for response-replay attention (test infrastructure only).

Imported by the tests, the smoke check and the benchmark's CPU-baseline leg;
never by the library or its binding.
"""
from .attention import (attn_bwd, attn_fwd, decode, gather, lse_merge,  # noqa: F401
                        sparse_bwd, sparse_fwd)
