"""CPU oracle for the block-quantised prefill GEMM and prefill attention (test infrastructure only).

Only the tests, the smoke check and the bench's CPU-baseline leg may import
this package. The GPU library never calls it, and it shares no code with the
GPU library.
"""
from .qgemm_oracle import *  # noqa: F401,F403
from .qgemm_oracle import __all__ as _qgemm_all
from .attention_oracle import *  # noqa: F401,F403
from .attention_oracle import __all__ as _attn_all

__all__ = list(_qgemm_all) + list(_attn_all)
