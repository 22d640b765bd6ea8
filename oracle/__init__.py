"""fp64 CPU oracle for fused scaled-dot-product attention (forward, backward,
paged prefill and decode) and for the BF16 GEMM C = A B^T.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports, calls or links
this package: only the test suite, the smoke check and the CPU-baseline leg of
the benchmark may use it.  It shares no code with the HIP library.

The oracle is the plain definition of attention (whole-row two-pass softmax in
fp64), not the tiled online-softmax method the GPU runs.  Every function is
pinned by the CPU tests in ``tests/test_oracle.py``,
``tests/test_oracle_paged.py`` and ``tests/test_oracle_gemm.py`` against closed forms,
invariants, finite differences, a pure-Python brute force and torch's own fp64
SDPA; no function is left "parity unpinned".
"""
from .attention import (
    attention_forward,
    attention_backward,
    attention_probs,
)
from .paged import attention_forward_paged
from .gemm import gemm_nt, abs_products

__all__ = ["attention_forward", "attention_backward", "attention_probs",
           "attention_forward_paged", "gemm_nt", "abs_products"]
