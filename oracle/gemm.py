"""BF16 GEMM C = A B^T in fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring): never used by the
library itself.

What is computed (PTXBench, Appendix A, paragraph "Workloads": the fifth
primary workload computes C = A B^T in BF16 with A of 8192 x 5120, B of
7168 x 5120 and C of 8192 x 7168): both operands store the reduction index
contiguously, and

    C[m, n] = sum_k A[m, k] B[n, k].

The oracle is that definition with a library matrix product as the step.
``abs_products`` returns sum_k |A[m, k] B[n, k]|, the quantity that bounds
the rounding error of any fp32 summation order (the parity tests derive
their tolerance from it).
"""
from __future__ import annotations

import torch

from .attention import _as64


def gemm_nt(a: torch.Tensor, b: torch.Tensor) -> torch.Tensor:
    """C = A B^T for A [M, K], B [N, K] (fp64 result [M, N])."""
    if a.dim() != 2 or b.dim() != 2 or a.shape[1] != b.shape[1]:
        raise ValueError("A is [M, K] and B is [N, K]")
    return _as64(a) @ _as64(b).transpose(0, 1)


def abs_products(a: torch.Tensor, b: torch.Tensor) -> torch.Tensor:
    """sum_k |A[m, k] B[n, k]| as an fp64 [M, N] tensor."""
    return _as64(a).abs() @ _as64(b).abs().transpose(0, 1)
