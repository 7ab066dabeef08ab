"""LoRA weight-update merge in float64 -- test infrastructure only.

The paper's workflows apply weight-update adapters (LoRA) that modify the
base model's weights before inference (Sec. 2.2, adapters; Sec. 3).  The merge
of one linear layer is ``W' = W + alpha * B A`` with ``A [rank, in]`` and
``B [out, rank]``.
"""
from __future__ import annotations

import numpy as np

F64 = np.float64


def merge(W, A, B, alpha):
    """``W + alpha * (B @ A)`` in float64."""
    W = np.asarray(W, dtype=F64)
    A = np.asarray(A, dtype=F64)
    B = np.asarray(B, dtype=F64)
    return W + float(alpha) * (B @ A)
