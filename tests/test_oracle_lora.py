"""Pins of the LoRA merge oracle (CPU)."""
import numpy as np

from oracle import lora


def test_rank_one_one_hot_changes_one_column():
    """A = e_j^T, B = b: only column j moves, by alpha * b."""
    rng = np.random.default_rng(0)
    W = rng.standard_normal((5, 7))
    A = np.zeros((1, 7))
    A[0, 3] = 1.0
    b = rng.standard_normal((5, 1))
    out = lora.merge(W, A, b, 0.75)
    expect = W.copy()
    expect[:, 3] += 0.75 * b[:, 0]
    assert np.array_equal(out, expect)


def test_two_merges_equal_one_merge_of_stacked_adapters():
    rng = np.random.default_rng(1)
    W = rng.standard_normal((6, 9))
    A1, B1 = rng.standard_normal((2, 9)), rng.standard_normal((6, 2))
    A2, B2 = rng.standard_normal((3, 9)), rng.standard_normal((6, 3))
    seq = lora.merge(lora.merge(W, A1, B1, 0.5), A2, B2, 0.5)
    once = lora.merge(W, np.vstack([A1, A2]), np.hstack([B1, B2]), 0.5)
    assert np.allclose(seq, once, rtol=1e-13, atol=1e-13)


def test_zero_alpha_or_zero_adapter_is_identity():
    rng = np.random.default_rng(2)
    W = rng.standard_normal((4, 4))
    A, B = rng.standard_normal((2, 4)), rng.standard_normal((4, 2))
    assert np.array_equal(lora.merge(W, A, B, 0.0), W)
    assert np.array_equal(lora.merge(W, A, np.zeros((4, 2)), 1.3), W)
