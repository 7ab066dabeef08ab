"""Seeded synthetic inputs shared by the oracle and the HIP path.

This module holds only workload definitions (shapes, seeds, request mixes) and
the random-number recipe that turns them into arrays.  It contains none of the
denoising method's arithmetic: no layer, no attention, no sampler.  Both the
oracle (``oracle/``) and the product binding draw their inputs from here, so
that the two sides see bit-identical latents, text embeddings and weights.

Recipe (one independent stream per tensor):

* tensor key ``k`` of a workload seeded ``s`` uses ``numpy.random.default_rng([s, *k])``;
* values are ``standard_normal`` drawn in float32, multiplied by ``std``;
* keys: latent of request ``r`` -> ``(0, r)``, text of request ``r`` -> ``(1, r)``,
  weight tensor ``i`` of the model's weight table -> ``(2, i)``;
* std: latents and text 1.0, every weight and bias 0.02 (gates included, so
  no block starts as an identity);
* bf16 workloads round weights and text to bfloat16 with round-to-nearest-even;
  latents always stay float32;
* per-request start times of the packed multi-tenant workload are
  ``default_rng([s, 999999]).random(n_requests)``.
"""
from __future__ import annotations

import dataclasses
from typing import List, Sequence, Tuple

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "workload", "normal", "f32_to_bf16_bits",
    "bf16_bits_to_f32", "round_bf16", "latents", "texts", "weights",
    "start_times", "reduced",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and seed of one synthetic denoising workload.

    ``requests`` lists each request's latent grid as (height, width) in latent
    pixels; ``guidance`` 1.0 means no classifier-free guidance.
    """
    name: str
    arch: str                  # "cross" (cross-attention DiT) or "mmdit" (joint attention)
    dtype: str                 # "f32" or "bf16": weights, text and GEMM/attention operands
    latent_channels: int
    patch: int
    hidden: int
    heads: int
    head_dim: int
    depth: int
    mlp_hidden: int
    text_dim: int
    text_tokens: int
    requests: Tuple[Tuple[int, int], ...]
    steps: int
    seed: int
    guidance: float = 1.0
    cache_tau: float = 0.0     # <= 0 disables the step-skip cache
    random_start: bool = False  # per-request start time drawn from U[0,1)
    freq_dim: int = 256
    ln_eps: float = 1e-6
    t_scale: float = 1000.0

    @property
    def n_req(self) -> int:
        return len(self.requests)

    def tokens(self, r: int) -> int:
        h, w = self.requests[r]
        return (h // self.patch) * (w // self.patch)

    @property
    def image_tokens(self) -> int:
        return sum(self.tokens(r) for r in range(self.n_req))

    @property
    def branches(self) -> int:
        return 1 if self.guidance == 1.0 else 2

    @property
    def patch_dim(self) -> int:
        return self.patch * self.patch * self.latent_channels


WORKLOADS = {
    # 4x16x16 latent, 64 tokens, width 128, 2 heads of 64, 2 blocks, fp32.
    "tiny_f32": Workload("tiny_f32", "cross", "f32", 4, 2, 128, 2, 64, 2, 512,
                         128, 16, ((16, 16),), 4, 0),
    # 512 px image: 4x64x64 latent, 1024 tokens, PixArt-scale DiT, bf16.
    "dit512": Workload("dit512", "cross", "bf16", 4, 2, 1152, 16, 72, 28, 4608,
                       4096, 120, ((64, 64),), 20, 1),
    # 1024 px image: 4x128x128 latent, 4096 tokens, CFG (cond + uncond), bf16.
    "dit1024_cfg": Workload("dit1024_cfg", "cross", "bf16", 4, 2, 1152, 16, 72,
                            28, 4608, 4096, 120, ((128, 128),), 20, 2,
                            guidance=4.5),
    # Joint-attention model: 16x128x128 latent + 512 text tokens, width 3072.
    "mmdit1024": Workload("mmdit1024", "mmdit", "bf16", 16, 2, 3072, 24, 128,
                          19, 12288, 4096, 512, ((128, 128),), 28, 3),
    # Eight requests of mixed resolution packed into one batch, cache skip on.
    "packed8": Workload("packed8", "cross", "bf16", 4, 2, 1152, 16, 72, 28,
                        4608, 4096, 120,
                        ((32, 32),) * 3 + ((64, 64),) * 3 + ((128, 128),) * 2,
                        20, 4, cache_tau=0.1, random_start=True),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def reduced(w: Workload, **changes) -> Workload:
    """A copy of ``w`` with some fields replaced (smaller test variants)."""
    return dataclasses.replace(w, **changes)


# --------------------------------------------------------------------------
# number formats

def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); uint16 bits."""
    # finite inputs only: the sum below stays below 2^32 for every finite float
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    u = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_bf16(a: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(f32_to_bf16_bits(a))


# --------------------------------------------------------------------------
# generators

def normal(seed: int, key: Sequence[int], shape, std: float = 1.0) -> np.ndarray:
    rng = np.random.default_rng([int(seed), *[int(k) for k in key]])
    a = rng.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return a


def latents(w: Workload, seed: int | None = None) -> List[np.ndarray]:
    """Initial latent of every request, float32 ``[C, h, w]``."""
    s = w.seed if seed is None else seed
    return [normal(s, (0, r), (w.latent_channels, h, ww))
            for r, (h, ww) in enumerate(w.requests)]


def texts(w: Workload, seed: int | None = None) -> List[np.ndarray]:
    """Text embeddings of every request ``[text_tokens, text_dim]``.

    float32 values, already rounded to bfloat16 for bf16 workloads."""
    s = w.seed if seed is None else seed
    out = []
    for r in range(w.n_req):
        a = normal(s, (1, r), (w.text_tokens, w.text_dim))
        out.append(round_bf16(a) if w.dtype == "bf16" else a)
    return out


def weights(w: Workload, layout: Sequence[Tuple[str, Tuple[int, ...]]],
            seed: int | None = None, only: int | None = None,
            pick: Sequence[int] | None = None) -> List[np.ndarray]:
    """Weight tensors for a weight table given as (name, shape) pairs.

    Tensor ``i`` depends only on (seed, i, shape), so a caller may generate a
    prefix of the table (``only`` = number of leading tensors) or the tensors
    at chosen indices (``pick``, returned in that order)."""
    s = w.seed if seed is None else seed
    idx = list(pick) if pick is not None else range(len(layout) if only is None else only)
    out = []
    for i in idx:
        a = normal(s, (2, i), tuple(layout[i][1]), std=0.02)
        out.append(round_bf16(a) if w.dtype == "bf16" else a)
    return out


def start_times(w: Workload, seed: int | None = None) -> np.ndarray:
    """Start time of every request's schedule (float64)."""
    s = w.seed if seed is None else seed
    if not w.random_start:
        return np.ones(w.n_req)
    return np.random.default_rng([int(s), 999999]).random(w.n_req)
