"""Load/compute pipeline of first-layers caching -- test infrastructure only.

Sec. 5.1 ("Caching the first layers"): a model of L layers keeps its first
L_e layers in GPU memory and the rest in host memory.  When a request
arrives (t = 0) inference starts on the resident layers while the other
layers are copied from host memory one after another, in layer order; layer
i runs once layer i-1 has finished and, for i >= L_e, once its copy has
finished.  T_load is one layer's copy time, T_comp one layer's inference
time.

* ``e2e_uniform``    Eq. 1, end-to-end latency of L uniform layers;
* ``prefix_uniform`` Eq. 2, the smallest prefix that hides loading;
* ``timeline``       the same pipeline stepped layer by layer for arbitrary
                     per-layer times (the paper notes the equations extend to
                     non-uniform layers; this is that extension);
* ``serial``         loading and inference one after the other (the "w/o
                     ppl." bound of the loading breakdown, Sec. 8.3).

Readings: Eq. 1 is exact under the paper's premise T_load >= T_comp; with
T_load < T_comp and L_e = 0 the first layer's copy precedes all compute and
the timeline gives T_load + L T_comp where Eq. 1 gives L T_comp.  Eq. 2's
value is clamped to [0, L].  All functions accept fractions.Fraction for
exact arithmetic.
"""
from __future__ import annotations

import math
from typing import Sequence


def e2e_uniform(L, Le, t_load, t_comp):
    """Eq. 1: max(L T_comp, (L - L_e) T_load + T_comp)."""
    return max(L * t_comp, (L - Le) * t_load + t_comp)


def prefix_uniform(L, t_load, t_comp) -> int:
    """Eq. 2: ceil((L (T_load - T_comp) + T_comp) / T_load), within [0, L]."""
    v = math.ceil((L * (t_load - t_comp) + t_comp) / t_load)
    return min(max(v, 0), L)


def timeline(load: Sequence, comp: Sequence, Le: int):
    """Finish time of the last layer: copies of layers Le.. back to back from
    t = 0, each layer starting after its predecessor and its own copy."""
    L = len(comp)
    assert len(load) == L and 0 <= Le <= L
    copied = 0
    finish = 0
    for i in range(L):
        ready = 0
        if i >= Le:
            copied = copied + load[i]
            ready = copied
        finish = max(finish, ready) + comp[i]
    return finish


def serial(load: Sequence, comp: Sequence, Le: int):
    """Every missing layer copied first, then the whole inference."""
    return sum(load[Le:], 0) + sum(comp, 0)
