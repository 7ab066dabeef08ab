"""Pins of the first-layers caching model (Sec. 5.1, Eq. 1-2), CPU only.

* hand-stepped pipelines (copies back to back, layers in order) worked out
  on paper in the comments below;
* Eq. 2 equals the brute-force smallest prefix whose Eq. 1 latency is
  L T_comp, and is the smallest prefix for which the stepped timeline hides
  loading (exact rationals);
* the stepped timeline equals a different derivation -- the max over the
  last layer j that waited for its copy, of (copies up to j) + (compute from
  j on) -- on random non-uniform layers, and equals Eq. 1 for uniform layers
  whenever T_load >= T_comp;
* limits: all layers resident gives L T_comp; serial loading bounds the
  pipeline from above."""
import itertools
from fractions import Fraction as Fr

import numpy as np
import pytest

from oracle import loading


def test_hand_stepped_pipeline():
    # L = 4, T_load = 3, T_comp = 1.
    # L_e = 0: copies end at 3, 6, 9, 12; layers run 3-4, 6-7, 9-10, 12-13 -> 13
    # L_e = 2: copies of layers 2, 3 end at 3, 6; layers 0-1, 1-2, 3-4, 6-7 -> 7
    # L_e = 3: copy of layer 3 ends at 3; layers 0-1, 1-2, 2-3, 3-4 -> 4
    load, comp = [3] * 4, [1] * 4
    assert [loading.timeline(load, comp, le) for le in (0, 1, 2, 3, 4)] == [13, 10, 7, 4, 4]
    assert [loading.e2e_uniform(4, le, 3, 1) for le in (0, 1, 2, 3, 4)] == [13, 10, 7, 4, 4]
    # Eq. 2: ceil((4 * 2 + 1) / 3) = 3
    assert loading.prefix_uniform(4, 3, 1) == 3
    assert loading.serial(load, comp, 0) == 16 and loading.serial(load, comp, 3) == 7


def test_hand_stepped_non_uniform():
    # layers cost (copy, compute) = (2, 1), (5, 2), (1, 3), (4, 1), L_e = 1:
    # copies of layers 1, 2, 3 end at 5, 6, 10; layer 0 0-1, layer 1 5-7,
    # layer 2 7-10, layer 3 10-11 -> 11
    assert loading.timeline([2, 5, 1, 4], [1, 2, 3, 1], 1) == 11
    # L_e = 0: copies end at 2, 7, 8, 12: 2-3, 7-9, 9-12, 12-13 -> 13
    assert loading.timeline([2, 5, 1, 4], [1, 2, 3, 1], 0) == 13


def _closed_form(load, comp, Le):
    L = len(comp)
    best = sum(comp) if Le > 0 else 0
    for j in range(Le, L):
        best = max(best, sum(load[Le:j + 1]) + sum(comp[j:]))
    return best


@pytest.mark.parametrize("seed", range(20))
def test_timeline_equals_max_plus_closed_form(seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(1, 12))
    load = [Fr(int(v), 7) for v in rng.integers(0, 40, L)]
    comp = [Fr(int(v), 5) for v in rng.integers(1, 40, L)]
    for Le in range(L + 1):
        assert loading.timeline(load, comp, Le) == _closed_form(load, comp, Le)
        assert loading.timeline(load, comp, Le) <= loading.serial(load, comp, Le)


@pytest.mark.parametrize("L", [1, 2, 5, 28, 57])
def test_eq1_is_the_uniform_timeline_and_eq2_its_smallest_hiding_prefix(L):
    for tl, tc in itertools.product([Fr(1), Fr(3, 2), Fr(7, 3), Fr(10), Fr(61, 60)],
                                    [Fr(1), Fr(1, 3), Fr(2, 7)]):
        if tl < tc:
            continue
        e2e = [loading.timeline([tl] * L, [tc] * L, le) for le in range(L + 1)]
        assert e2e == [loading.e2e_uniform(L, le, tl, tc) for le in range(L + 1)]
        hiding = [le for le in range(L + 1) if e2e[le] == L * tc]
        assert loading.prefix_uniform(L, tl, tc) == min(hiding)
        # more resident layers never hurt
        assert all(a >= b for a, b in zip(e2e, e2e[1:]))
    # the paper's premise aside: with T_load < T_comp and nothing resident the
    # first copy is exposed; Eq. 1 drops it
    assert loading.timeline([Fr(1)] * L, [Fr(2)] * L, 0) == 1 + 2 * L
    assert loading.e2e_uniform(L, 0, 1, 2) == max(2 * L, L + 2)


def test_limits():
    assert loading.timeline([5] * 6, [2] * 6, 6) == 12
    assert loading.timeline([0] * 6, [2] * 6, 0) == 12
    assert loading.prefix_uniform(6, 1, 1) == 1       # equal times: one resident layer
    assert loading.prefix_uniform(6, 100, 1) == 6     # copies far slower: all resident


def test_library_prefix_planner():
    """t2i_first_layers: Eq. 2 of the oracle when T_load >= T_comp, and the
    smallest prefix whose stepped timeline hides loading in every case."""
    import paper_2607_26566_amd as t2i
    rng = np.random.default_rng(5)
    n_eq2 = 0
    for _ in range(400):
        L = int(rng.integers(1, 60))
        tl = float(rng.uniform(0.05, 5.0))
        tc = float(rng.uniform(0.05, 2.0))
        q = (L * (Fr(tl) - Fr(tc)) + Fr(tc)) / Fr(tl)
        if abs(q - round(q)) < Fr(1, 10 ** 9):
            continue                      # a tie decided by rounding
        got = t2i.t2i_first_layers(L, tl, tc)
        e2e = [loading.timeline([Fr(tl)] * L, [Fr(tc)] * L, le) for le in range(L + 1)]
        assert got == min(le for le in range(L + 1) if e2e[le] == L * Fr(tc)), (L, tl, tc)
        if tl >= tc:
            assert got == loading.prefix_uniform(L, Fr(tl), Fr(tc))
            n_eq2 += 1
    assert n_eq2 > 100
    assert t2i.t2i_first_layers(0, 1.0, 1.0) == -1
    assert t2i.t2i_first_layers(4, float("nan"), 1.0) == -1
    assert t2i.t2i_first_layers(4, 3.0, 1.0) == 3
