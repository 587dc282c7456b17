"""Pins for the oracle's budget mapping (Algorithm 1, allocation half; Section 4.4).

Hand-derived exact cases from Eqs. sensitivity-normalization .. layer-budget, and
the properties Section 4.4 states: constant profile -> uniform, invariance to
positive affine maps of s, max/min multiplier = r before clipping, monotonicity,
mean(w) = 1, and the global budget sum (Eq. global-budget).
"""
import math
import random

import pytest

from oracle import budgets as BG


def test_exact_example_r4():
    # s_hat = (0, 1/2, 1) -> w~ = (1, 2, 4) -> w = (3/7, 6/7, 12/7) -> b = 70/3 * w
    w, b = BG.layer_budgets([0.0, 0.5, 1.0], 70, 4.0)
    assert w == pytest.approx([3 / 7, 6 / 7, 12 / 7], rel=1e-15)
    assert b == [10, 20, 40]


def test_exact_example_clip():
    # w~ = (1, 2, 4) clipped to [1/2, 2] -> (1, 2, 2) -> w = (0.6, 1.2, 1.2); B/3 = 25
    w, b = BG.layer_budgets([0.0, 0.5, 1.0], 75, 4.0, gamma=2.0)
    assert w == pytest.approx([0.6, 1.2, 1.2], rel=1e-15)
    assert b == [15, 30, 30]


def test_exact_example_two_layers():
    w, b = BG.layer_budgets([0.0, 1.0], 300, 2.0)
    assert w == pytest.approx([2 / 3, 4 / 3], rel=1e-15)
    assert b == [100, 200]


def test_constant_profile_is_uniform():
    w, b = BG.layer_budgets([0.3] * 8, 800, 4.0)
    assert w == [1.0] * 8
    assert b == [100] * 8
    # remainder units go to the lowest indices when s ties
    w, b = BG.layer_budgets([0.3] * 4, 205, 4.0)
    assert b == [52, 51, 51, 51]


def test_r_one_is_uniform():
    s = [0.1, 0.7, 0.2, 0.9, 0.4]
    w, b = BG.layer_budgets(s, 1003, 1.0)
    assert w == pytest.approx([1.0] * 5, abs=0)
    assert sum(b) == 1003 and max(b) - min(b) <= 1
    # the leftover units go to the more sensitive layers first
    assert b[3] == 201 and b[1] == 201 and b[0] == 200


def test_nearest_even_is_literal_rounding():
    w, b = BG.layer_budgets([0.0, 1.0], 3, 1.0, rounding="nearest_even")
    assert b == [2, 2]      # 1.5 -> 2 twice: the literal rule overshoots B = 3


@pytest.mark.parametrize("seed", range(20))
def test_properties_random(seed):
    rng = random.Random(seed)
    n = rng.randint(1, 40)
    s = [rng.random() * 10 ** rng.uniform(-6, 0) for _ in range(n)]
    r = rng.choice([1.0, 1.25, 1.5, 2.0, 4.0, 8.0])
    B = rng.randint(0, 10 ** 6)
    w, b = BG.layer_budgets(s, B, r)
    assert sum(b) == B
    assert all(x >= 0 for x in b)
    assert sum(w) / n == pytest.approx(1.0, rel=1e-12)
    # before clipping the extreme multipliers differ by exactly r
    wt = BG.exp_map(BG.normalize(s), r)
    if max(s) != min(s):
        assert max(wt) / min(wt) == pytest.approx(r, rel=1e-12)
    # monotone: larger s never gets a smaller multiplier
    order = sorted(range(n), key=lambda i: s[i])
    for a_, b_ in zip(order, order[1:]):
        assert w[a_] <= w[b_] + 1e-15
    # affine invariance of the normalised profile
    s2 = [3.5 * x + 7.0 for x in s]
    w2, _ = BG.layer_budgets(s2, B, r)
    assert w2 == pytest.approx(w, rel=1e-9)
    # each budget is within one unit of the real-valued share
    for x, bi in zip(w, b):
        assert abs(bi - B * x / n) < 1.0 + 1e-9


@pytest.mark.parametrize("bad", [dict(r=0.5), dict(gamma=0.5), dict(B=-1), dict(s=[]), dict(s=[1.0, math.nan])])
def test_rejects_invalid(bad):
    args = dict(s=[0.1, 0.2], B=10, r=2.0, gamma=None)
    args.update(bad)
    with pytest.raises(ValueError):
        BG.layer_budgets(args["s"], args["B"], args["r"], args["gamma"])
