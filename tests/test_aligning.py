"""Fill-clamp-refill allocation (paper Sec. 3.2.2): the oracle against the
water-filling form it must reach and closed forms; the host routine of the
library against the oracle."""
import random

import numpy as np
import pytest

from oracle import aligning as A
from paper_2608_16188_amd import vmoe as V


def _water_fill(m, s, w, budget):
    """min(s_i, m_i + lam w_i) with sum = min(budget, sum of the caps), lam by bisection."""
    caps = [s[i] if w[i] > 0 else m[i] for i in range(len(m))]
    target = min(budget, sum(caps))
    f = lambda lam: sum(min(caps[i], m[i] + lam * w[i]) for i in range(len(m)))
    lo, hi = 0.0, 1.0
    while f(hi) < target - 1e-12 and hi < 1e30:
        hi *= 2
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        lo, hi = (mid, hi) if f(mid) < target else (lo, mid)
    return [min(caps[i], m[i] + hi * w[i]) for i in range(len(m))]


def _instance(rng, n):
    m = [rng.randint(0, 4) for _ in range(n)]
    s = [m[i] + rng.randint(0, 40) for i in range(n)]
    w = [rng.choice([0.0, rng.uniform(0.1, 10.0), rng.uniform(0.1, 10.0)]) for _ in range(n)]
    budget = sum(m) + rng.randint(0, 3 * sum(s) // 2 + 1)
    return m, s, w, budget


def test_reaches_the_water_filling_shares():
    rng = random.Random(0)
    for _ in range(200):
        m, s, w, budget = _instance(rng, rng.randint(1, 12))
        a, rounds = A.fill_clamp_refill(m, s, w, budget)
        np.testing.assert_allclose(a, _water_fill(m, s, w, budget), rtol=1e-9, atol=1e-7)
        assert rounds <= len(m)


def test_closed_forms():
    # nothing saturates: minima plus shares proportional to the coefficients
    a, rounds = A.fill_clamp_refill([1, 2, 0], [100, 100, 100], [1.0, 3.0, 4.0], 19)
    np.testing.assert_allclose(a, [1 + 2, 2 + 6, 0 + 8])
    assert rounds == 1
    # a heavy expert saturates; its excess goes to the others 1:1
    a, rounds = A.fill_clamp_refill([0, 0, 0], [2, 50, 50], [8.0, 1.0, 1.0], 20)
    np.testing.assert_allclose(a, [2, 9, 9])
    assert rounds == 2
    # budget beyond every saturation stays unused
    a, _ = A.fill_clamp_refill([1, 1], [3, 4], [1.0, 1.0], 100)
    assert a == [3.0, 4.0]
    # zero coefficient keeps its minimum; equal experts split evenly
    a, _ = A.fill_clamp_refill([2, 0, 0], [9, 9, 9], [0.0, 1.0, 1.0], 10)
    assert a == [2.0, 4.0, 4.0]


def test_rounding_to_whole_units():
    assert A.round_units([1.5, 1.5, 1.0]) == [2, 1, 1]          # ties: lower index
    assert A.round_units([0.2, 0.7, 2.1]) == [0, 1, 2]          # floor(3.0) = 3 units
    assert A.round_units([3.0, 4.0]) == [3, 4]


def test_errors():
    with pytest.raises(ValueError):
        A.fill_clamp_refill([3, 3], [5, 5], [1.0, 1.0], 5)     # minima exceed the budget
    with pytest.raises(ValueError):
        A.fill_clamp_refill([3], [2], [1.0], 5)                # saturation below minimum
    with pytest.raises(V.VmoeError):
        V.vmoe_fill_clamp_refill([3, 3], [5, 5], [1.0, 1.0], 5)
    with pytest.raises(V.VmoeError):
        V.vmoe_fill_clamp_refill([3], [2], [1.0], 5)
    with pytest.raises(V.VmoeError):
        V.vmoe_fill_clamp_refill([0], [2], [-1.0], 5)


def test_library_matches_oracle():
    rng = random.Random(1)
    for _ in range(300):
        m, s, w, budget = _instance(rng, rng.randint(0, 16))
        a, rounds = A.fill_clamp_refill(m, s, w, budget)
        got, units, got_rounds = V.vmoe_fill_clamp_refill(m, s, w, budget)
        np.testing.assert_allclose(got, a, rtol=1e-12, atol=1e-12)
        assert got_rounds == rounds
        assert list(units) == A.round_units(a)
        assert all(units[i] <= s[i] for i in range(len(m)))
