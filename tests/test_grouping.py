"""Cross-task expert grouping (Sec. 3.2.1): the oracle pinned to brute force,
textbook knapsack optima, a hand-worked example and closed forms; the
library's host routine against the oracle."""
import itertools
import json
import math
import os
import random

import pytest

from oracle import grouping as OG

HERE = os.path.dirname(os.path.abspath(__file__))
MB = 1 << 20


def _brute_force(weights, values, capacity):
    best = 0.0
    for r in range(len(weights) + 1):
        for sub in itertools.combinations(range(len(weights)), r):
            if sum(weights[i] for i in sub) <= capacity:
                best = max(best, sum(values[i] for i in sub))
    return best


def test_knapsack_matches_brute_force():
    rng = random.Random(1)
    for _ in range(300):
        n = rng.randint(0, 9)
        w = [rng.randint(0, 12) for _ in range(n)]
        v = [rng.uniform(-1.0, 2.0) for _ in range(n)]
        cap = rng.randint(0, 30)
        chosen, opt = OG.knapsack(w, v, cap)
        assert sum(w[i] for i in chosen) <= cap
        assert math.isclose(sum(v[i] for i in chosen), opt, rel_tol=0, abs_tol=1e-12)
        assert math.isclose(opt, _brute_force(w, v, cap), rel_tol=0, abs_tol=1e-12)


def test_knapsack_textbook_instances():
    assert OG.knapsack([10, 20, 30], [60.0, 100.0, 120.0], 50) == ([1, 2], 220.0)
    assert OG.knapsack([1, 3, 4, 5], [1.0, 4.0, 5.0, 7.0], 7) == ([1, 2], 9.0)
    assert OG.knapsack([], [], 5) == ([], 0.0)
    assert OG.knapsack([3], [-1.0], 5) == ([], 0.0)   # a loss is never taken


def _hand():
    with open(os.path.join(HERE, "golden", "grouping_hand_example.json")) as f:
        return json.load(f)


def test_hand_worked_example():
    h = _hand()
    mt = [u * h["unit_bytes"] for u in h["mtmp_units"]]
    got = OG.group_experts(mt, h["lifespan"], h["mem_budget"], h["mem_static"], h["eta"],
                           h["unit_bytes"])
    assert got == (h["slice_of"], h["n_slices"])
    fb = h["fallback_case"]
    mt = [u * h["unit_bytes"] for u in fb["mtmp_units"]]
    got = OG.group_experts(mt, fb["lifespan"], h["mem_budget"], h["mem_static"], fb["eta"],
                           h["unit_bytes"])
    assert got == (fb["slice_of"], fb["n_slices"])


def test_everything_fits_one_slice():
    mt = [1.5 * MB, 2 * MB, 0.25 * MB]
    assert OG.group_experts(mt, [1, 2, 3], 64 * MB, 8 * MB, 0.0, MB) == ([0, 0, 0], 1)


def test_equal_experts_fill_slices_in_order():
    # eight equal experts, room for three: slices of three, first experts first
    so, ns = OG.group_experts([4 * MB] * 8, [1.0] * 8, 14 * MB, 2 * MB, 0.0, MB)
    assert ns == 3 and so == [0, 0, 0, 1, 1, 1, 2, 2]


def test_expert_over_budget_is_an_error():
    with pytest.raises(ValueError):
        OG.group_experts([5 * MB, 11 * MB], [1, 1], 12 * MB, 2 * MB, 0.0, MB)
    with pytest.raises(ValueError):
        OG.group_experts([MB], [1], 2 * MB, 2 * MB, 0.0, MB)


def _random_instance(rng, n):
    mt = [rng.randint(0, 40) * MB + rng.randint(0, MB - 1) for _ in range(n)]
    life = [rng.choice([0.5, 1.0, 2.0, 3.0]) * rng.randint(1, 5) for _ in range(n)]
    return mt, life


def test_grouping_invariants():
    rng = random.Random(2)
    for _ in range(100):
        n = rng.randint(1, 24)
        mt, life = _random_instance(rng, n)
        budget, static = rng.randint(60, 120) * MB, rng.randint(0, 10) * MB
        eta = rng.choice([0.0, 0.001, 0.01, 0.1])
        so, ns = OG.group_experts(mt, life, budget, static, eta, MB)
        W = (budget - static) // MB
        w = [math.ceil(m / MB) for m in mt]
        assert sorted(set(so)) == list(range(ns))          # slices 0..ns-1, none empty
        for s in range(ns):
            assert sum(w[i] for i in range(n) if so[i] == s) <= W
        assert ns >= math.ceil(sum(w) / W) if sum(w) else ns >= 1


def test_first_slice_is_the_knapsack_optimum():
    rng = random.Random(3)
    for _ in range(100):
        n = rng.randint(1, 9)
        mt, life = _random_instance(rng, n)
        budget, static, eta = 50 * MB, 5 * MB, rng.choice([0.0, 0.01])
        so, _ = OG.group_experts(mt, life, budget, static, eta, MB)
        w = [math.ceil(m / MB) for m in mt]
        v = [mt[i] / budget - eta * life[i] for i in range(n)]
        first = [i for i in range(n) if so[i] == 0]
        opt = _brute_force(w, v, 45)
        if opt > 0:
            assert math.isclose(sum(v[i] for i in first), opt, abs_tol=1e-12)


def test_mtmp_estimator_scaling():
    # m_c is linear in T with theta2 = 0, quadratic with theta1 = 0; T = 0 leaves m_f
    lin = [OG.expert_mtmp(t, 64, 2.0, 3.0, 0.0, 1000.0) - 1000.0 for t in (100, 200)]
    assert lin[1] == 2 * lin[0]
    quad = [OG.expert_mtmp(t, 64, 2.0, 0.0, 1.0, 1000.0) - 1000.0 for t in (100, 200)]
    assert quad[1] == 4 * quad[0]
    assert OG.expert_mtmp(0, 64, 4.0, 3.0, 1.0, 777.0) == 777.0
    # bytes scale with the element width B_p
    assert OG.expert_mtmp(50, 64, 4.0, 3.0, 1.0, 0.0) == 2 * OG.expert_mtmp(50, 64, 2.0, 3.0,
                                                                            1.0, 0.0)


# ------------------------------------------- the library's host routine

def _lib():
    from paper_2608_16188_amd import vmoe as V
    return V


def test_library_matches_oracle():
    V = _lib()
    rng = random.Random(4)
    for trial in range(300):
        n = rng.randint(0, 40)
        mt, life = _random_instance(rng, n)
        unit = rng.choice([MB, MB // 4, 3 * MB])
        budget, static = rng.randint(60, 200) * MB, rng.randint(0, 20) * MB
        eta = rng.choice([0.0, 1e-3, 1e-2, 0.05, 1.0])
        try:
            ref = OG.group_experts(mt, life, budget, static, eta, unit)
        except ValueError:
            with pytest.raises(V.VmoeError):
                V.vmoe_group_experts(mt, life, budget, static, eta, unit)
            continue
        so, ns = V.vmoe_group_experts(mt, life, budget, static, eta, unit)
        assert (list(so), ns) == ref, f"trial {trial}"


def test_library_hand_worked_example():
    V = _lib()
    h = _hand()
    mt = [u * h["unit_bytes"] for u in h["mtmp_units"]]
    so, ns = V.vmoe_group_experts(mt, h["lifespan"], h["mem_budget"], h["mem_static"], h["eta"],
                                  h["unit_bytes"])
    assert (list(so), ns) == (h["slice_of"], h["n_slices"])
    fb = h["fallback_case"]
    mt = [u * h["unit_bytes"] for u in fb["mtmp_units"]]
    so, ns = V.vmoe_group_experts(mt, fb["lifespan"], h["mem_budget"], h["mem_static"], fb["eta"],
                                  h["unit_bytes"])
    assert (list(so), ns) == (fb["slice_of"], fb["n_slices"])


def test_library_errors():
    import ctypes
    import numpy as np
    V = _lib()
    with pytest.raises(V.VmoeError):          # an expert alone over the budget
        V.vmoe_group_experts([5 * MB, 11 * MB], [1, 1], 12 * MB, 2 * MB, 0.0, MB)
    with pytest.raises(V.VmoeError):          # no room
        V.vmoe_group_experts([MB], [1], 2 * MB, 2 * MB, 0.0, MB)
    with pytest.raises(V.VmoeError):          # negative lifespan
        V.vmoe_group_experts([MB], [-1.0], 8 * MB, 0, 0.0, MB)
    need = V._lib.vmoe_group_experts_workspace_bytes(2, 8.0 * MB, 0.0, float(MB))
    assert need > 0
    m = np.array([MB, MB], np.float64)
    ws = np.empty(need, np.uint8)
    out = np.empty(2, np.int32)
    ns = ctypes.c_int32(0)
    assert V._lib.vmoe_group_experts(2, m.ctypes.data, m.ctypes.data, 8.0 * MB, 0.0, 0.0,
                                     float(MB), out.ctypes.data, ctypes.addressof(ns),
                                     ws.ctypes.data, need - 1) == V.VMOE_ERR_WORKSPACE
    assert V._lib.vmoe_group_experts_workspace_bytes(2, 1.0, 2.0, 1.0) == 0


def test_library_mtmp_matches_oracle():
    V = _lib()
    rng = random.Random(5)
    for _ in range(200):
        args = (rng.randint(0, 100000), rng.choice([32, 64, 768, 1024]), rng.choice([1.0, 2.0, 4.0]),
                rng.uniform(0, 8), rng.uniform(0, 2), rng.uniform(0, 1e7))
        assert V.vmoe_expert_mtmp(*args) == OG.expert_mtmp(*args)
