"""Oracle of the cross-task expert grouping (TEST INFRASTRUCTURE ONLY).

Plain Python, written from the paper's Sec. 3.2.1 (fragmentation-aware expert
grouping): a per-expert temporary-DRAM estimate, then experts are cut into
ordered time slices, each slice the 0/1 knapsack optimum over the experts not
yet placed, with every expert's footprint as its weight and
  v_i = M_tmp(i) / M_c - eta * r_i
as its value, under the budget M_c - M_s. Where the paper leaves the
procedure open, the readings below fix it (they are listed with the design
notes too):

  * weights are whole multiples of `unit` bytes: w_i = ceil(M_tmp(i) / unit),
    capacity W = floor((M_c - M_s) / unit);
  * the table runs over the remaining experts in increasing index, and a
    candidate replaces the current best only when strictly larger (ties keep
    the choice without the expert); the set is read back from capacity W;
  * if a slice would be empty (no remaining expert has a positive value
    that fits), the remaining expert with the shortest lifespan (ties: lower
    index) forms the slice alone, so every expert is placed;
  * an expert whose weight alone exceeds W cannot be placed: an error.

Shares no code with the library; only tests import it.
"""
from __future__ import annotations

import math


def expert_mtmp(tokens: int, d_k: int, bytes_per_elem: float, theta1: float, theta2: float,
                m_f: float) -> float:
    """Temporary DRAM of one expert (Sec. 3.2.1): M_tmp = m_c + m_f with the
    compute-dependent part m_c = B_p (theta1 T d_k + theta2 T^2), T tokens."""
    T = float(tokens)
    m_c = bytes_per_elem * (theta1 * T * d_k + theta2 * T * T)
    return m_c + m_f


def knapsack(weights, values, capacity):
    """0/1 knapsack by the recurrence dp[i][j] = max(dp[i-1][j],
    dp[i-1][j - w_i] + v_i), full table, items in the given order; returns the
    chosen item positions (ascending) and the optimum dp[n][capacity]."""
    n = len(weights)
    dp = [[0.0] * (capacity + 1) for _ in range(n + 1)]
    take = [[False] * (capacity + 1) for _ in range(n + 1)]
    for i in range(1, n + 1):
        w, v = weights[i - 1], values[i - 1]
        for j in range(capacity + 1):
            best = dp[i - 1][j]
            if j >= w and dp[i - 1][j - w] + v > best:
                best = dp[i - 1][j - w] + v
                take[i][j] = True
            dp[i][j] = best
    chosen = []
    j = capacity
    for i in range(n, 0, -1):
        if take[i][j]:
            chosen.append(i - 1)
            j -= weights[i - 1]
    return sorted(chosen), dp[n][capacity]


def group_experts(mtmp, lifespan, mem_budget, mem_static, eta, unit):
    """Ordered time slices of the experts: returns slice_of (one slice index
    per expert) and the number of slices. Raises ValueError on an expert that
    cannot fit or on a budget that leaves no room."""
    n = len(mtmp)
    if mem_budget <= mem_static or unit <= 0:
        raise ValueError("no room under the budget")
    W = int(math.floor((mem_budget - mem_static) / unit))
    w = [int(math.ceil(m / unit)) for m in mtmp]
    if any(x > W for x in w):
        raise ValueError("an expert alone exceeds the budget")
    v = [mtmp[i] / mem_budget - eta * lifespan[i] for i in range(n)]
    slice_of = [-1] * n
    remaining = list(range(n))
    s = 0
    while remaining:
        pos, _ = knapsack([w[i] for i in remaining], [v[i] for i in remaining], W)
        chosen = [remaining[p] for p in pos]
        if not chosen:
            chosen = [min(remaining, key=lambda i: (lifespan[i], i))]
        for i in chosen:
            slice_of[i] = s
        remaining = [i for i in remaining if slice_of[i] < 0]
        s += 1
    return slice_of, s
