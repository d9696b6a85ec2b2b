"""Oracle of the expert lifespan-aligning allocation (TEST INFRASTRUCTURE ONLY).

Plain Python, written from the paper's Sec. 3.2.2 (expert lifespan-aware
aligning): within a time slice each expert receives a share of the GPU's
compute units by the fill-clamp-refill procedure, in the paper's order:
  1. fill: every expert starts from its minimum units m_i;
  2. share: the budget left over is split among the experts still below
     saturation in proportion to their work coefficients w_i;
  3. clamp and refill: an expert pushed past its saturation s_i is held at
     s_i and its excess goes back into the pool, which is split again among
     the rest; repeat until nothing is returned.
Readings where the paper is open (listed with the design notes too):
  * units, minima, saturations and the budget are whole numbers of units
    (compute units or workgroup slots), the coefficients real; an expert with
    w_i = 0 keeps its minimum;
  * the budget must cover the minima, and m_i <= s_i; otherwise an error;
  * budget beyond sum(s_i) stays unassigned;
  * whole-unit shares: the largest-remainder rounding of the real shares to
    floor(sum of shares) units, each share rounded down or up, larger
    fractional parts first, ties to the lower index.
Shares no code with the library; only tests import it.
"""
from __future__ import annotations

import math


def fill_clamp_refill(m, s, w, budget):
    """Real-valued shares and the number of share-clamp rounds."""
    n = len(m)
    if any(x < 0 for x in m) or any(s[i] < m[i] for i in range(n)) or any(x < 0 for x in w):
        raise ValueError("invalid expert limits")
    if budget < sum(m):
        raise ValueError("the budget does not cover the minima")
    a = [float(x) for x in m]
    left = float(budget - sum(m))
    active = [i for i in range(n) if a[i] < s[i] and w[i] > 0]
    rounds = 0
    while left > 0 and active:
        W = sum(w[i] for i in active)
        for i in active:
            a[i] += left * w[i] / W
        rounds += 1
        left = 0.0
        still = []
        for i in active:
            if a[i] > s[i]:
                left += a[i] - s[i]
                a[i] = float(s[i])
            else:
                still.append(i)
        active = still
    return a, rounds


def round_units(a):
    """Largest-remainder rounding to floor(sum(a)) whole units."""
    base = [math.floor(x) for x in a]
    total = math.floor(sum(a) + 1e-9)
    extra = total - sum(base)
    order = sorted((i for i in range(len(a)) if a[i] > base[i]), key=lambda i: (base[i] - a[i], i))
    out = list(base)
    for i in order[:max(extra, 0)]:
        out[i] += 1
    return out
