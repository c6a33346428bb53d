"""Independent brute-force references used to pin the oracle.

These share nothing with ``oracle/``: softmax is evaluated with Python's
``decimal`` module at 50 significant digits (Eq. 1 of Section 2, which equals
Eq. 2 in exact arithmetic), and top-k by enumerating every K-subset of a tiny
row and keeping the ones that satisfy Eq. 5 (Section 4) together with the
lower-index rule for ties.
"""
from __future__ import annotations

import itertools
from decimal import Decimal, getcontext


def softmax_decimal(row, digits: int = 50):
    """Eq. 1 evaluated with ``digits`` significant decimal digits."""
    getcontext().prec = digits
    xs = [Decimal(float(v)) for v in row]  # exact: every binary float is a decimal
    m = max(xs)  # shifting by the max keeps exp() small; exact in decimal
    es = [(v - m).exp() for v in xs]
    d = sum(es)
    return [float(e / d) for e in es]


def topk_enumerate(row, k: int):
    """All index sets z of size k with x_{z_i} >= x_j for every j outside z
    (Eq. 5 applied to x, whose order softmax preserves), then the one that the
    lower-index tie rule picks, returned in (value desc, index asc) order."""
    n = len(row)
    valid = []
    for z in itertools.combinations(range(n), k):
        inside = set(z)
        lo = min(row[i] for i in z)
        if all(row[j] <= lo for j in range(n) if j not in inside):
            valid.append(z)
    assert valid, "Eq. 5 always has a solution"
    # Tie rule: among the valid sets, the one whose indices at the boundary
    # value are the smallest; equivalently the lexicographically smallest set
    # after ordering each by (value desc, index asc).
    def ordered(z):
        return sorted(z, key=lambda i: (-row[i], i))
    best = min((ordered(z) for z in valid), key=lambda zz: [(-row[i], i) for i in zz])
    return best, valid
