"""Checks that pin the oracle to facts fixed by the paper and by mathematics.

Each check takes an oracle object (the default build of ``oracle/oracle.c``,
or a deliberately broken copy in the mutant tests) and raises AssertionError
when the oracle disagrees with:

* an independent computation (``decimal`` brute force, K-subset enumeration,
  numpy / torch library routines);
* a closed form (all-equal rows, V = 1, V = 2 logistic, x_i = ln i);
* an invariant stated in the paper (Theorem 1, the bound 1 <= d_j <= j, the
  merge operator being associative and commutative, overflow safety);
* the paper's tie semantics for top-k (Alg. 4's strictly-less insertion).

Every check is sized to run in well under a second.
"""
from __future__ import annotations

import json
import math
import os
import random

import numpy as np
import torch

import brute

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------- softmax ---
def check_softmax_decimal(orc):
    """Eq. 1 at 50 digits (brute force) vs the oracle, tiny rows, f32 and f64."""
    rng = _rng(1)
    for V in (1, 2, 3, 5, 8, 13, 16):
        for scale in (0.5, 3.0, 30.0):
            for dt in (np.float32, np.float64):
                x = (rng.standard_normal(V) * scale).astype(dt)
                y = orc.softmax(x)[0]
                ref = brute.softmax_decimal(x.tolist())
                np.testing.assert_allclose(y, ref, rtol=1e-13, atol=0)


def check_softmax_bf16_input(orc):
    """bfloat16 patterns are widened exactly: same answer as their f32 values."""
    rng = _rng(2)
    x = (rng.standard_normal((3, 40)) * 4).astype(np.float32)
    bits = (x.view(np.uint32) >> 16).astype(np.uint16)
    xw = (bits.astype(np.uint32) << 16).view(np.float32)
    y_bf = orc.softmax(bits, "bf16")
    y_f = orc.softmax(xw)
    assert np.array_equal(y_bf, y_f)
    for r in range(3):
        np.testing.assert_allclose(y_bf[r], brute.softmax_decimal(xw[r].tolist()),
                                   rtol=1e-13, atol=0)


def check_softmax_sums_to_one(orc):
    rng = _rng(3)
    for V in (1, 7, 100, 4097):
        x = (rng.standard_normal((4, V)) * 5).astype(np.float32)
        s = orc.softmax(x).sum(axis=1)
        assert np.all(np.abs(s - 1.0) <= V * 2.0 ** -52 + 1e-15), s


def check_softmax_closed_forms(orc):
    # all-equal rows: y = 1/V exactly (e^0 = 1, d = V exactly)
    for V in (1, 3, 10, 1000):
        for c in (-7.25, 0.0, 1000.0):
            y = orc.softmax(np.full(V, c, np.float32))[0]
            assert np.all(y == 1.0 / V), (V, c, y[:3])
    # V = 2: the logistic function of the difference
    for a, b in ((0.0, 1.0), (3.5, -2.0), (100.0, 99.0), (-1e3, -1e3 + 2.0)):
        y = orc.softmax(np.array([a, b], np.float64))[0]
        want0 = 1.0 / (1.0 + math.exp(b - a))
        assert abs(y[0] - want0) <= 1e-15 and abs(y[1] - (1.0 - want0)) <= 1e-15
    # x_i = ln i (i = 1..V): y_i = i / (V (V + 1) / 2)
    for V in (4, 100, 5000):
        i = np.arange(1, V + 1, dtype=np.float64)
        y = orc.softmax(np.log(i))[0]
        np.testing.assert_allclose(y, i / (V * (V + 1) / 2.0), rtol=1e-12, atol=0)


def check_softmax_shift_and_overflow(orc):
    """Shift invariance (Eq. 1 = Eq. 2) with shifts that are exact in binary64,
    and finite results at +-1000 where e^x itself overflows or underflows."""
    rng = _rng(4)
    base = np.round(rng.standard_normal((3, 257)) * 64.0) / 64.0  # dyadic grid
    y0 = orc.softmax(base)
    for c in (1000.0, -1000.0, 2.0 ** 20):
        y = orc.softmax(base + c)
        assert np.all(np.isfinite(y))
        np.testing.assert_allclose(y, y0, rtol=1e-13, atol=0)
    # the unprotected form overflows exactly where the paper says it does
    yn = orc.softmax_naive(base + 1000.0)
    assert not np.any(np.isfinite(yn))
    np.testing.assert_allclose(orc.softmax_naive(base), y0, rtol=1e-13, atol=0)


def check_softmax_nonfinite(orc):
    ninf, pinf, nan = -np.inf, np.inf, np.nan
    y = orc.softmax(np.array([0.0, ninf, math.log(3.0), ninf]))[0]
    np.testing.assert_allclose(y, [0.25, 0.0, 0.75, 0.0], rtol=1e-15, atol=0)
    assert y[1] == 0.0 and y[3] == 0.0
    for row in ([ninf, ninf], [1.0, pinf], [nan, 1.0]):
        assert np.all(np.isnan(orc.softmax(np.array(row))[0])), row


# ----------------------------------------------------------------- (m, d) ---
def check_theorem1(orc):
    """Alg. 3's recurrence yields m = max x and d = sum e^{x - m} (Theorem 1)."""
    rng = _rng(5)
    for V in (1, 2, 17, 1000, 30000):
        x = (rng.standard_normal((3, V)) * 3).astype(np.float32)
        m_on, d_on = orc.md_online(x)
        m_di, d_di = orc.md_direct(x)
        assert np.array_equal(m_on, x.max(axis=1).astype(np.float64))
        assert np.array_equal(m_di, m_on)
        np.testing.assert_allclose(d_on, d_di, rtol=1e-13, atol=0)
        # 1 <= d_V <= V
        assert np.all(d_on >= 1.0 - 1e-15) and np.all(d_on <= V * (1 + 1e-15))
    # d against the brute force for tiny rows
    for V in (1, 3, 9):
        x = rng.standard_normal(V) * 10
        m, d = orc.md_online(x)
        getcontext = __import__("decimal").getcontext
        getcontext().prec = 50
        D = __import__("decimal").Decimal
        want = sum((D(float(v)) - D(float(x.max()))).exp() for v in x)
        assert abs(d[0] - float(want)) <= 1e-14 * float(want)


def check_prefix_bound(orc):
    """1 <= d_j <= j for every prefix j of a row (the safety bound)."""
    rng = _rng(6)
    x = rng.standard_normal(300) * 20
    for j in range(1, 301):
        _, d = orc.md_online(x[:j])
        assert 1.0 - 1e-15 <= d[0] <= j * (1 + 1e-15), (j, d)


def check_combine_algebra(orc):
    """The merge operator: identity (-inf, 0), commutativity (bit-exact),
    associativity (random trees), and agreement with the meaning of a pair,
    d * e^m, evaluated in 50-digit decimal."""
    from decimal import Decimal, getcontext
    getcontext().prec = 50
    rng = _rng(7)
    ident = (-math.inf, 0.0)
    for _ in range(200):
        a = (float(rng.standard_normal() * 50), float(rng.uniform(1, 1000)))
        b = (float(rng.standard_normal() * 50), float(rng.uniform(1, 1000)))
        assert orc.md_combine(a, ident) == a and orc.md_combine(ident, a) == a
        ab, ba = orc.md_combine(a, b), orc.md_combine(b, a)
        assert ab == ba
        assert ab[0] == max(a[0], b[0])
        want = Decimal(a[1]) * Decimal(a[0]).exp() + Decimal(b[1]) * Decimal(b[0]).exp()
        got = Decimal(ab[1]) * Decimal(ab[0]).exp()
        assert abs(got - want) <= Decimal("1e-14") * want
    assert orc.md_combine(ident, ident) == ident
    # random splits, merge orders and trees give the pair of the whole row
    for V in (2, 5, 64, 999):
        x = rng.standard_normal(V) * 8
        m_all, d_all = orc.md_direct(x)
        for trial in range(20):
            cuts = sorted(set(rng.integers(1, V, size=min(V - 1, 6)).tolist())) if V > 1 else []
            bounds = [0] + cuts + [V]
            parts = []
            for lo, hi in zip(bounds[:-1], bounds[1:]):
                m, d = orc.md_direct(x[lo:hi])
                parts.append((m[0], d[0]))
            parts.append(ident)  # an empty chunk anywhere changes nothing
            random.Random(trial).shuffle(parts)
            while len(parts) > 1:  # random binary tree
                i = random.Random(trial * 7 + len(parts)).randrange(len(parts) - 1)
                parts[i:i + 2] = [orc.md_combine(parts[i], parts[i + 1])]
            assert parts[0][0] == m_all[0]
            assert abs(parts[0][1] - d_all[0]) <= 1e-13 * d_all[0]


# ------------------------------------------------------------------ top-k ---
def check_topk_enumeration(orc):
    """Eq. 5 plus the lower-index tie rule, by enumerating every K-subset of
    tiny rows drawn from a few values so that ties are common."""
    rng = _rng(8)
    for trial in range(60):
        V = int(rng.integers(1, 10))
        row = rng.choice([-1.5, 0.0, 0.5, 2.0, 2.0, 3.25], size=V).astype(np.float32)
        y = orc.softmax(row)[0]
        for K in range(1, V + 1):
            vals, idx = orc.topk(row, K)
            best, valid = brute.topk_enumerate(row.tolist(), K)
            assert idx[0].tolist() == best, (row, K, idx, best)
            assert np.array_equal(vals[0], y[idx[0]])


def check_topk_library(orc):
    """A stable argsort of -x (numpy) gives the same indices; invariants."""
    rng = _rng(9)
    x = np.round(rng.standard_normal((20, 3000)) * 4, 1).astype(np.float32)  # many ties
    for K in (1, 5, 50, 3000):
        vals, idx = orc.topk(x, K)
        y = orc.softmax(x)
        for r in range(x.shape[0]):
            want = np.argsort(-x[r].astype(np.float64), kind="stable")[:K]
            assert np.array_equal(idx[r], want)
            assert np.all(np.diff(vals[r]) <= 0)
            assert len(set(idx[r].tolist())) == K
            rest = np.setdiff1d(np.arange(3000), idx[r])
            if rest.size:
                assert vals[r].min() >= y[r, rest].max()
            assert vals[r].sum() <= 1.0 + 1e-12
            np.testing.assert_array_equal(vals[r], y[r, idx[r]])


def check_topk_select(orc):
    """K selection passes (Eq. 5 taken one rank at a time, online normalizer)
    agree with the sort, ties included."""
    rng = _rng(10)
    for trial in range(30):
        V = int(rng.integers(1, 400))
        K = int(rng.integers(1, min(V, 20) + 1))
        x = np.round(rng.standard_normal((2, V)) * 2, 1).astype(np.float32)
        v4, z4 = orc.topk_select(x, K)
        vs, zs = orc.topk(x, K)
        assert np.array_equal(z4, zs), (V, K)
        np.testing.assert_allclose(v4, vs, rtol=1e-13, atol=0)


def check_topk_signed_zero(orc):
    vals, idx = orc.topk(np.array([0.0, -0.0, 0.0, -1.0], np.float32), 3)
    assert idx[0].tolist() == [0, 1, 2]
    vals, idx = orc.topk(np.array([-0.0, 0.0], np.float32), 1)
    assert idx[0].tolist() == [0]


# --------------------------------------------------------------- bfloat16 ---
def _bf16_to_f64(bits):
    return (np.asarray(bits, np.uint32) << 16).view(np.float32).astype(np.float64)


def check_bf16_widening(orc):
    """Every one of the 65536 bfloat16 patterns widens to the value torch's
    bfloat16 -> float32 conversion gives (exact by the format's definition:
    the pattern is the upper half of a binary32), signed zeros and
    infinities included; NaN patterns stay NaN."""
    allb = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    got = orc.bf16_to_f64(allb)
    ref = torch.from_numpy(allb.view(np.int16)).view(torch.bfloat16).float().numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    ref64 = ref[~nan].astype(np.float64)  # signalling NaN patterns left out of the cast
    assert np.array_equal(got[~nan], ref64)
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref64))
    # a few patterns by hand: 1.0, -2.0, the smallest subnormal, -inf
    assert orc.bf16_to_f64(np.array([0x3F80, 0xC000, 0x0001, 0xFF80], np.uint16)).tolist() == \
        [1.0, -2.0, 2.0 ** -133, -math.inf]


def check_bf16_rounding(orc):
    """Every bfloat16 value maps to itself; exact midpoints go to the even
    neighbour; a hair off the midpoint goes to the nearer one; values that are
    binary32 agree with torch's float32 -> bfloat16 conversion."""
    allb = np.arange(0, 0x7F80, dtype=np.uint16)  # +0 .. largest finite
    v = _bf16_to_f64(allb)
    assert np.array_equal(orc.bf16_round(v), allb)
    assert np.array_equal(orc.bf16_round(-v), allb | 0x8000)
    lo, hi = v[:-1], v[1:]
    mid = (lo + hi) / 2.0  # exact in binary64
    got = orc.bf16_round(mid)
    even = np.where(allb[:-1] % 2 == 0, allb[:-1], allb[1:])
    assert np.array_equal(got, even)
    up = orc.bf16_round(mid + (hi - lo) * 2.0 ** -20)
    dn = orc.bf16_round(mid - (hi - lo) * 2.0 ** -20)
    assert np.array_equal(up, allb[1:]) and np.array_equal(dn, allb[:-1])
    # overflow: the largest finite value is odd, so the midpoint above it rounds
    # to the even neighbour 2^128, i.e. infinity; just below stays finite
    big = _bf16_to_f64(np.array([0x7F7F]))[0]
    assert orc.bf16_round(np.array([big + 2.0 ** 119]))[0] == 0x7F80
    assert orc.bf16_round(np.array([big + 2.0 ** 118]))[0] == 0x7F7F
    rng = _rng(11)
    f = (rng.standard_normal(100000) * np.exp(rng.uniform(-80, 80, 100000))).astype(np.float32)
    want = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(orc.bf16_round(f.astype(np.float64)), want)


# ----------------------------------------------------------------- golden ---
def check_golden(orc):
    """Hand-derived exact cases stored under tests/golden (see their notes)."""
    for name in sorted(os.listdir(GOLDEN)):
        if not name.endswith(".json"):
            continue
        with open(os.path.join(GOLDEN, name)) as f:
            case = json.load(f)
        x = np.array(case["x"], dtype={"f32": np.float32, "f64": np.float64}[case["dtype"]])
        if "y" in case:
            y = orc.softmax(x)
            np.testing.assert_allclose(y, np.array(case["y"], np.float64).reshape(y.shape),
                                       rtol=case.get("rtol", 1e-15), atol=0, err_msg=name)
        if "topk" in case:
            K = case["topk"]["K"]
            vals, idx = orc.topk(x, K)
            assert idx.tolist() == case["topk"]["idx"], name
            if "vals" in case["topk"]:
                np.testing.assert_allclose(vals, np.array(case["topk"]["vals"]),
                                           rtol=case.get("rtol", 1e-15), atol=0,
                                           err_msg=name)


def check_projection(orc):
    """The projection h . w^T against: integer arithmetic (small-integer inputs
    make every sum exact), numpy's matmul, the identity matrix, linearity in
    w, and bfloat16 inputs widened exactly."""
    rng = _rng(31)
    # exact: small integers scaled by powers of two
    h = (rng.integers(-4, 5, (7, 37)) * 0.125).astype(np.float32)
    w = (rng.integers(-4, 5, (11, 37)) * 0.0625).astype(np.float32)
    want = (np.rint(h * 8).astype(np.int64) @ np.rint(w * 16).astype(np.int64).T) / 128.0
    assert np.array_equal(orc.proj(h, w), want)
    # a library matmul on random inputs, non-square (a transposed operand fails)
    h = rng.standard_normal((5, 23)).astype(np.float32)
    w = rng.standard_normal((13, 23)).astype(np.float32)
    got = orc.proj(h, w)
    ref = h.astype(np.float64) @ w.astype(np.float64).T
    assert got.shape == (5, 13)
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)
    # identity weights give the hidden vectors back
    assert np.array_equal(orc.proj(h, np.eye(23, dtype=np.float32)), h.astype(np.float64))
    # linearity: doubling w doubles every logit exactly
    assert np.array_equal(orc.proj(h, 2 * w), 2 * orc.proj(h, w))
    # bfloat16 inputs: the same as their exact binary32 widening
    hb = torch.from_numpy(h).to(torch.bfloat16)
    wb = torch.from_numpy(w).to(torch.bfloat16)
    hbits = hb.view(torch.int16).numpy().view(np.uint16)
    wbits = wb.view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(orc.proj(hbits, wbits, "bf16", "bf16"),
                          orc.proj(hb.float().numpy(), wb.float().numpy()))


ALL = [
    check_softmax_decimal, check_softmax_bf16_input, check_softmax_sums_to_one,
    check_softmax_closed_forms, check_softmax_shift_and_overflow,
    check_softmax_nonfinite, check_theorem1, check_prefix_bound,
    check_combine_algebra, check_topk_enumeration, check_topk_library,
    check_topk_select, check_topk_signed_zero, check_bf16_widening, check_bf16_rounding,
    check_golden,
    check_projection,
]
