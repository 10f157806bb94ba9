"""Pins for the LARS oracle (Eq. lars and the step of the LARS method):
checks against facts fixed by the definitions and by mathematics.

Each ``pin_*`` takes the oracle module (``oracle.lars`` or a broken copy).
Sources of truth:
  * closed forms: constant layers (w = c, g = e on n positions with n a power
    of four, so every square root is exact): rate = gamma eta |c| /
    (|e| + eps |c|), independent of n;
  * the norm as a decimal computation (60 significant digits) of the square
    root of the exact sum of squares;
  * hand-worked steps in exact dyadic arithmetic (rate 2 by construction:
    w = 2, g = 1/2, eps = 1/4, gamma = eta = 1), with and without momentum;
  * layer independence: a layer's rate does not depend on the other layers in
    the list;
  * Eq. (lars) at zero norms: ||w|| = 0 < ||g|| gives 0 and ||g|| = 0 < ||w||
    gives gamma eta / eps (the equation's value, checked against exact
    rationals), and a hand-worked dyadic step for the zero-gradient layer;
    a zero denominator (0/0, or eps = 0 with g = 0) gives the reading's 0;
  * the step over several layers against the same step layer by layer;
  * a hand-worked case where binary32 rounding of the rate and of D decides
    the result (exactly 0 in binary32, about 2^-25 with wider arithmetic).
"""
from __future__ import annotations

from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np


def pin_lars_constant_layers(lars):
    for n in (1, 4, 16, 4096):
        for c, e in ((2.0, 0.5), (-0.75, 3.0), (1e-3, 2.0 ** -20)):
            for gamma, eta, eps in ((1.0, 1.0, 0.0), (0.001, 0.1, 5e-5), (0.5, 2.0, 0.25)):
                w = np.full(n, c, np.float32)
                g = np.full(n, e, np.float32)
                r = lars.lars_rates([w], [g], gamma, eta, eps)[0]
                C, E = abs(float(np.float32(c))), abs(float(np.float32(e)))
                exp = gamma * eta * C / (E + eps * C)
                assert abs(r - exp) <= 4e-16 * exp, (n, c, e, gamma, eta, eps, r, exp)


def pin_lars_norm_decimal(lars):
    getcontext().prec = 60
    rng = np.random.default_rng(71)
    for n in (3, 1000, 65_537):
        v = (rng.standard_normal(n) * np.exp2(rng.integers(-20, 20, n))).astype(np.float32)
        S = sum(Decimal(float(x)) * Decimal(float(x)) for x in v)
        exact = S.sqrt()
        got = Decimal(lars.layer_norm(v))
        assert abs(got - exact) <= exact * Decimal(2) ** -52, (n, got, exact)


def pin_lars_zero_norms(lars):
    # n = 16 positions of 0 or 1: the norms are 0 or exactly 4
    z = np.zeros(16, np.float32)
    o = np.ones(16, np.float32)
    # ||w|| = 0 < ||g||: gamma eta 0 / (4 + eps 0) = 0
    for eps in (0.0, 0.25, 1e-4):
        assert lars.lars_rates([z], [o], 0.5, 0.25, eps)[0] == 0.0
    # ||g|| = 0 < ||w||: gamma eta 4 / (eps 4) = gamma eta / eps
    for gamma, eta, eps in ((0.5, 0.25, 0.25), (0.001, 0.1, 5e-5), (2.0, 3.0, 1e-4)):
        r = lars.lars_rates([o], [z], gamma, eta, eps)[0]
        exact = Fraction(gamma) * Fraction(eta) / Fraction(eps)
        assert abs(Fraction(r) - exact) <= exact * Fraction(1, 2 ** 50), (gamma, eta, eps, r)
    assert lars.lars_rates([o], [z], 0.5, 0.25, 0.25)[0] == 0.5
    # a zero denominator: 0/0, and ||w|| / 0 with eps = 0 (the reading: 0)
    assert lars.lars_rates([z], [z], 0.5, 0.25, 0.25)[0] == 0.0
    assert lars.lars_rates([o], [z], 0.5, 0.25, 0.0)[0] == 0.0
    # the zero-gradient layer's step: rate 1/2, D = w / 4 = 1/4, U = 1/8,
    # w' = 7/8 (every value dyadic, so exact); momentum 1/2 on b = 1:
    # b' = 1/2 + 1/8 = 5/8, w' = 1 - 5/8 = 3/8
    w2, _, rates = lars.lars_update([o], None, [z], 0.5, 0.25, 0.25, 0.0)
    assert rates[0] == 0.5 and np.all(w2[0] == np.float32(0.875))
    w3, b3, _ = lars.lars_update([o], [np.ones(16, np.float32)], [z], 0.5, 0.25, 0.25, 0.5)
    assert np.all(b3[0] == np.float32(0.625)) and np.all(w3[0] == np.float32(0.375))
    # the zero-weight layer does not move (rate 0, D = g, U = 0)
    w4, _, _ = lars.lars_update([z], None, [o], 0.5, 0.25, 0.25, 0.0)
    assert np.all(w4[0] == 0.0)


def pin_lars_worked_steps(lars):
    # n = 16: ||w|| = 8, ||g|| = 2, eps = 1/4 -> rate = 8 / (2 + 2) = 2
    n = 16
    w = np.full(n, 2.0, np.float32)
    g = np.full(n, 0.5, np.float32)
    w[::3] = -2.0
    g[::3] = -0.5
    w2, b2, rates = lars.lars_update([w], None, [g], 1.0, 1.0, 0.25, 0.0)
    assert rates[0] == 2.0
    # D = g + w / 4 = +-1, U = 2 D = +-2: w - U = 0 everywhere
    assert np.all(w2[0] == 0.0) and b2 is None
    b = np.full(n, 1.0, np.float32)
    w3, b3, _ = lars.lars_update([w], [b], [g], 1.0, 1.0, 0.25, 0.5)
    for i in range(n):
        s = -1 if i % 3 == 0 else 1
        B = Fraction(1, 2) * 1 + 2 * s            # mu b + rate D
        W = Fraction(2 * s) - B
        assert Fraction(float(b3[0][i])) == B and Fraction(float(w3[0][i])) == W, i


def pin_lars_layer_independence(lars):
    rng = np.random.default_rng(72)
    A = [rng.standard_normal(500).astype(np.float32) for _ in range(2)]
    B = [rng.standard_normal(70).astype(np.float32) * 9 for _ in range(2)]
    r_both = lars.lars_rates([A[0], B[0]], [A[1], B[1]], 0.01, 0.1, 1e-4)
    r_a = lars.lars_rates([A[0]], [A[1]], 0.01, 0.1, 1e-4)
    r_b = lars.lars_rates([B[0]], [B[1]], 0.01, 0.1, 1e-4)
    assert r_both[0] == r_a[0] and r_both[1] == r_b[0]
    assert r_both[0] != r_both[1]


def pin_lars_rate_direction(lars):
    # a larger weight norm raises the rate, a larger gradient norm lowers it
    w = np.ones(64, np.float32)
    g = np.ones(64, np.float32)
    base = lars.lars_rates([w], [g], 1.0, 1.0, 0.1)[0]
    assert lars.lars_rates([2 * w], [g], 1.0, 1.0, 0.1)[0] > base
    assert lars.lars_rates([w], [2 * g], 1.0, 1.0, 0.1)[0] < base
    # eps = 0: exactly ||w|| / ||g|| times gamma eta
    assert lars.lars_rates([3 * w], [g], 1.0, 1.0, 0.0)[0] == 3.0


def pin_lars_step_layerwise(lars):
    rng = np.random.default_rng(73)
    sizes = [5, 300, 1]
    ws = [rng.standard_normal(n).astype(np.float32) for n in sizes]
    gs = [rng.standard_normal(n).astype(np.float32) * 0.01 for n in sizes]
    bs = [rng.standard_normal(n).astype(np.float32) * 0.1 for n in sizes]
    w2, b2, rates = lars.lars_update(ws, bs, gs, 0.001, 2.0, 5e-4, 0.9)
    for t in range(3):
        w1, b1, r1 = lars.lars_update([ws[t]], [bs[t]], [gs[t]], 0.001, 2.0, 5e-4, 0.9)
        assert r1[0] == rates[t]
        assert np.array_equal(w1[0], w2[t]) and np.array_equal(b1[0], b2[t])
    # momentum 0 with b given equals the plain step (b = rate D)
    w4, b4, _ = lars.lars_update(ws, [np.zeros(n, np.float32) for n in sizes], gs,
                                 0.001, 2.0, 5e-4, 0.0)
    w5, _, _ = lars.lars_update(ws, None, gs, 0.001, 2.0, 5e-4, 0.0)
    for t in range(3):
        assert np.array_equal(w4[t], w5[t])


def pin_lars_binary32_rounding(lars):
    # w = g = 1 (one position), eps = 2^-25, gamma = eta = 1: the rate is
    # 1 / (1 + 2^-25), just above the midpoint between 1 - 2^-24 and 1, so it
    # rounds to 1 in binary32; D = 1 + 2^-25 rounds to 1 (below half an ulp
    # of 1); U = 1 and w - U = 0 exactly. Any wider intermediate leaves
    # about 2^-25 behind.
    w = np.ones(1, np.float32)
    g = np.ones(1, np.float32)
    eps = 2.0 ** -25
    w2, b2, rates = lars.lars_update([w], None, [g], 1.0, 1.0, eps, 0.0)
    assert rates[0] == 1.0 / (1.0 + eps) and np.float32(rates[0]) == np.float32(1.0)
    assert w2[0].dtype == np.float32 and w2[0][0] == 0.0
    w3, b3, _ = lars.lars_update([w], [np.zeros(1, np.float32)], [g], 1.0, 1.0, eps, 0.5)
    assert b3[0].dtype == np.float32 and b3[0][0] == 1.0 and w3[0][0] == 0.0


ALL_LARS_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_lars_")]
