"""Pins for the CPU oracle: checks against facts fixed by the paper's
definitions and by mathematics, not against the oracle's own formulas.

Each ``pin_*`` takes an ``oracle.Oracle`` and raises AssertionError (or
OracleError) on a mismatch. ``test_oracle_pins.py`` runs them on the real
oracle; ``test_oracle_mutants.py`` runs them on deliberately broken builds of
the oracle source and requires every broken build to fail at least one pin.

Sources of truth used here:
  * the rank definition of the TopK operator (Sec. 3.1) evaluated by brute
    force, O(d^2), in plain numpy / Python;
  * exhaustive enumeration of tie patterns on tiny vectors;
  * reductions to library routines: argmax (k = 1), argpartition (distinct
    magnitudes), lexsort (a third, independent ordering);
  * binary32 arithmetic emulated in float64: a float32 sum or difference of
    two float32 values equals float32(float64 sum) (double rounding is
    innocuous because 53 >= 2*24 + 2), and a float32 product of two float32
    values is exact in float64 before its one rounding;
  * exact rational arithmetic (fractions) on dyadic inputs, where every
    binary32 operation is exact in any order;
  * closed forms: geometric momentum series, (1 - lr*wd)^t decay, P-fold sums.
"""
from __future__ import annotations

import itertools
from decimal import Decimal, ROUND_CEILING
from fractions import Fraction

import numpy as np

from oracle import GLOBAL, PER_TENSOR

F32 = np.float32


def bits(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def brute_select(x: np.ndarray, k: int) -> np.ndarray:
    """{i : rank_i < k}, rank_i = #{|x_j| > |x_i|} + #{j < i, |x_j| == |x_i|}."""
    a = np.abs(x.astype(np.float64))
    n = a.size
    gt = (a[None, :] > a[:, None]).sum(1)
    eq_before = ((a[None, :] == a[:, None]) & (np.arange(n)[None, :] < np.arange(n)[:, None])).sum(1)
    rank = gt + eq_before
    return np.nonzero(rank < k)[0]


def _rng(seed):
    return np.random.default_rng(seed)


def _tie_vector(rng, n, levels):
    mags = rng.integers(0, levels, n).astype(np.float32) * F32(0.25)
    signs = np.where(rng.random(n) < 0.5, F32(-1), F32(1))
    return (mags * signs).astype(np.float32)


# ---------------------------------------------------------------- selection

def pin_brute_force_rank(orc):
    rng = _rng(11)
    for n in (1, 2, 3, 7, 64, 257, 700):
        for trial in range(3):
            if trial == 0:
                x = rng.standard_normal(n).astype(np.float32)
            elif trial == 1:
                x = _tie_vector(rng, n, 5)
            else:
                x = _tie_vector(rng, n, max(2, n // 3))
            ks = range(1, n + 1) if n <= 64 else sorted({1, 2, n // 7 + 1, n // 2, n - 1, n})
            for k in ks:
                sel = orc.topk_select(x, k)
                exp = brute_select(x, k)
                assert np.array_equal(sel, exp), (n, trial, k)


def pin_exhaustive_ties(orc):
    alphabet = [F32(-2), F32(-1), F32(-0.0), F32(0.0), F32(1), F32(2)]
    for n in range(1, 6):
        for combo in itertools.product(range(len(alphabet)), repeat=n):
            x = np.array([alphabet[c] for c in combo], dtype=np.float32)
            for k in range(1, n + 1):
                sel = orc.topk_select(x, k)
                assert np.array_equal(sel, brute_select(x, k)), (x.tolist(), k)


def pin_k1_is_first_argmax(orc):
    rng = _rng(12)
    for n in (1, 5, 100, 4097):
        for levels in (3, 50):
            x = _tie_vector(rng, n, levels)
            sel = orc.topk_select(x, 1)
            assert sel.tolist() == [int(np.argmax(np.abs(x)))]
        y = rng.standard_normal(n).astype(np.float32)
        assert orc.topk_select(y, 1).tolist() == [int(np.argmax(np.abs(y)))]


def pin_distinct_matches_argpartition(orc):
    rng = _rng(13)
    for n in (10, 1000, 50_000):
        x = rng.permutation(np.arange(1, n + 1, dtype=np.float64)).astype(np.float32)
        x *= np.where(rng.random(n) < 0.5, -1, 1).astype(np.float32)
        for k in (1, 3, n // 10 + 1, n - 1, n):
            exp = np.sort(np.argpartition(-np.abs(x), k - 1)[:k])
            assert np.array_equal(orc.topk_select(x, k), exp), (n, k)
            # the k largest of a permutation of 1..n are the values n-k+1..n
            assert set(np.abs(x[orc.topk_select(x, k)]).astype(np.int64).tolist()) == \
                set(range(n - k + 1, n + 1))


def pin_k_equals_d_and_all_equal(orc):
    rng = _rng(14)
    for n in (1, 9, 1000):
        x = rng.standard_normal(n).astype(np.float32)
        assert np.array_equal(orc.topk_select(x, n), np.arange(n))
        c = np.where(rng.random(n) < 0.5, F32(-3.5), F32(3.5)).astype(np.float32)
        for k in (1, n // 2 + 1, n):
            assert np.array_equal(orc.topk_select(c, k), np.arange(k))


def pin_zero_inf_denormal_order(orc):
    tiny = np.float32(np.finfo(np.float32).smallest_subnormal)
    x = np.array([0.0, -0.0, tiny, -2 * tiny, np.inf, 1.0, -np.inf, -tiny, 3 * tiny,
                  np.float32(np.finfo(np.float32).max)], dtype=np.float32)
    # magnitude order: inf(4), inf(6), max(9), 1(5), 3t(8), 2t(3), t(2), t(7), 0(0), 0(1)
    order = [4, 6, 9, 5, 8, 3, 2, 7, 0, 1]
    for k in range(1, x.size + 1):
        assert np.array_equal(orc.topk_select(x, k), np.sort(order[:k])), k
    z = np.array([-0.0, 0.0, -0.0, 0.0, -0.0], dtype=np.float32)
    g = z.copy()
    r = np.zeros_like(z)
    idx, val, r_out = orc.sparsify_flat(g, r, 3)
    assert idx.tolist() == [0, 1, 2]
    # -0 + +0 = +0 under round-to-nearest, so every x here is +0
    assert bits(val).tolist() == [0, 0, 0]
    idx, val, r_out = orc.sparsify_flat(z, z.copy(), 2)
    # -0 + -0 = -0: the sign of zero survives into val
    assert bits(val).tolist() == [0x80000000, 0]


def pin_lexsort_midsize(orc):
    rng = _rng(15)
    n = 200_000
    x = (np.round(rng.standard_normal(n) * 64) / 64).astype(np.float32)  # many ties
    for k in (1, 200, 20_000):
        order = np.lexsort((np.arange(n), -np.abs(x.astype(np.float64))))
        exp = np.sort(order[:k])
        assert np.array_equal(orc.topk_select(x, k), exp), k


def pin_sorted_known_answer(orc):
    # values are the positions themselves: the top-k are the last k positions
    n = 4096
    x = np.arange(n, dtype=np.float32)
    for k in (1, 17, n):
        assert np.array_equal(orc.topk_select(x, k), np.arange(n - k, n))
    # reversed: the first k positions; negated magnitudes do not change that
    assert np.array_equal(orc.topk_select(-x[::-1].copy(), 5), np.arange(5))


# ---------------------------------------------------------- residual add

def _awkward_pairs(rng, n):
    # exponents from below the subnormal range up to 2^120: subnormal sums,
    # cancellations and sums where one operand is far below the other's ulp
    e = rng.integers(-155, 90, n).astype(np.float64)
    g = (rng.standard_normal(n) * np.exp2(e)).astype(np.float32)
    r = (rng.standard_normal(n) * np.exp2(e + rng.integers(-30, 30, n))).astype(np.float32)
    g[::7] = -r[::7]                       # exact cancellation
    g[::11] = np.float32(np.finfo(np.float32).smallest_subnormal)
    r[::13] = 0.0
    r[::17] = -0.0
    g[::19] = -0.0
    return g, r


def pin_ef_add_binary32(orc):
    rng = _rng(16)
    g, r = _awkward_pairs(rng, 100_000)
    x = orc.ef_add(g, r)
    with np.errstate(over="ignore"):
        exp = (g.astype(np.float64) + r.astype(np.float64)).astype(np.float32)
    assert np.array_equal(bits(x), bits(exp))


def pin_sparsify_invariants(orc):
    rng = _rng(17)
    for n, k in ((1, 1), (100, 7), (10_000, 10), (65_537, 655)):
        g = rng.standard_normal(n).astype(np.float32)
        r = (rng.standard_normal(n) * 0.5).astype(np.float32)
        r[: n // 3] = 0.0
        x = (g.astype(np.float64) + r.astype(np.float64)).astype(np.float32)
        idx, val, r_out = orc.sparsify_flat(g, r, k)
        assert idx.size == k and np.all(np.diff(idx.astype(np.int64)) > 0)
        assert np.array_equal(bits(val), bits(x[idx]))
        mask = np.zeros(n, bool)
        mask[idx] = True
        assert np.all(bits(r_out[mask]) == 0)
        assert np.array_equal(bits(r_out[~mask]), bits(x[~mask]))
        if k < n:
            assert np.abs(val).min() >= np.abs(r_out[~mask]).max()
        assert np.array_equal(np.sort(idx), brute_select(x, k)) if n <= 2000 else True


def pin_residual_carry_conserves_mass(orc):
    """Over several error-feedback steps, everything fed in is either sent
    or still held in the residual: sum_t g_t == sum_t sent_t + r_T, exactly
    on a dyadic grid where every float32 addition is exact."""
    rng = _rng(18)
    n, k, steps = 5000, 50, 6
    r = np.zeros(n, np.float32)
    sent = np.zeros(n, np.float64)
    fed = np.zeros(n, np.float64)
    for t in range(steps):
        g = (rng.integers(-64, 65, n) / 64.0).astype(np.float32)
        fed += g
        idx, val, r = orc.sparsify_flat(g, r, k)
        np.add.at(sent, idx, val.astype(np.float64))
    assert np.array_equal(fed, sent + r.astype(np.float64))


def pin_k_from_rho(orc):
    cases = {(1_048_576, "0.001"): 1049, (25_557_032, "0.001"): 25_558,
             (25_600_000, "0.001"): 25_600, (109_708_544, "0.001"): 109_709,
             (109_708_544, "0.01"): 1_097_086, (340_000_000, "0.001"): 340_000,
             (3_194_629, "0.001"): 3195, (1, "0.001"): 1, (10, "1"): 10, (7, "0.5"): 4}
    for (d, rho), k in cases.items():
        exact = int((Decimal(rho) * d).to_integral_value(rounding=ROUND_CEILING))
        assert max(1, min(d, exact)) == k
        assert orc.k_from_rho(d, float(rho)) == k, (d, rho)
    assert orc.k_from_rho(10, 0.0) < 0 and orc.k_from_rho(10, 1.5) < 0


def pin_per_tensor_groups(orc):
    rng = _rng(19)
    sizes = [1, 5, 64, 300, 1000]
    grads = [_tie_vector(rng, n, 6) for n in sizes]
    res = [np.zeros(n, np.float32) for n in sizes]
    idx, val, outs, ks = orc.sparsify(grads, res, rho=0.05, mode=PER_TENSOR)
    offs = np.concatenate([[0], np.cumsum(sizes)])
    assert ks == [max(1, min(n, int(np.ceil(0.05 * n)))) for n in sizes]
    pos = 0
    for t, n in enumerate(sizes):
        exp = brute_select(grads[t], ks[t]) + offs[t]
        assert np.array_equal(idx[pos:pos + ks[t]], exp)
        pos += ks[t]
    gidx, _, _, gk = orc.sparsify(grads, res, rho=0.05, mode=GLOBAL)
    cat = np.concatenate(grads)
    assert gk == [int(np.ceil(0.05 * cat.size))]
    assert np.array_equal(gidx, brute_select(cat, gk[0]))


# ---------------------------------------------------------------- update

def _f32_mul(a, b):
    return (np.asarray(a, np.float64) * np.asarray(b, np.float64)).astype(np.float32)


def _f32_sub(a, b):
    return (np.asarray(a, np.float64) - np.asarray(b, np.float64)).astype(np.float32)


def pin_update_single_worker_closed_form(orc):
    rng = _rng(21)
    d, k = 50_000, 777
    w0 = rng.standard_normal(d).astype(np.float32)
    idx = np.sort(rng.choice(d, k, replace=False)).astype(np.int32)
    val = rng.standard_normal(k).astype(np.float32)
    lr = np.float32(0.1)
    w, _ = orc.update(w0, None, idx, val, lr=lr)
    exp = w0.copy()
    exp[idx] = _f32_sub(w0[idx], _f32_mul(lr, val))
    assert np.array_equal(bits(w), bits(exp))


def _dyadic_lists(rng, d, P, k, overlap=True):
    idx = np.empty((P, k), np.int32)
    pool = rng.choice(d, size=min(d, 3 * k), replace=False) if overlap else None
    for p in range(P):
        src = pool if overlap else np.arange(d)
        idx[p] = np.sort(rng.choice(src, size=k, replace=False))
    e = rng.integers(-8, -3, (P, k)).astype(np.float64)
    val = (np.exp2(e) * np.where(rng.random((P, k)) < 0.5, -1, 1)).astype(np.float32)
    return idx, val


def pin_update_dyadic_exact(orc):
    rng = _rng(22)
    d, P, k = 4096, 9, 300
    w0 = (rng.integers(-4095, 4096, d) / 256.0).astype(np.float32)
    lr, mu = Fraction(1, 4), Fraction(1, 2)
    for wd in (Fraction(0), Fraction(1, 16)):
        steps = 3 if wd == 0 else 1
        w = w0.copy()
        b = np.zeros(d, np.float32)
        W = [Fraction(float(v)) for v in w0]
        B = [Fraction(0)] * d
        for s in range(steps):
            idx, val = _dyadic_lists(rng, d, P, k)
            w, b = orc.update(w, b, idx, val, lr=float(lr), mu=float(mu), wd=float(wd))
            G = [Fraction(0)] * d
            for p in range(P):
                for j in range(k):
                    G[idx[p, j]] += Fraction(float(val[p, j]))
            for i in range(d):
                D = G[i] + wd * W[i]
                B[i] = mu * B[i] + D
                W[i] = W[i] - lr * B[i]
            assert np.array_equal(w, np.array([float(v) for v in W], np.float32)), (wd, s)
            assert np.array_equal(b, np.array([float(v) for v in B], np.float32)), (wd, s)
    # plain mode, several workers, dyadic: exact against a float64 densification
    idx, val = _dyadic_lists(rng, d, P, k)
    w, _ = orc.update(w0, None, idx, val, lr=0.25)
    G = np.zeros(d, np.float64)
    np.add.at(G, idx.ravel(), val.ravel().astype(np.float64))
    touched = np.zeros(d, bool)
    touched[idx.ravel()] = True
    exp = w0.astype(np.float64) - np.where(touched, 0.25 * G, 0.0)
    assert np.array_equal(w, exp.astype(np.float32))


def pin_update_float64_densify_bound(orc):
    rng = _rng(23)
    d, P, k = 20_000, 16, 2000
    w0 = (rng.standard_normal(d) * 0.1).astype(np.float32)
    idx = np.stack([np.sort(rng.choice(d, k, replace=False)) for _ in range(P)]).astype(np.int32)
    val = (rng.standard_normal((P, k)) * 1e-2).astype(np.float32)
    lr = 0.1
    w, _ = orc.update(w0, None, idx, val, lr=lr)
    G = np.zeros(d)
    A = np.zeros(d)
    np.add.at(G, idx.ravel(), val.ravel().astype(np.float64))
    np.add.at(A, idx.ravel(), np.abs(val.ravel().astype(np.float64)))
    cnt = np.bincount(idx.ravel(), minlength=d)
    touched = cnt > 0
    exp = w0.astype(np.float64) - np.where(touched, np.float64(np.float32(lr)) * G, 0.0)
    u = 2.0 ** -24
    bound = 2 * u * np.abs(exp) + np.float32(lr) * (cnt + 2) * u * A + 1e-45
    assert np.all(np.abs(w.astype(np.float64) - exp) <= bound)
    assert np.array_equal(bits(w[~touched]), bits(w0[~touched]))


def pin_update_sum_not_mean(orc):
    d, P = 64, 7
    w0 = np.full(d, 1.0, np.float32)
    idx = np.full((P, 1), 5, np.int32)
    val = np.full((P, 1), 0.125, np.float32)
    w, _ = orc.update(w0, None, idx, val, lr=0.5)
    assert w[5] == np.float32(1.0 - 0.5 * P * 0.125)
    assert np.all(w[np.arange(d) != 5] == 1.0)


def pin_update_duplicates_within_list(orc):
    w0 = np.zeros(10, np.float32)
    idx = np.array([[2, 2, 2, 7]], np.int32)
    val = np.array([[1.0, 2.0, 4.0, 8.0]], np.float32)
    w, _ = orc.update(w0, None, idx, val, lr=1.0)
    assert w[2] == -7.0 and w[7] == -8.0 and np.count_nonzero(w) == 2


def pin_momentum_geometric_series(orc):
    # constant gradient G each step, wd = 0, b0 = 0:
    # b_t = G (1 - mu^t) / (1 - mu); w_t = w0 - lr * sum_{s<=t} b_s
    d = 16
    G = np.array([2.0 ** -(i % 5 + 2) * (-1) ** i for i in range(d)], np.float32)
    idx = np.arange(d, dtype=np.int32)[None, :]
    w = np.full(d, 3.0, np.float32)
    b = np.zeros(d, np.float32)
    lr, mu = Fraction(1, 4), Fraction(1, 2)
    for t in range(1, 6):
        w, b = orc.update(w, b, idx, G[None, :], lr=float(lr), mu=float(mu), wd=0.0)
        for i in range(d):
            g = Fraction(float(G[i]))
            bt = g * (1 - mu ** t) / (1 - mu)
            wt = 3 - lr * sum(g * (1 - mu ** s) / (1 - mu) for s in range(1, t + 1))
            assert Fraction(float(b[i])) == bt and Fraction(float(w[i])) == wt, (t, i)


def pin_weight_decay_power(orc):
    # no gradient, mu = 0, wd != 0: w_t = w0 (1 - lr wd)^t
    d = 8
    w0 = np.array([1, -2, 4, -8, 0.5, 3, -0.25, 16], np.float32)
    w = w0.copy()
    lr, wd = Fraction(1, 4), Fraction(1, 16)
    idx = np.zeros((1, 0), np.int32)
    val = np.zeros((1, 0), np.float32)
    for t in range(1, 4):
        w, _ = orc.update(w, None, idx, val, lr=float(lr), mu=0.0, wd=float(wd))
        for i in range(d):
            assert Fraction(float(w[i])) == Fraction(float(w0[i])) * (1 - lr * wd) ** t


def pin_update_worker_permutation(orc):
    rng = _rng(24)
    d, P, k = 30_000, 12, 3000
    w0 = (rng.standard_normal(d) * 0.1).astype(np.float32)
    b0 = (rng.standard_normal(d) * 0.01).astype(np.float32)
    idx = np.stack([np.sort(rng.choice(d, k, replace=False)) for _ in range(P)]).astype(np.int32)
    val = (rng.standard_normal((P, k)) * 1e-2).astype(np.float32)
    perm = rng.permutation(P)
    w1, b1 = orc.update(w0, b0, idx, val, lr=0.1, mu=0.9, wd=5e-5)
    w2, b2 = orc.update(w0, b0, idx[perm], val[perm], lr=0.1, mu=0.9, wd=5e-5)
    cnt = np.bincount(idx.ravel(), minlength=d)
    # with at most two contributions a float32 sum does not depend on order
    le2 = cnt <= 2
    assert np.array_equal(bits(w1[le2]), bits(w2[le2])) and np.array_equal(bits(b1[le2]), bits(b2[le2]))
    A = np.zeros(d)
    np.add.at(A, idx.ravel(), np.abs(val.ravel().astype(np.float64)))
    S = 0.1 * (A + 5e-5 * np.abs(w0) + 0.9 * np.abs(b0))
    assert np.all(np.abs(w1.astype(np.float64) - w2) <= 1e-6 * (np.abs(w1) + S))
    assert np.all(np.abs(b1.astype(np.float64) - b2) <= 1e-6 * (np.abs(b1) + S / 0.1))


def pin_aggregate_dyadic_exact(orc):
    # dyadic values with a small exponent range: every binary32 partial sum is
    # exact, so the dense sum equals the rational sum of each position
    rng = _rng(25)
    d, P, k = 3000, 11, 400
    idx, val = _dyadic_lists(rng, d, P, k)
    nnz = rng.integers(0, k + 1, P)
    nnz[0] = k
    out = orc.aggregate(d, idx, val, nnz)
    G = [Fraction(0)] * d
    for p in range(P):
        for j in range(int(nnz[p])):
            G[idx[p, j]] += Fraction(float(val[p, j]))
    exp = np.array([float(v) for v in G], np.float32)
    assert np.array_equal(bits(out), bits(np.where(exp == 0, np.float32(0), exp)))


def pin_aggregate_worker_order_and_zero(orc):
    # g~ starts at +0 and the lists are added one worker after the other:
    # 1 + 2^-24 rounds to 1 (tie to even), so two such terms after a 1 vanish,
    # while the same terms first would give 1 + 2^-23
    t = np.float32(2.0 ** -24)
    idx = np.array([[0, 3], [0, 3], [0, 3]], np.int32)
    val = np.array([[1.0, t], [t, t], [t, 1.0]], np.float32)
    out = orc.aggregate(6, idx, val)
    assert out[0] == np.float32(1.0)
    assert out[3] == np.float32(1.0 + 2.0 ** -23)
    # untouched positions are +0; a lone -0 added to +0 gives +0; P = 0 gives zeros
    assert np.array_equal(bits(out[[1, 2, 4, 5]]), np.zeros(4, np.uint32))
    out = orc.aggregate(4, np.array([[2]], np.int32), np.array([[-0.0]], np.float32))
    assert np.array_equal(bits(out), np.zeros(4, np.uint32))
    out = orc.aggregate(5, np.zeros((0, 3), np.int32), np.zeros((0, 3), np.float32),
                        np.zeros(0, np.int64))
    assert np.array_equal(bits(out), np.zeros(5, np.uint32))


def pin_aggregate_float64_bound(orc):
    # worker-ordered binary32 sum of c terms: within (c - 1) u sum|v| of the
    # exact sum (standard recursive-summation bound), duplicates included
    rng = _rng(26)
    d, P, k = 20_000, 16, 2500
    idx = np.stack([np.sort(rng.choice(d, k, replace=False)) for _ in range(P)]).astype(np.int32)
    idx[3, :40] = 17  # one list naming the same position many times
    val = (rng.standard_normal((P, k)) * 1e-2).astype(np.float32)
    out = orc.aggregate(d, idx, val)
    G, A = np.zeros(d), np.zeros(d)
    np.add.at(G, idx.ravel(), val.ravel().astype(np.float64))
    np.add.at(A, idx.ravel(), np.abs(val.ravel().astype(np.float64)))
    cnt = np.bincount(idx.ravel(), minlength=d)
    u = 2.0 ** -24
    assert np.all(np.abs(out.astype(np.float64) - G) <= np.maximum(cnt - 1, 0) * u * A * 1.0001 + 1e-45)
    assert np.array_equal(bits(out[cnt == 0]), np.zeros(int((cnt == 0).sum()), np.uint32))
    # a position named once carries its value bit for bit
    one = cnt == 1
    assert np.array_equal(bits(out[one]), bits(G[one].astype(np.float32)))


def pin_f16_known_conversions(orc):
    # IEEE binary16 facts: largest finite 65504; 65520 is the midpoint to the
    # next (absent) step and rounds to infinity; 2^-24 is the least subnormal,
    # 2^-25 ties to 0 (even), 3*2^-25 ties up to 2^-23; 1/3 -> 0x3555;
    # 1 + 2^-11 ties to 1, 1 + 3*2^-11 ties up to 1 + 2^-9
    from oracle import f16_rne
    cases = [(65504.0, 0x7BFF), (65519.0, 0x7BFF), (65520.0, 0x7C00), (-1e9, 0xFC00),
             (2.0 ** -24, 0x0001), (2.0 ** -25, 0x0000), (3 * 2.0 ** -25, 0x0002),
             (-(2.0 ** -14), 0x8400), (np.float32(1 / 3), 0x3555), (1.0 + 2.0 ** -11, 0x3C00),
             (1.0 + 3 * 2.0 ** -11, 0x3C02), (-0.0, 0x8000), (np.inf, 0x7C00)]
    got = f16_rne(np.array([c[0] for c in cases], np.float32)).view(np.uint16)
    assert [int(v) for v in got] == [c[1] for c in cases], [hex(v) for v in got]
    assert np.isnan(f16_rne(np.array([np.nan], np.float32))[0])
    # round-trip: every finite binary16 value is a binary32 value and maps to itself
    h = np.arange(0, 0x7C00, dtype=np.uint16).view(np.float16)
    assert np.array_equal(f16_rne(h.astype(np.float32)).view(np.uint16), h.view(np.uint16))


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
