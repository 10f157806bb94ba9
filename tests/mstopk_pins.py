"""Pins for the MSTopK oracle (Alg. 1): checks against facts fixed by the
algorithm and by mathematics, not against the oracle's own formulas.

Each ``pin_*`` takes the oracle module (``oracle.mstopk`` or a deliberately
broken copy of it) and raises on a mismatch. Sources of truth:
  * hand-worked cases (tests/golden/mstopk_worked.json): the trial thresholds,
    counts, recorded thresholds and the result, derived by hand in exact
    dyadic arithmetic;
  * the mean as a rational: the exact sum of the binary32 magnitudes as a
    Fraction, rounded once to double, then divided by d;
  * reductions to the exact operator: when a trial count equals k exactly and
    the k largest magnitudes are separated from the rest, the result is the
    exact top-k set (numpy argpartition);
  * closed forms: equal magnitudes (a contiguous window of length k starting
    at the offset), k = d (every position);
  * set relations the algorithm implies on any input: |result| = k, every
    element at or above thres1 taken, nothing below thres2 taken, the band
    members taken form one run of the band in position order starting at the
    offset, k1 and k2 are the counts at thres1 and thres2, and the offset is
    window_word mod (band - (k - k1) + 1);
  * brute force over all offsets of a small band.
"""
from __future__ import annotations

import json
import math
import os
from fractions import Fraction

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "mstopk_worked.json")


def _num(v):
    return math.inf if v == "inf" else float(v)


def pin_ms_worked_examples(ms):
    cases = json.load(open(GOLDEN))["cases"]
    for c in cases:
        x = np.array(c["x"], np.float32)
        iota, val, tr = ms.mstopk(x, c["k"], c["n_search"], c["window_word"])
        assert [list(map(float, s[:2])) + [int(s[2])] for s in tr.steps] == \
            [[float(a), float(b), int(n)] for a, b, n in c["steps"]], c["name"]
        assert (tr.k1, tr.k2, tr.band) == (c["k1"], c["k2"], c["band"]), c["name"]
        assert tr.thres1 == _num(c["thres1"]) and tr.thres2 == _num(c["thres2"]), c["name"]
        assert iota.tolist() == c["iota"], (c["name"], iota.tolist())
        assert np.array_equal(val.view(np.uint32), x[c["iota"]].view(np.uint32)), c["name"]


def pin_ms_mean_is_rounded_exact_sum(ms):
    rng = np.random.default_rng(61)
    for d in (1, 7, 1000, 4099):
        # magnitudes over many binades, so a careless sum would round differently
        x = (rng.standard_normal(d) * np.exp2(rng.integers(-30, 30, d))).astype(np.float32)
        _, _, tr = ms.mstopk(x, max(1, d // 3), 1, 0)
        S = sum(Fraction(float(v)) for v in np.abs(x))
        assert tr.abar == float(S) / d, d
        assert tr.u == float(np.max(np.abs(x)))


def pin_ms_exact_when_separated(ms):
    rng = np.random.default_rng(62)
    d, k = 20_000, 150
    x = rng.uniform(-1, 1, d).astype(np.float32)
    top = rng.choice(d, k, replace=False)
    x[top] = (rng.uniform(5, 6, k) * rng.choice([-1, 1], k)).astype(np.float32)
    for n in (1, 5, 30):
        iota, val, tr = ms.mstopk(x, k, n, 99)
        assert tr.k1 == k
        assert np.array_equal(iota, np.sort(top)), n
        assert np.array_equal(iota, np.sort(np.argpartition(-np.abs(x), k - 1)[:k]))


def pin_ms_equal_magnitudes_window(ms):
    d, k = 50, 7
    x = np.where(np.arange(d) % 3 == 0, -0.75, 0.75).astype(np.float32)
    for w in (0, 1, 43, 44, 2 ** 63 + 5):
        iota, _, tr = ms.mstopk(x, k, 30, w)
        s = w % (d - k + 1)
        assert iota.tolist() == list(range(s, s + k)), w
        assert (tr.k1, tr.k2) == (0, d)


def pin_ms_k_equals_d(ms):
    rng = np.random.default_rng(63)
    x = rng.standard_normal(777).astype(np.float32)
    for n in (1, 2, 30):
        iota, val, _ = ms.mstopk(x, x.size, n, 5)
        assert iota.tolist() == list(range(x.size))
        assert np.array_equal(val.view(np.uint32), x.view(np.uint32))


def _check_relations(x, k, w, iota, tr):
    a = np.abs(x).astype(np.float64)
    d = x.size
    assert iota.size == k and np.all(np.diff(iota) > 0)
    assert tr.k1 <= k < tr.k2 or (tr.k2 == d and k == d) or tr.k1 == k
    above1 = np.flatnonzero(a >= tr.thres1)
    assert above1.size == tr.k1
    assert tr.k2 == np.count_nonzero(a >= tr.thres2)
    sel = np.zeros(d, bool)
    sel[iota] = True
    assert sel[above1].all()
    assert np.all(a[iota] >= tr.thres2)
    band = np.flatnonzero((a < tr.thres1) & (a >= tr.thres2))
    assert band.size == tr.band
    taken = np.flatnonzero(sel[band])
    assert taken.size == k - tr.k1
    if taken.size:
        assert taken[0] == tr.rand and np.all(np.diff(taken) == 1)
    assert tr.rand == w % (band.size - (k - tr.k1) + 1)
    # every trial threshold lies between the mean and the maximum, and the
    # counts do not grow with the threshold
    th = np.array([s[1] for s in tr.steps])
    nz = np.array([s[2] for s in tr.steps])
    assert np.all(th >= tr.abar) and np.all(th <= tr.u)
    order = np.argsort(th, kind="stable")
    assert np.all(np.diff(nz[order]) <= 0)


def pin_ms_set_relations(ms):
    rng = np.random.default_rng(64)
    for d, k, n in ((10_000, 10, 30), (10_000, 1, 30), (50_001, 5000, 7), (3000, 2999, 30),
                    (65_536, 66, 13), (5, 3, 1)):
        x = rng.standard_normal(d).astype(np.float32)
        x[rng.random(d) < 0.01] *= 100
        w = int(rng.integers(0, 2 ** 63))
        iota, val, tr = ms.mstopk(x, k, n, w)
        _check_relations(x, k, w, iota, tr)
        assert np.array_equal(val.view(np.uint32), x[iota].view(np.uint32))


def pin_ms_every_offset_small_band(ms):
    # ties at the boundary: a band of 12 equal magnitudes, 4 positions to
    # fill from it; the 9 possible offsets give the 9 runs of 4
    x = np.zeros(40, np.float32)
    x[:5] = 10.0
    band_pos = np.arange(10, 34, 2)
    x[band_pos] = -3.0
    seen = set()
    for w in range(30):
        iota, _, tr = ms.mstopk(x, 9, 30, w)
        assert iota[:5].tolist() == [0, 1, 2, 3, 4]
        run = iota[5:].tolist()
        s = w % 9
        assert run == band_pos[s:s + 4].tolist(), (w, run)
        seen.add(tuple(run))
    assert len(seen) == 9


def pin_ms_quality_normal(ms):
    # not a definition but a behaviour the paper reports: on gradient-like
    # data N = 30 rounds select nearly the exact top-k (overlap above 0.99)
    rng = np.random.default_rng(65)
    d, k = 200_000, 200
    x = rng.standard_normal(d).astype(np.float32)
    iota, _, _ = ms.mstopk(x, k, 30, 1)
    exact = np.argpartition(-np.abs(x), k - 1)[:k]
    assert np.intersect1d(iota, exact).size >= 0.99 * k


def pin_ms_sparsify_residual(ms):
    rng = np.random.default_rng(66)
    g = rng.standard_normal(5000).astype(np.float32)
    r = (rng.standard_normal(5000) * 0.5).astype(np.float32)
    idx, val, r_out, tr = ms.mstopk_sparsify(g, r, 50, 30, 3, index_base=100)
    x = (g.astype(np.float64) + r.astype(np.float64)).astype(np.float32)
    iota, v2, _ = ms.mstopk(x, 50, 30, 3)
    assert np.array_equal(idx, iota + 100) and np.array_equal(val.view(np.uint32), v2.view(np.uint32))
    expect = x.copy()
    expect[iota] = 0.0
    assert np.array_equal(r_out.view(np.uint32), expect.view(np.uint32))


def pin_ms_rejects_nonfinite(ms):
    for bad in (np.inf, -np.inf, np.nan):
        x = np.ones(10, np.float32)
        x[3] = bad
        try:
            ms.mstopk(x, 2, 30, 0)
        except ValueError:
            continue
        raise AssertionError(f"accepted {bad}")


ALL_MS_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_ms_")]
