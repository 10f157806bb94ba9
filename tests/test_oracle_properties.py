"""Property tests of the oracle (Hypothesis, CPU only): random small inputs,
each checked against a definition written independently of the oracle's
code, with Hypothesis shrinking any counterexample to a minimal one.

* top-k: the first k positions of a Python sort by (|x| descending,
  position ascending) (the exactly-k reading of the TopK definition, Sec.
  3.1), on values drawn with many ties, signed zeros, infinities and
  subnormals;
* sparsify with error feedback: x = fl32(g + r) (numpy binary32 add), the
  values are x at the indices bit for bit, the residual is x with +0 at the
  selected positions;
* the aggregate of Alg. 2 and the update of Eq. (1) on dyadic values (every
  sum exact in binary32), against float64 sums and the update written out;
* MSTopK (Alg. 1): exactly k positions, ascending; every position at or above
  the first threshold is taken, the rest is a window of the band between the
  thresholds, contiguous in band rank and starting at the offset the window
  word gives;
* the LARS rate of Eq. (lars) against the formula in exact rationals.
"""
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import oracle.lars as lars
import oracle.mstopk as mst

SETTINGS = settings(max_examples=200, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow])
ORC = None


def orc():
    global ORC
    if ORC is None:
        ORC = oracle.Oracle()
    return ORC


SPECIAL = [0.0, -0.0, 1.0, -1.0, 0.5, -0.5, 2.0, 3.0e-39, -3.0e-39, 1.0e-45, np.inf, -np.inf,
           7.25, -7.25]
values = st.one_of(st.sampled_from(SPECIAL),
                   st.floats(width=32, allow_nan=False, allow_infinity=True))


@st.composite
def vec_and_k(draw, max_n=48):
    x = np.array(draw(st.lists(values, min_size=0, max_size=max_n)), dtype=np.float32)
    k = draw(st.integers(0, x.size))
    return x, k


@SETTINGS
@given(vec_and_k())
def test_topk_is_the_sorted_prefix(xk):
    x, k = xk
    order = sorted(range(x.size), key=lambda i: (-abs(float(x[i])), i))
    want = np.array(sorted(order[:k]), dtype=np.int64)
    got = orc().topk_select(x, k)
    assert np.array_equal(got, want)


@SETTINGS
@given(st.data())
def test_sparsify_error_feedback_identity(data):
    n = data.draw(st.integers(1, 40))
    g = np.array(data.draw(st.lists(values, min_size=n, max_size=n)), dtype=np.float32)
    r = np.array(data.draw(st.lists(values, min_size=n, max_size=n)), dtype=np.float32)
    with np.errstate(invalid="ignore", over="ignore"):
        x = g + r                                    # one binary32 add per element
    if np.isnan(x).any():
        return                                       # inf + -inf: no order exists
    k = data.draw(st.integers(1, n))
    idx, val, r_out = orc().sparsify_flat(g, r, k)
    assert np.array_equal(idx, orc().topk_select(x, k).astype(np.int32))
    assert np.array_equal(val.view(np.uint32), x[idx].view(np.uint32))
    expect = x.copy()
    expect[idx] = np.float32(0.0)
    assert np.array_equal(r_out.view(np.uint32), expect.view(np.uint32))


@SETTINGS
@given(st.data())
def test_dyadic_aggregate_and_update(data):
    d = data.draw(st.integers(1, 64))
    P = data.draw(st.integers(1, 6))
    stride = data.draw(st.integers(0, 12))
    idx = np.zeros((P, stride), np.int32)
    val = np.zeros((P, stride), np.float32)
    nnz = np.zeros(P, np.int64)
    for p in range(P):
        m = data.draw(st.integers(0, stride))
        nnz[p] = m
        idx[p, :m] = sorted(data.draw(st.lists(st.integers(0, d - 1), min_size=m, max_size=m)))
        val[p, :m] = [v / 16 for v in data.draw(st.lists(st.integers(-64, 64), min_size=m,
                                                         max_size=m))]
    G = np.zeros(d)
    for p in range(P):
        for j in range(nnz[p]):
            G[idx[p, j]] += float(val[p, j])
    got = orc().aggregate(d, idx, val, nnz)
    assert np.array_equal(got.astype(np.float64), G)
    w = np.array([v / 8 for v in data.draw(st.lists(st.integers(-64, 64), min_size=d,
                                                   max_size=d))], np.float32)
    b = np.array([v / 8 for v in data.draw(st.lists(st.integers(-64, 64), min_size=d,
                                                   max_size=d))], np.float32)
    lr, mu, wd = 0.25, 0.5, 0.0625
    w2, b2 = orc().update(w, b, idx, val, nnz=nnz, lr=lr, mu=mu, wd=wd)
    D = G + wd * w.astype(np.float64)
    bb = mu * b.astype(np.float64) + D
    assert np.array_equal(b2.astype(np.float64), bb)
    assert np.array_equal(w2.astype(np.float64), w.astype(np.float64) - lr * bb)


@SETTINGS
@given(st.data())
def test_mstopk_structure(data):
    n = data.draw(st.integers(1, 60))
    x = np.array(data.draw(st.lists(st.one_of(st.sampled_from([0.0, -1.0, 1.0, 2.0, -0.5]),
                                              st.floats(-1e6, 1e6, width=32)),
                                    min_size=n, max_size=n)), dtype=np.float32)
    k = data.draw(st.integers(1, n))
    N = data.draw(st.integers(1, 30))
    word = data.draw(st.integers(0, 2**64 - 1))
    iota, vals, tr = mst.mstopk(x, k, N, word)
    a = np.abs(x).astype(np.float64)
    assert iota.size == k and np.all(np.diff(iota) > 0)
    assert np.array_equal(vals.view(np.uint32), x[iota].view(np.uint32))
    top = np.flatnonzero(a >= tr.thres1)
    assert set(top.tolist()) <= set(iota.tolist()) and top.size == tr.k1
    members = np.flatnonzero((a >= tr.thres2) & (a < tr.thres1))
    taken = sorted(set(iota.tolist()) - set(top.tolist()))
    take = k - tr.k1
    assert len(taken) == take and members.size == tr.band
    off = word % (members.size - take + 1)
    assert off == tr.rand and taken == members[off:off + take].tolist()


# norms of binary32 layers: 0, or between the smallest subnormal and far
# above any real layer's norm
norms = st.one_of(st.just(0.0), st.floats(1e-45, 1e30))


@SETTINGS
@given(norms, norms, st.floats(1e-6, 10), st.floats(1e-6, 10),
       st.one_of(st.just(0.0), st.floats(1e-12, 1)))   # eps: the weight decay
def test_lars_rate_formula(nw, ng, gamma, eta, eps):
    got = lars.lars_rate(nw, ng, gamma, eta, eps)
    den = Fraction(ng) + Fraction(eps) * Fraction(nw)
    if den == 0:
        assert got == 0.0
        return
    exact = Fraction(gamma) * Fraction(eta) * Fraction(nw) / den
    # the oracle evaluates the formula in double: a few roundings
    assert abs(Fraction(got) - exact) <= abs(exact) * Fraction(1, 2**49) + Fraction(1, 10**300)
