"""MSTopK, the approximate top-k selector of Sec. 3.1 (Alg. 1), as a plain
float64 reference (test infrastructure only; see the package docstring).

What the algorithm computes, restated as definitions. With a = |x| (d
entries), abar their mean and u their maximum:

  * trial n = 1..N bisects the ratio interval [0, 1]: its ratio is the
    midpoint (2 p + 1) / 2^n of the interval the earlier trials left, p being
    the path taken so far (one bit per trial, 1 when that trial counted more
    than k elements and the search moved up, 0 when it moved down);
  * its threshold is t_n = abar + ratio_n (u - abar) and its count is
    c_n = #{i : a_i >= t_n};
  * the lower record (k1, thres1) is the largest count that does not exceed
    k and the threshold of the first trial that reached it; the upper record
    (k2, thres2) is the smallest count above k and the threshold of the first
    trial that reached it;
  * the result is every position with a >= thres1, plus k - k1 positions of
    the band thres2 <= a < thres1: the band members of rank offset ..
    offset + k - k1 - 1 in position order, the offset drawn at random.

Readings of points the algorithm leaves open (each also listed with the
design notes):
  * the mean is the correctly rounded double of the exact sum of the binary32
    magnitudes, divided by d in double (math.fsum gives that rounded sum);
  * thresholds and comparisons are in double; a binary32 magnitude is compared
    exactly after widening;
  * before any record the lower one is (0, +infinity) and the upper one
    (d, 0): a count of 0 or d adds nothing to a record, and the sets
    {a >= +inf} and {a >= 0} are exactly those counts (the printed start 0
    for thres1 would select every element whenever no trial count falls at
    or below k);
  * the random offset is uniform over 0 .. band - (k - k1) inclusive (the
    printed bound read as half-open); it is taken as window_word modulo
    (band - (k - k1) + 1), window_word being a 64-bit value the caller
    supplies;
  * the returned positions are sorted ascending (the algorithm concatenates
    two index lists), values are x at those positions;
  * non-finite inputs are rejected (the mean and the thresholds are then
    undefined); N is at most 53, so that every ratio is an exact double.
"""
from __future__ import annotations

import math
from typing import NamedTuple, Tuple

import numpy as np


class MsTrace(NamedTuple):
    abar: float
    u: float
    steps: tuple          # (ratio, thres, count) per trial
    k1: int
    k2: int
    thres1: float
    thres2: float
    band: int             # members of the band thres2 <= a < thres1
    rand: int             # offset of the window in the band


def _trials(asc: np.ndarray, abar: float, u: float, k: int, n_search: int) -> list:
    """The N trials of the bisection: (ratio, threshold, count) each. asc is
    a sorted ascending, so #{a >= t} = d - (number of entries below t)."""
    d = int(asc.size)
    out = []
    path = 0
    for n in range(1, n_search + 1):
        ratio = math.ldexp(2 * path + 1, -n)
        thres = abar + ratio * (u - abar)
        count = d - int(np.searchsorted(asc, thres, side="left"))
        out.append((ratio, thres, count))
        path = 2 * path + (1 if count > k else 0)
    return out


def _records(trials: list, k: int, d: int) -> Tuple[int, float, int, float]:
    """(k1, thres1, k2, thres2) from the trials: the largest count <= k and
    the smallest count > k, each with the threshold of the first trial that
    reached it; counts of 0 and d leave the start records (0, +inf) and
    (d, 0)."""
    low = [(c, t) for (_, t, c) in trials if 0 < c <= k]
    high = [(c, t) for (_, t, c) in trials if k < c < d]
    k1, thres1 = 0, math.inf
    if low:
        k1 = max(c for c, _ in low)
        thres1 = next(t for c, t in low if c == k1)
    k2, thres2 = d, 0.0
    if high:
        k2 = min(c for c, _ in high)
        thres2 = next(t for c, t in high if c == k2)
    return k1, thres1, k2, thres2


def mstopk(x, k: int, n_search: int, window_word: int) -> Tuple[np.ndarray, np.ndarray, MsTrace]:
    """Alg. 1 on a flat binary32 vector. Returns (positions ascending, values
    x[positions], trace)."""
    x = np.ascontiguousarray(x, dtype=np.float32).ravel()
    d = int(x.size)
    if not 1 <= k <= d:
        raise ValueError("k outside [1, d]")
    if not 1 <= n_search <= 53:
        raise ValueError("n_search outside [1, 53]")
    a = np.abs(x).astype(np.float64)
    if not np.all(np.isfinite(a)):
        raise ValueError("non-finite input")
    abar = math.fsum(a.tolist()) / d
    u = float(a.max())
    trials = _trials(np.sort(a), abar, u, k, n_search)
    k1, thres1, k2, thres2 = _records(trials, k, d)

    top = a >= thres1
    band = (a >= thres2) & ~top
    nband = int(np.count_nonzero(band))
    take = k - k1
    offset = int(window_word) % (nband - take + 1)
    rank = np.cumsum(band) - 1          # rank of each band member in position order
    window = band & (rank >= offset) & (rank < offset + take)
    iota = np.flatnonzero(top | window).astype(np.int64)
    trace = MsTrace(abar, u, tuple(trials), k1, k2, thres1, thres2, nband, offset)
    return iota, x[iota], trace


def mstopk_sparsify(g, r, k: int, n_search: int, window_word: int, index_base: int = 0):
    """Error-feedback form: x = fl32(g + r); select with Alg. 1; the residual
    becomes x with the selected positions set to +0. Returns (idx int32,
    val float32, new residual, trace)."""
    g = np.ascontiguousarray(g, dtype=np.float32).ravel()
    r = np.ascontiguousarray(r, dtype=np.float32).ravel()
    x = g + r
    iota, val, trace = mstopk(x, k, n_search, window_word)
    r_out = x.copy()
    r_out[iota] = np.float32(0.0)
    return (iota + index_base).astype(np.int32), val, r_out, trace
