"""MSTopK, the approximate top-k selector of Alg. 1, as a plain float64
reference (test infrastructure only; see the package docstring).

Alg. 1 takes a = |x|, its mean and its maximum u, and bisects a ratio in
[0, 1] for N rounds: the trial threshold is mean + ratio * (u - mean); a count
of elements at or above it that does not exceed k moves the upper end r down
(and records the largest such count k1 with its threshold thres1), a larger
count moves the lower end l up (and records the smallest such count k2 with
thres2). The result is every element at or above thres1 plus a window of
k - k1 consecutive elements, in position order, of the band
thres2 <= a < thres1, the window starting at a random offset.

Readings of points the algorithm leaves open (each also listed with the
design notes):
  * the mean is the correctly rounded double of the exact sum of the binary32
    magnitudes, divided by d in double: math.fsum gives that rounded sum;
  * thresholds and comparisons are in double; a binary32 magnitude is compared
    exactly after widening;
  * thres1 starts at +infinity, so that "k1 = 0" and "thres1" describe the
    same (empty) set; the printed start value 0 would select every element
    whenever no trial count falls at or below k. thres2 starts at 0, which
    matches k2 = d;
  * the random offset is uniform over 0 .. len(band) - (k - k1) inclusive
    (the printed bound read as half-open); it is taken as window_word modulo
    (len(band) - (k - k1) + 1), window_word being a 64-bit value the caller
    supplies;
  * the returned positions are sorted ascending (the concatenation in the
    algorithm is not), values are x at those positions;
  * non-finite inputs are rejected (the mean and the thresholds are then
    undefined).
"""
from __future__ import annotations

import math
from typing import NamedTuple, Tuple

import numpy as np


class MsTrace(NamedTuple):
    abar: float
    u: float
    steps: tuple          # (ratio, thres, nnz) per round
    k1: int
    k2: int
    thres1: float
    thres2: float
    band: int             # len of the band thres2 <= a < thres1
    rand: int


def mstopk(x, k: int, n_search: int, window_word: int) -> Tuple[np.ndarray, np.ndarray, MsTrace]:
    """Alg. 1 on a flat binary32 vector. Returns (positions ascending, values
    x[positions], trace)."""
    x = np.ascontiguousarray(x, dtype=np.float32).ravel()
    d = int(x.size)
    if not 1 <= k <= d:
        raise ValueError("k outside [1, d]")
    if n_search < 1:
        raise ValueError("n_search < 1")
    a = np.abs(x).astype(np.float64)
    if not np.all(np.isfinite(a)):
        raise ValueError("non-finite input")
    abar = math.fsum(a.tolist()) / d
    u = float(a.max())
    l, r = 0.0, 1.0
    k1, k2 = 0, d
    thres1, thres2 = math.inf, 0.0
    steps = []
    for _ in range(n_search):
        ratio = l + (r - l) / 2
        thres = abar + ratio * (u - abar)
        nnz = int(np.count_nonzero(a >= thres))
        steps.append((ratio, thres, nnz))
        if nnz <= k:
            r = ratio
            if nnz > k1:
                k1 = nnz
                thres1 = thres
        elif nnz > k:
            l = ratio
            if nnz < k2:
                k2 = nnz
                thres2 = thres
    iota1 = np.flatnonzero(a >= thres1)
    iota2 = np.flatnonzero((a < thres1) & (a >= thres2))
    take = k - k1
    rand = int(window_word) % (len(iota2) - take + 1)
    iota = np.sort(np.concatenate([iota1, iota2[rand:rand + take]])).astype(np.int64)
    trace = MsTrace(abar, u, tuple(steps), k1, k2, thres1, thres2, int(len(iota2)), rand)
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
