"""LARS (Eq. lars) as a plain reference (test infrastructure only; see the
package docstring).

Eq. (lars) gives layer l the learning rate
    lambda_l = gamma * eta * ||w_l|| / (||g_l|| + eps * ||w_l||)
with gamma a coefficient, eta the global learning rate and eps the weight
decay. The paper computes these rates (and measures that computation); the
step that uses them is the one of the LARS method it cites:
    D = g + eps * w,   b = mu * b + lambda * D,   w = w - b
(without momentum: w = w - lambda * D).

Readings (each also listed with the design notes):
  * a layer is one tensor of the parameter list;
  * norms are Euclidean, in double: the squares of the binary32 values are
    exact in double, their sum is rounded once (math.fsum), then the square
    root; the rate is (gamma * eta * ||w||) / (||g|| + eps * ||w||) in double;
  * the equation is taken as printed wherever its denominator is positive:
    ||w|| = 0 < ||g|| gives rate 0, ||g|| = 0 < ||w|| gives gamma * eta / eps;
  * eps >= 0 (a weight decay). The denominator ||g|| + eps ||w|| is then zero
    only when g = 0 and eps w = 0 on the whole layer (0/0, or ||w|| / 0 with
    eps = 0), where the equation is undefined; the rate is read as 0 there.
    D = g + eps w is then zero at every position, so any finite rate gives
    the same step;
  * the step is binary32, one rounding per operation, with lambda rounded to
    binary32 once: D = g + eps * w, U = lambda * D, b = mu * b + U, w = w - U
    (or w = w - b with momentum), b starting at 0;
  * with sparse gradients, g is the dense sum of the workers' lists (Alg. 2),
    every position of every layer is updated (the weight-decay term touches
    untouched positions too).
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence, Tuple

import numpy as np


def layer_norm(v) -> float:
    v = np.ascontiguousarray(v, dtype=np.float32).astype(np.float64).ravel()
    return math.sqrt(math.fsum((v * v).tolist()))


def lars_rate(nw: float, ng: float, gamma: float, eta: float, eps: float) -> float:
    if eps < 0.0:
        raise ValueError("eps (the weight decay) must be >= 0")
    den = ng + eps * nw
    if den > 0.0:
        return (gamma * eta * nw) / den
    return 0.0


def lars_rates(ws: Sequence[np.ndarray], gs: Sequence[np.ndarray], gamma: float, eta: float,
               eps: float) -> np.ndarray:
    """Per-layer rates (float64), one per tensor."""
    return np.array([lars_rate(layer_norm(w), layer_norm(g), gamma, eta, eps)
                     for w, g in zip(ws, gs)], dtype=np.float64)


def lars_step(ws: Sequence[np.ndarray], bs: Optional[Sequence[np.ndarray]],
              gs: Sequence[np.ndarray], rates: np.ndarray, eps: float, mu: float
              ) -> Tuple[List[np.ndarray], Optional[List[np.ndarray]]]:
    """The binary32 step with the given per-layer rates. Returns new copies."""
    e32, m32 = np.float32(eps), np.float32(mu)
    w_out, b_out = [], ([] if bs is not None else None)
    for t, (w, g) in enumerate(zip(ws, gs)):
        w = np.array(w, dtype=np.float32, copy=True).ravel()
        g = np.ascontiguousarray(g, dtype=np.float32).ravel()
        lam = np.float32(rates[t])
        D = g + e32 * w
        U = lam * D
        if bs is not None:
            b = np.array(bs[t], dtype=np.float32, copy=True).ravel()
            b = m32 * b + U
            w = w - b
            b_out.append(b)
        else:
            w = w - U
        w_out.append(w)
    return w_out, b_out


def lars_update(ws, bs, gs, gamma: float, eta: float, eps: float, mu: float):
    """Rates from (w, g), then the step. Returns (w', b', rates)."""
    rates = lars_rates(ws, gs, gamma, eta, eps)
    w2, b2 = lars_step(ws, bs, gs, rates, eps, mu)
    return w2, b2, rates
