"""Helpers shared by the GPU parity tests (inputs to the device, comparisons,
exact selection properties)."""
from __future__ import annotations

import sys
from typing import Sequence

import numpy as np
import pytest

F32 = np.float32


def announce(msg: str) -> None:
    """Name the case on the real stderr before a GPU step (survives a crash
    of the process, unlike pytest's captured output)."""
    sys.__stderr__.write(f"[gpu-case] {msg}\n")
    sys.__stderr__.flush()


def need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a GPU")
    return torch.device("cuda:0")


def bits(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def to_dev(arrs: Sequence[np.ndarray], dev):
    import torch
    return [torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32).ravel()).to(dev)
            for a in arrs]


def to_host(ts) -> list:
    return [t.detach().cpu().numpy() for t in ts]


def assert_bitwise(a, b, what: str) -> None:
    a, b = np.asarray(a), np.asarray(b)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    if a.dtype == np.float32:
        bad = np.nonzero(bits(a) != bits(b))[0]
    else:
        bad = np.nonzero(a != b)[0]
    assert bad.size == 0, f"{what}: {bad.size} mismatches, first at {bad[:5].tolist()}: " \
                          f"{a[bad[:5]].tolist()} vs {b[bad[:5]].tolist()}"


def check_selection(x: np.ndarray, idx: np.ndarray, val: np.ndarray, r_out: np.ndarray,
                    k: int, base: int = 0) -> None:
    """Exact check of one selection group without sorting.

    With |S| = k, every selected magnitude >= every unselected one, and the
    selected members of the boundary magnitude class forming a prefix in
    position order, S is exactly the first k positions in the order
    (|x| descending, position ascending). x must be NaN-free.
    """
    n = x.size
    assert not np.isnan(x).any()
    loc = idx.astype(np.int64) - base
    assert loc.size == k, (loc.size, k)
    if k == 0:
        assert_bitwise(r_out, x, "residual")
        return
    assert loc.min() >= 0 and loc.max() < n
    assert np.all(np.diff(loc) > 0), "indices not strictly ascending"
    assert_bitwise(val, x[loc], "val == x[idx]")
    mask = np.zeros(n, bool)
    mask[loc] = True
    assert np.all(bits(r_out[mask]) == 0), "selected residual entries must be +0.0"
    assert_bitwise(r_out[~mask], x[~mask], "unselected residual == x")
    a = np.abs(x)
    T = a[loc].min()
    if k < n:
        assert a[~mask].max() <= T, "an unselected magnitude exceeds a selected one"
    eq = np.nonzero(a == T)[0]
    sel_eq = mask[eq]
    assert not np.any(~sel_eq[:-1] & sel_eq[1:]), "ties not broken toward lower positions"
