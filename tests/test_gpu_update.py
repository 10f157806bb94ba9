"""GPU parity: tkef sparse aggregate + SGD update (through the C ABI) against
the CPU oracle.

The oracle sums each position's contributions in worker order. A binary32
sum of one or two terms does not depend on order, so every position with at
most two contributions must match bit for bit; positions with three or more
must agree within |w_gpu - w_ref| <= 1e-6 (|w_ref| + S), S = lr (sum |v| +
wd |w| + mu |b|), a bound that covers any summation order of those few
terms. On dyadic inputs every order is exact, so those runs match bit for
bit everywhere.
"""
import zlib

import numpy as np
import pytest

import gen
import oracle
import paper_2010_10458_amd as tk
from gpu_common import announce, assert_bitwise, bits, need_gpu, to_dev, to_host

pytestmark = pytest.mark.gpu

ORC = None


def orc():
    global ORC
    if ORC is None:
        ORC = oracle.Oracle()
    return ORC


def gpu_update(sizes, w_host, b_host, idx, val, lr, mu, wd, nnz=None, views=None):
    import torch
    dev = need_gpu()
    w = to_dev(w_host, dev)
    b = to_dev(b_host, dev) if b_host is not None else None
    it = torch.from_numpy(np.ascontiguousarray(idx, np.int32)).to(dev)
    vt = torch.from_numpy(np.ascontiguousarray(val, np.float32)).to(dev)
    nt = torch.from_numpy(np.asarray(nnz, np.int32)).to(dev) if nnz is not None else None
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    P, stride = idx.shape
    plan = tk.UpdatePlan(sizes, P=P, stride=stride)
    plan.bind(w, b)
    plan.execute(it, vt, lr=lr, mu=mu, wd=wd, nnz=nt, status=status)
    torch.cuda.synchronize()
    return (to_host(w), to_host(b) if b is not None else None, int(status.item()))


def compare(sizes, w0, b0, idx, val, lr, mu, wd, nnz=None, exact=False, label="", runner=None):
    """runner(sizes, w0, b0, idx, val, lr, mu, wd, nnz) -> (w, b, status):
    the GPU call under test (default: an UpdatePlan over the gathered
    lists)."""
    announce(f"update {label} P={idx.shape[0]} stride={idx.shape[1]} mu={mu} wd={wd}")
    w_gpu, b_gpu, status = (runner or gpu_update)(sizes, w0, b0, idx, val, lr, mu, wd, nnz)
    assert status == 0
    w_ref, b_ref = orc().update(gen.concat(w0), None if b0 is None else gen.concat(b0), idx, val,
                                nnz=None if nnz is None else np.asarray(nnz, np.int64),
                                lr=lr, mu=mu, wd=wd)
    wg = gen.concat(w_gpu)
    bg = gen.concat(b_gpu) if b_gpu is not None else None
    if exact:
        assert_bitwise(wg, w_ref, "w")
        if b_ref is not None:
            assert_bitwise(bg, b_ref, "b")
        return wg, bg
    d = wg.size
    P, stride = idx.shape
    nn = np.full(P, stride) if nnz is None else np.clip(np.asarray(nnz), 0, stride)
    flat_i = np.concatenate([idx[p, :nn[p]] for p in range(P)]).astype(np.int64)
    flat_v = np.concatenate([val[p, :nn[p]] for p in range(P)]).astype(np.float64)
    cnt = np.bincount(flat_i, minlength=d)
    A = np.zeros(d)
    np.add.at(A, flat_i, np.abs(flat_v))
    le2 = cnt <= 2
    assert_bitwise(wg[le2], w_ref[le2], "w (<= 2 contributions)")
    w0c = np.abs(gen.concat(w0)).astype(np.float64)
    b0c = np.abs(gen.concat(b0)).astype(np.float64) if b0 is not None else 0.0
    S = lr * (A + wd * w0c + mu * b0c)
    assert np.all(np.abs(wg.astype(np.float64) - w_ref) <= 1e-6 * (np.abs(w_ref) + S))
    if b_ref is not None:
        assert_bitwise(bg[le2], b_ref[le2], "b (<= 2 contributions)")
        Sb = A + wd * w0c + mu * b0c
        assert np.all(np.abs(bg.astype(np.float64) - b_ref) <= 1e-6 * (np.abs(b_ref) + Sb))
    return wg, bg


def _lists(rng, d, P, k, std=1e-2, sorted_=True, overlap=False):
    idx = np.empty((P, k), np.int32)
    pool = rng.choice(d, size=min(d, 2 * k), replace=False) if overlap else None
    for p in range(P):
        idx[p] = np.sort(rng.choice(pool if overlap else d, size=k, replace=False))
    val = (rng.standard_normal((P, k)) * std).astype(np.float32)
    return idx, val


SIZE_SETS = {
    "single": [100_003],
    "ragged": [1, 5, 64, 8193, 100, 30_000, 0, 17, 16_384, 3],
    "tiny": [3],
}


@pytest.mark.parametrize("sizes_name", sorted(SIZE_SETS))
@pytest.mark.parametrize("mode", ["plain", "wd", "momentum"])
def test_update_small(sizes_name, mode):
    sizes = SIZE_SETS[sizes_name]
    d = sum(sizes)
    rng = np.random.default_rng(zlib.crc32(f"{sizes_name}/{mode}".encode()))
    w0 = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    b0 = [(rng.standard_normal(n) * 0.01).astype(np.float32) for n in sizes] if mode == "momentum" else None
    mu, wd = {"plain": (0.0, 0.0), "wd": (0.0, 5e-5), "momentum": (0.9, 5e-5)}[mode]
    for P in (1, 3, 40):
        k = max(1, min(d, d // 50 + 1))
        idx, val = _lists(rng, d, P, k, overlap=(P > 1))
        compare(sizes, w0, b0, idx, val, 0.1, mu, wd, label=f"{sizes_name} {mode}")


def test_update_dyadic_bit_exact():
    rng = np.random.default_rng(31)
    sizes = [8192 * 3 + 11, 517, 4096]
    d = sum(sizes)
    w0 = [(rng.integers(-4095, 4096, n) / 256.0).astype(np.float32) for n in sizes]
    b0 = [np.zeros(n, np.float32) for n in sizes]
    P, k = 24, 3000
    idx = np.empty((P, k), np.int32)
    pool = rng.choice(d, 4000, replace=False)
    for p in range(P):
        idx[p] = np.sort(rng.choice(pool, k, replace=False))
    e = rng.integers(-8, -3, (P, k)).astype(np.float64)
    val = (np.exp2(e) * np.where(rng.random((P, k)) < 0.5, -1, 1)).astype(np.float32)
    compare(sizes, w0, b0, idx, val, 0.25, 0.5, 0.0625, exact=True, label="dyadic momentum")
    compare(sizes, w0, None, idx, val, 0.25, 0.0, 0.0, exact=True, label="dyadic plain")


@pytest.mark.parametrize("P,stride", [(257, 150), (1000, 40), (65535, 2)])
def test_update_many_workers(P, stride):
    """More workers than one update workgroup takes at a time (256): several
    worker batches per tile, up to the largest P the plan accepts."""
    rng = np.random.default_rng(34 + P)
    sizes = [30_011, 4096, 17]
    d = sum(sizes)
    w0 = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    b0 = [np.zeros(n, np.float32) for n in sizes]
    idx = np.sort(rng.integers(0, d, (P, stride)), axis=1).astype(np.int32)
    val = (rng.standard_normal((P, stride)) * 1e-2).astype(np.float32)
    nnz = rng.integers(0, stride + 1, P).astype(np.int32)
    compare(sizes, w0, b0, idx, val, 0.1, 0.9, 5e-5, nnz=nnz, label=f"P={P}")
    compare(sizes, w0, None, idx, val, 0.5, 0.0, 0.0, nnz=nnz, label=f"P={P} plain")


def test_update_duplicates_ragged_nnz_and_empty():
    rng = np.random.default_rng(32)
    sizes = [20_000, 333]
    d = sum(sizes)
    w0 = [(rng.standard_normal(n)).astype(np.float32) for n in sizes]
    P, stride = 5, 400
    idx = np.sort(rng.integers(0, d, (P, stride)), axis=1).astype(np.int32)   # repeats allowed
    idx[2, :50] = 7                                                           # many repeats
    idx[2] = np.sort(idx[2])
    val = (rng.standard_normal((P, stride)) * 0.1).astype(np.float32)
    nnz = [400, 0, 123, 1, 399]
    compare(sizes, w0, None, idx, val, 0.5, 0.0, 0.0, nnz=nnz, label="dups ragged plain")
    b0 = [np.zeros(n, np.float32) for n in sizes]
    compare(sizes, w0, b0, idx, val, 0.5, 0.9, 1e-4, nnz=nnz, label="dups ragged momentum")
    empty_i = np.zeros((3, 0), np.int32)
    empty_v = np.zeros((3, 0), np.float32)
    compare(sizes, w0, None, empty_i, empty_v, 0.5, 0.0, 0.0, exact=True, label="empty plain")
    compare(sizes, w0, b0, empty_i, empty_v, 0.5, 0.9, 1e-4, exact=True, label="empty momentum")


def test_update_bad_lists_flag_status():
    """Unsorted and out-of-range lists are reported in the status word and
    handled without touching memory outside the buffers (the result for
    such input is unspecified)."""
    rng = np.random.default_rng(33)
    sizes = [50_000]
    w0 = [np.ones(50_000, np.float32)]
    idx = np.sort(rng.integers(0, 50_000, (2, 100)), axis=1).astype(np.int32)
    idx[0] = idx[0][::-1]                 # descending list
    val = np.ones((2, 100), np.float32)
    announce("update unsorted list")
    _, _, status = gpu_update(sizes, w0, None, idx, val, 0.1, 0.0, 0.0)
    assert status & tk.STATUS_UNSORTED
    idx2 = np.sort(rng.integers(0, 50_000, (2, 100)), axis=1).astype(np.int32)
    idx2[1, -1] = 50_000 + 5              # past the end
    idx2[0, 0] = -3
    announce("update out-of-range index")
    w, _, status = gpu_update(sizes, w0, None, idx2, val, 0.1, 0.0, 0.0)
    assert status & tk.STATUS_INDEX_RANGE


def test_c1_plain_update_after_sparsify():
    """The 1 M workload: sparsify, then a one-worker plain update (lr = 0.1)
    of N(0, 0.1) parameters with the selected pairs; bit-exact."""
    import torch
    dev = need_gpu()
    n = gen.C1_D
    g = gen.flat_normal(n, config=1)
    w0 = gen.params_like([n], config=1)
    announce("c1 sparsify + plain update")
    gt, rt, wt = to_dev([g], dev), to_dev([np.zeros(n, np.float32)], dev), to_dev(w0, dev)
    sp = tk.SparsifyPlan([n], rho=0.001)
    sp.bind(gt, rt)
    idx, val = sp.execute()
    up = tk.UpdatePlan([n], P=1, stride=sp.k_total)
    up.bind(wt)
    up.execute(idx, val, lr=0.1)
    torch.cuda.synchronize()
    oi, ov, _, _ = orc().sparsify([g], [np.zeros(n, np.float32)], rho=0.001)
    w_ref, _ = orc().update(w0[0], None, oi, ov, lr=0.1)
    assert_bitwise(idx.cpu().numpy(), oi, "idx")
    assert_bitwise(wt[0].cpu().numpy(), w_ref, "w")


def test_c5_resnet50_p128_momentum_3_steps():
    """P = 128 workers x 25,600 pairs into ResNet-50-shaped parameters with
    momentum 0.9 and weight decay 5e-5, lr 0.1, three steps (fresh lists each
    step, parameters and momentum carried on the GPU)."""
    import torch
    dev = need_gpu()
    sizes = gen.numels(gen.resnet50_shapes())
    d = sum(sizes)
    w_host = gen.params_like(sizes, config=5)
    b_host = [np.zeros(n, np.float32) for n in sizes]
    w = to_dev(w_host, dev)
    b = to_dev(b_host, dev)
    P, k = 128, 25_600
    plan = tk.UpdatePlan(sizes, P=P, stride=k)
    plan.bind(w, b)
    w_ref, b_ref = gen.concat(w_host), gen.concat(b_host)
    for step in range(3):
        announce(f"c5 step {step}")
        idx, val = gen.sparse_lists(d, P, k, step=step)
        it = torch.from_numpy(idx).to(dev)
        vt = torch.from_numpy(val).to(dev)
        plan.execute(it, vt, lr=0.1, mu=0.9, wd=5e-5)
        torch.cuda.synchronize()
        w_prev, b_prev = w_ref, b_ref
        w_ref, b_ref = orc().update(w_prev, b_prev, idx, val, lr=0.1, mu=0.9, wd=5e-5)
        wg, bg = gen.concat(to_host(w)), gen.concat(to_host(b))
        cnt = np.bincount(idx.ravel(), minlength=d)
        A = np.zeros(d)
        np.add.at(A, idx.ravel(), np.abs(val.ravel().astype(np.float64)))
        S = 0.1 * (A + 5e-5 * np.abs(w_prev) + 0.9 * np.abs(b_prev))
        # every step starts from the GPU's own state, so positions with at
        # most two contributions in this step match bit for bit on each step
        le2 = cnt <= 2
        assert_bitwise(wg[le2], w_ref[le2], f"w (<= 2 contributions, step {step})")
        assert_bitwise(bg[le2], b_ref[le2], f"b (<= 2 contributions, step {step})")
        assert np.all(np.abs(wg.astype(np.float64) - w_ref) <= 1e-6 * (np.abs(w_ref) + S))
        assert np.all(np.abs(bg.astype(np.float64) - b_ref) <= 1e-6 * (np.abs(b_ref) + S / 0.1))
        # carry the GPU state forward so later steps test one step at a time
        w_ref, b_ref = wg, bg


@pytest.mark.parametrize("mu,wd", [(0.0, 0.0), (0.9, 5e-5)])
def test_update_worker_order_permuted(mu, wd):
    """The same 24 overlapping lists in a permuted worker order: each
    position's sum then runs in another order, so the result must agree with
    the oracle's original-order result within the bound that covers any
    order, and bit for bit where a position has at most two contributions."""
    rng = np.random.default_rng(808 + int(mu * 10))
    sizes = [100_003, 4097]
    d = sum(sizes)
    P, k = 24, 3000
    idx, val = _lists(rng, d, P, k, std=0.1, overlap=True)
    perm = rng.permutation(P)
    assert not np.array_equal(perm, np.arange(P))
    w0 = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    b0 = [(rng.standard_normal(n) * 0.01).astype(np.float32) for n in sizes] if mu else None
    lr = 0.05
    announce(f"update worker order permuted mu={mu}")
    w_gpu, b_gpu, status = gpu_update(sizes, w0, b0, idx[perm], val[perm], lr, mu, wd)
    assert status == 0
    w_ref, b_ref = orc().update(gen.concat(w0), None if b0 is None else gen.concat(b0), idx, val,
                                lr=lr, mu=mu, wd=wd)
    wg = gen.concat(w_gpu)
    cnt = np.bincount(idx.ravel().astype(np.int64), minlength=d)
    assert (cnt >= 3).sum() > 1000  # the overlap makes many positions order-sensitive
    le2 = cnt <= 2
    assert_bitwise(wg[le2], w_ref[le2], "w (<= 2 contributions)")
    A = np.zeros(d)
    np.add.at(A, idx.ravel().astype(np.int64), np.abs(val.ravel().astype(np.float64)))
    w0c = np.abs(gen.concat(w0)).astype(np.float64)
    b0c = np.abs(gen.concat(b0)).astype(np.float64) if b0 is not None else 0.0
    S = lr * (A + wd * w0c + mu * b0c)
    assert np.all(np.abs(wg.astype(np.float64) - w_ref) <= 1e-6 * (np.abs(w_ref) + S))
    if b_ref is not None:
        bg = gen.concat(b_gpu)
        assert_bitwise(bg[le2], b_ref[le2], "b (<= 2 contributions)")
        Sb = A + wd * w0c + mu * b0c
        assert np.all(np.abs(bg.astype(np.float64) - b_ref) <= 1e-6 * (np.abs(b_ref) + Sb))
