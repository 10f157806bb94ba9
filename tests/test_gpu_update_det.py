"""GPU parity of the deterministic update mode (UpdatePlan(deterministic=True),
tkef_update_plan_set_deterministic) through the C ABI.

In this mode every position's entries are added in worker order, then list
order, from +0 (the order of Alg. 2's loop over the gathered lists), which
is the order in which the C oracle adds them. G is then the oracle's G bit
for bit, and so is every result computed from it with the same binary32
operations: the plain, weight-decay and momentum updates and the dense
aggregate match bit for bit at every position, whatever the number of
contributions per position. The cases cover many contributions per
position (heavy overlap, repeats within and across workers), more than one
chunk of entries per tile and more than one batch of workers (P > 256),
ragged and zero counts, binary16 values, and repeated calls.
"""
import numpy as np
import pytest

import gen
import oracle
import oracle.lars as lars
import paper_2010_10458_amd as tk
from gpu_common import announce, assert_bitwise, bits, need_gpu, to_dev, to_host

pytestmark = pytest.mark.gpu

ORC = None


def orc():
    global ORC
    if ORC is None:
        ORC = oracle.Oracle()
    return ORC


def _tensors(idx, val, nnz, dev):
    import torch
    it = torch.from_numpy(np.ascontiguousarray(idx, np.int32)).to(dev)
    vt = torch.from_numpy(np.ascontiguousarray(val)).to(dev)
    nt = torch.from_numpy(np.asarray(nnz, np.int32)).to(dev) if nnz is not None else None
    return it, vt, nt


def det_update_vs_oracle(sizes, w0, b0, idx, val, lr, mu, wd, nnz=None, label="",
                         val_dtype=None):
    """One deterministic update on the GPU; w (and b) bit for bit against
    the oracle at every position."""
    import torch
    dev = need_gpu()
    announce(f"det update {label} P={idx.shape[0]} stride={idx.shape[1]} mu={mu} wd={wd}")
    w = to_dev(w0, dev)
    b = to_dev(b0, dev) if b0 is not None else None
    it, vt, nt = _tensors(idx, val, nnz, dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    P, stride = idx.shape
    plan = tk.UpdatePlan(sizes, P=P, stride=stride, val_dtype=val_dtype or torch.float32,
                         deterministic=True)
    plan.bind(w, b)
    plan.execute(it, vt, lr=lr, mu=mu, wd=wd, nnz=nt, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    w_ref, b_ref = orc().update(gen.concat(w0), None if b0 is None else gen.concat(b0), idx,
                                np.asarray(val).astype(np.float32),
                                nnz=None if nnz is None else np.asarray(nnz, np.int64),
                                lr=lr, mu=mu, wd=wd)
    assert_bitwise(gen.concat(to_host(w)), w_ref, f"w ({label})")
    if b is not None:
        assert_bitwise(gen.concat(to_host(b)), b_ref, f"b ({label})")


def _overlapping_lists(rng, d, P, k, pool_size, std=1e-2):
    """Ascending lists drawn from a small common pool: many positions get
    contributions from many workers."""
    pool = rng.choice(d, size=pool_size, replace=False)
    idx = np.stack([np.sort(rng.choice(pool, size=k, replace=False)) for _ in range(P)])
    val = (rng.standard_normal((P, k)) * std).astype(np.float32)
    return idx.astype(np.int32), val


@pytest.mark.parametrize("mode", ["plain", "wd", "momentum"])
def test_det_overlap_bitwise(mode):
    rng = np.random.default_rng({"plain": 61, "wd": 62, "momentum": 63}[mode])
    sizes = [1, 5, 64, 8193, 100, 30_000, 0, 17, 16_384, 3]
    d = sum(sizes)
    w0 = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    b0 = [(rng.standard_normal(n) * 0.01).astype(np.float32) for n in sizes] if mode == "momentum" else None
    mu, wd = {"plain": (0.0, 0.0), "wd": (0.0, 5e-5), "momentum": (0.9, 5e-5)}[mode]
    for P, k, pool in ((3, 900, 1000), (40, 1500, 2000), (128, 600, 700)):
        idx, val = _overlapping_lists(rng, d, P, k, pool)
        det_update_vs_oracle(sizes, w0, b0, idx, val, 0.1, mu, wd, label=f"overlap {mode} P={P}")


def test_det_many_chunks_and_worker_batches():
    """P = 300 workers (two batches of 256), 2,000 entries each over three
    tiles: tens of chunks of 1,024 entries per tile."""
    rng = np.random.default_rng(64)
    sizes = [8192 * 3]
    d = sizes[0]
    w0 = [(rng.standard_normal(d) * 0.1).astype(np.float32)]
    b0 = [np.zeros(d, np.float32)]
    idx, val = _overlapping_lists(rng, d, 300, 2000, 6000)
    det_update_vs_oracle(sizes, w0, b0, idx, val, 0.1, 0.9, 5e-5, label="300 workers")


def test_det_largest_worker_count():
    """P = 65,535 workers of two entries each (256 worker batches per tile)."""
    rng = np.random.default_rng(69)
    sizes = [40_000, 123]
    d = sum(sizes)
    w0 = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    b0 = [np.zeros(n, np.float32) for n in sizes]
    idx = np.sort(rng.integers(0, d, (65_535, 2)), axis=1).astype(np.int32)
    val = (rng.standard_normal((65_535, 2)) * 1e-2).astype(np.float32)
    det_update_vs_oracle(sizes, w0, b0, idx, val, 0.1, 0.9, 5e-5, label="P=65535")


def test_det_repeats_hot_position_ragged_nnz_empty():
    """Repeats within a worker (one worker names position 7 fifty times),
    forty workers all naming positions 7 and 8 (over a thousand entries of
    one position in a chunk), zero and partial counts, empty lists."""
    rng = np.random.default_rng(65)
    sizes = [20_000, 333]
    d = sum(sizes)
    w0 = [rng.standard_normal(n).astype(np.float32) for n in sizes]
    b0 = [np.zeros(n, np.float32) for n in sizes]
    P, stride = 45, 400
    idx = np.sort(rng.integers(0, d, (P, stride)), axis=1).astype(np.int32)
    idx[2, :50] = 7
    for p in range(5, 45):
        idx[p, :30] = 7
        idx[p, 30:60] = 8
    idx = np.sort(idx, axis=1)
    val = (rng.standard_normal((P, stride)) * 0.1).astype(np.float32)
    nnz = [400, 0, 123, 1, 399] + [400] * 40
    det_update_vs_oracle(sizes, w0, None, idx, val, 0.5, 0.0, 0.0, nnz=nnz, label="dups plain")
    det_update_vs_oracle(sizes, w0, b0, idx, val, 0.5, 0.9, 1e-4, nnz=nnz, label="dups momentum")
    empty_i = np.zeros((3, 0), np.int32)
    empty_v = np.zeros((3, 0), np.float32)
    det_update_vs_oracle(sizes, w0, b0, empty_i, empty_v, 0.5, 0.9, 1e-4, label="empty")


def test_det_binary16_values():
    import torch
    rng = np.random.default_rng(66)
    sizes = [50_000, 333, 8192]
    d = sum(sizes)
    idx, val = _overlapping_lists(rng, d, 24, 3000, 4000, std=0.1)
    v16 = oracle.f16_rne(val)
    w0 = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    b0 = [np.zeros(n, np.float32) for n in sizes]
    det_update_vs_oracle(sizes, w0, b0, idx, v16, 0.1, 0.9, 5e-5, label="binary16",
                         val_dtype=torch.float16)


def test_det_c5_resnet50_p128_momentum_3_steps():
    """The P = 128 x 25,600 momentum update on ResNet-50-shaped parameters,
    three steps carried on the GPU, against the oracle run from the same
    start: bit for bit at every position on every step."""
    import torch
    dev = need_gpu()
    sizes = gen.numels(gen.resnet50_shapes())
    d = sum(sizes)
    w_host = gen.params_like(sizes, config=5)
    b_host = [np.zeros(n, np.float32) for n in sizes]
    w, b = to_dev(w_host, dev), to_dev(b_host, dev)
    P, k = 128, 25_600
    plan = tk.UpdatePlan(sizes, P=P, stride=k, deterministic=True).bind(w, b)
    w_ref, b_ref = gen.concat(w_host), gen.concat(b_host)
    for step in range(3):
        announce(f"det c5 step {step}")
        idx, val = gen.sparse_lists(d, P, k, step=step)
        plan.execute(torch.from_numpy(idx).to(dev), torch.from_numpy(val).to(dev),
                     lr=0.1, mu=0.9, wd=5e-5)
        torch.cuda.synchronize()
        w_ref, b_ref = orc().update(w_ref, b_ref, idx, val, lr=0.1, mu=0.9, wd=5e-5)
        assert_bitwise(gen.concat(to_host(w)), w_ref, f"w step {step}")
        assert_bitwise(gen.concat(to_host(b)), b_ref, f"b step {step}")


def test_det_aggregate_repeatable_and_exact():
    """The dense sum of the P = 128 lists (Alg. 2's g~) 100 times: identical
    bytes every time, equal to the oracle's worker-ordered sum."""
    import torch
    dev = need_gpu()
    sizes = gen.numels(gen.resnet50_shapes())
    d = sum(sizes)
    P, k = 128, 25_600
    idx, val = gen.sparse_lists(d, P, k, step=7)
    out = to_dev([np.zeros(n, np.float32) for n in sizes], dev)
    plan = tk.UpdatePlan(sizes, P=P, stride=k, deterministic=True).bind(out)
    it, vt, _ = _tensors(idx, val, None, dev)
    announce("det aggregate x100")
    plan.aggregate(it, vt)
    torch.cuda.synchronize()
    first = torch.cat(out).clone()
    assert_bitwise(first.cpu().numpy(), orc().aggregate(d, idx, val), "aggregate")
    for rep in range(99):
        plan.aggregate(it, vt)
        if rep % 33 == 32:
            torch.cuda.synchronize()
            assert torch.equal(torch.cat(out).view(torch.int32), first.view(torch.int32)), rep
    torch.cuda.synchronize()
    assert torch.equal(torch.cat(out).view(torch.int32), first.view(torch.int32))


@pytest.mark.parametrize("mom", [False, True])
def test_det_lars_step(mom):
    """LARS with the deterministic sum: G is the oracle's, so the rates
    agree to the double sums' rounding (1e-12), and every tensor whose
    binary32 rate agrees matches bit for bit at every position."""
    import torch
    dev = need_gpu()
    rng = np.random.default_rng(67 + mom)
    sizes = [50_000, 333, 8192, 1]
    d = sum(sizes)
    idx, val = _overlapping_lists(rng, d, 40, 3000, 4000, std=0.1)
    w0 = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    b0 = [(rng.standard_normal(n) * 0.01).astype(np.float32) for n in sizes] if mom else None
    gamma, eta, eps, mu = 0.001, 0.1, 5e-5, (0.9 if mom else 0.0)
    announce(f"det lars mom={mom}")
    w = to_dev(w0, dev)
    b = to_dev(b0, dev) if b0 is not None else None
    plan = tk.UpdatePlan(sizes, P=40, stride=3000, deterministic=True).bind(w, b)
    it, vt, _ = _tensors(idx, val, None, dev)
    rates = plan.lars_execute(it, vt, gamma, eta, eps, mu=mu).cpu().numpy()
    torch.cuda.synchronize()
    G = orc().aggregate(d, idx, val)
    Gs = np.split(G, np.cumsum(sizes)[:-1])
    w_ref, b_ref, r_ref = lars.lars_update(w0, b0, Gs, gamma, eta, eps, mu)
    rel = np.abs(np.asarray(rates, np.float64) - r_ref)
    assert np.all(rel <= 1e-12 * np.abs(r_ref)), (rates, r_ref)
    wg = to_host(w)
    bg = to_host(b) if b is not None else None
    same32 = np.float32(rates) == np.float32(r_ref)
    assert same32.sum() >= len(sizes) - 1
    for t in range(len(sizes)):
        if not same32[t]:
            continue
        assert_bitwise(wg[t], w_ref[t], f"w[{t}]")
        if bg is not None:
            assert_bitwise(bg[t], b_ref[t], f"b[{t}]")
