"""GPU parity: the dense aggregation of P sparse lists (Alg. 2 returns the
accumulated vector) and 16-bit values on the wire (Sec. 5.3 sends FP16
elements), through the C ABI, against the CPU oracle.

Aggregation: the oracle adds each position's contributions in worker order;
the GPU may add them in another order. A binary32 sum of one or two terms is
order-free, so positions with at most two contributions match bit for bit;
for c >= 3 terms both results are recursive sums of the same terms, each
within (c - 1) u sum|v| of the exact sum (u = 2^-24), so they differ by at
most 2 (c - 1) u sum|v|. Dyadic inputs make every order exact: bit for bit.

16-bit values: the index list and the residual are the exact path's, bit for
bit; each value is the oracle's binary32 value rounded to binary16 (nearest,
ties to even, overflow to infinity, subnormals kept).
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


def gpu_aggregate(sizes, idx, val, nnz=None, val_dtype=None):
    import torch
    dev = need_gpu()
    outs = [torch.full((n,), float("nan"), dtype=torch.float32, device=dev) for n in sizes]
    it = torch.from_numpy(np.ascontiguousarray(idx, np.int32)).to(dev)
    vt = torch.from_numpy(np.ascontiguousarray(val)).to(dev)
    nt = torch.from_numpy(np.asarray(nnz, np.int32)).to(dev) if nnz is not None else None
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    P, stride = idx.shape
    plan = tk.UpdatePlan(sizes, P=P, stride=stride, val_dtype=vt.dtype)
    plan.bind(outs)
    plan.aggregate(it, vt, nnz=nt, status=status)
    torch.cuda.synchronize()
    return gen.concat(to_host(outs)), int(status.item())


def compare_aggregate(sizes, idx, val, nnz=None, exact=False, label=""):
    announce(f"aggregate {label} P={idx.shape[0]} stride={idx.shape[1]} dtype={val.dtype}")
    out, status = gpu_aggregate(sizes, idx, val, nnz)
    assert status == 0
    d = sum(sizes)
    ref = orc().aggregate(d, idx, val, None if nnz is None else np.asarray(nnz, np.int64))
    if exact:
        assert_bitwise(out, ref, "g~")
        return out
    P, stride = idx.shape
    nn = np.full(P, stride) if nnz is None else np.clip(np.asarray(nnz), 0, stride)
    flat_i = np.concatenate([idx[p, :nn[p]] for p in range(P)]).astype(np.int64)
    flat_v = np.concatenate([val[p, :nn[p]] for p in range(P)]).astype(np.float64)
    cnt = np.bincount(flat_i, minlength=d)
    A = np.zeros(d)
    np.add.at(A, flat_i, np.abs(flat_v))
    le2 = cnt <= 2
    assert_bitwise(out[le2], ref[le2], "g~ (<= 2 contributions)")
    bound = 2 * np.maximum(cnt - 1, 0) * 2.0 ** -24 * A
    assert np.all(np.abs(out.astype(np.float64) - ref) <= bound)
    return out


def _lists(rng, d, P, k, std=1e-2, overlap=True):
    idx = np.empty((P, k), np.int32)
    pool = rng.choice(d, size=min(d, 2 * k), replace=False) if overlap else None
    for p in range(P):
        idx[p] = np.sort(rng.choice(pool if overlap else d, size=k, replace=False))
    val = (rng.standard_normal((P, k)) * std).astype(np.float32)
    return idx, val


SIZE_SETS = {
    "single": [100_003],
    "ragged": [1, 5, 64, 8193, 100, 30_000, 0, 17, 16_384, 3],
}


@pytest.mark.parametrize("sizes_name", sorted(SIZE_SETS))
@pytest.mark.parametrize("P", [1, 3, 40])
def test_aggregate_random(sizes_name, P):
    sizes = SIZE_SETS[sizes_name]
    d = sum(sizes)
    rng = np.random.default_rng(zlib.crc32(f"agg/{sizes_name}/{P}".encode()))
    k = max(1, d // 50 + 1)
    idx, val = _lists(rng, d, P, min(k, d), overlap=P > 1)
    out = compare_aggregate(sizes, idx, val, label=sizes_name)
    # every position is written: untouched ones are +0
    touched = np.zeros(d, bool)
    touched[idx.ravel()] = True
    assert np.array_equal(bits(out[~touched]), np.zeros(int((~touched).sum()), np.uint32))


def test_aggregate_dyadic_bit_exact_duplicates_ragged_and_empty():
    rng = np.random.default_rng(41)
    sizes = [8192 * 3 + 11, 517, 4096]
    d = sum(sizes)
    P, k = 24, 3000
    pool = rng.choice(d, 4000, replace=False)
    idx = np.stack([np.sort(rng.choice(pool, k, replace=False)) for _ in range(P)]).astype(np.int32)
    idx[5, :60] = 123                     # one list naming one position 60 times
    idx[5] = np.sort(idx[5])
    e = rng.integers(-8, -3, (P, k)).astype(np.float64)
    val = (np.exp2(e) * np.where(rng.random((P, k)) < 0.5, -1, 1)).astype(np.float32)
    compare_aggregate(sizes, idx, val, exact=True, label="dyadic")
    nnz = rng.integers(0, k + 1, P).astype(np.int32)
    nnz[0], nnz[1] = 0, 1
    compare_aggregate(sizes, idx, val, nnz=nnz, exact=True, label="dyadic ragged nnz")
    out = compare_aggregate(sizes, np.zeros((3, 0), np.int32), np.zeros((3, 0), np.float32),
                            exact=True, label="empty lists")
    assert not out.any()


def test_aggregate_worker_order_example():
    """1 + 2^-24 + 2^-24 added in worker order is 1; any order that adds the
    two small terms first gives 1 + 2^-23. Three terms are one case where the
    order shows; the test states which results are acceptable."""
    t = np.float32(2.0 ** -24)
    idx = np.array([[0], [0], [0]], np.int32)
    val = np.array([[1.0], [t], [t]], np.float32)
    announce("aggregate order example")
    out, status = gpu_aggregate([5], idx, val)
    assert status == 0
    assert out[0] in (np.float32(1.0), np.float32(1.0 + 2.0 ** -23))
    assert not out[1:].any()


def test_c5_resnet50_p128_aggregate():
    """P = 128 workers x 25,600 pairs summed densely into ResNet-50-shaped
    buffers (the update workload's lists, no optimizer)."""
    sizes = gen.numels(gen.resnet50_shapes())
    d = sum(sizes)
    idx, val = gen.sparse_lists(d, 128, 25_600, step=0)
    compare_aggregate(sizes, idx, val, label="resnet50 P=128")


# ----------------------------------------------------------------------------
# 16-bit values on the wire

def sparsify16(grads, residuals, rho=None, k=None, mode=tk.GLOBAL):
    import torch
    dev = need_gpu()
    g = to_dev(grads, dev)
    r = to_dev(residuals, dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    plan = tk.SparsifyPlan([a.size for a in grads], mode=mode, rho=rho, k=k,
                           val_dtype=torch.float16)
    plan.bind(g, r)
    idx, val = plan.execute(status=status)
    torch.cuda.synchronize()
    assert val.dtype == torch.float16
    return idx.cpu().numpy(), val.cpu().numpy(), to_host(r), int(status.item())


def compare16(grads, residuals, rho=None, k=None, mode=tk.GLOBAL, label=""):
    announce(f"sparsify fp16 {label} sizes={[a.size for a in grads][:6]} rho={rho} k={k}")
    idx, val, r, status = sparsify16(grads, residuals, rho=rho, k=k, mode=mode)
    oi, ov, orr, _ = orc().sparsify(grads, residuals, rho=rho, k=k,
                                    mode=oracle.GLOBAL if mode == tk.GLOBAL else oracle.PER_TENSOR)
    assert status == 0
    assert_bitwise(idx, oi, "idx")
    assert np.array_equal(val.view(np.uint16), oracle.f16_rne(ov).view(np.uint16)), "val (fp16)"
    for t, (a, b) in enumerate(zip(r, orr)):
        assert_bitwise(a, b.ravel(), f"residual[{t}]")
    return idx, val


def test_fp16_values_edge_magnitudes():
    """Values past the binary16 range (to infinity), at its top, in its
    subnormal range and exact ties, mixed into a normal vector."""
    rng = np.random.default_rng(51)
    n = 70_001
    g = (rng.standard_normal(n) * 1e-6).astype(np.float32)
    special = np.array([1e9, -7e4, 65520.0, 65519.0, 65504.0, -2.0 ** -24, 2.0 ** -25,
                        3 * 2.0 ** -25, 1.0 + 2.0 ** -11, -(1.0 + 3 * 2.0 ** -11), 1 / 3,
                        5.9604645e-08, 6.1035156e-05, -1.5e-5], np.float32)
    pos = rng.choice(n, special.size, replace=False)
    g[pos] = special
    r = np.zeros(n, np.float32)
    for k in (5, special.size, 700, n):
        compare16([g], [r], k=k, label=f"edge k={k}")


def test_fp16_values_dense_regions():
    """A dense selection with binary16 values: 2^21 elements on a grid of
    1/256 (ties), k = 150,000, so every selection region stores thousands of
    candidates and the finish kernel writes them in rounds of one per
    thread; globally and per tensor (two tensors)."""
    rng = np.random.default_rng(53)
    n = 1 << 21
    g = (np.round(rng.standard_normal(n) * 256) / 256).astype(np.float32)
    r = np.zeros(n, np.float32)
    compare16([g], [r], k=150_000, label="dense fp16")
    h = n // 2
    compare16([g[:h], g[h:]], [r[:h], r[h:]], rho=0.07, mode=tk.PER_TENSOR,
              label="dense fp16 per tensor")


@pytest.mark.parametrize("mode", [tk.GLOBAL, tk.PER_TENSOR])
def test_fp16_values_resnet_step(mode):
    sizes = gen.numels(gen.resnet50_shapes())
    grads = gen.resnet_grads(step=0)
    res = [np.zeros(n, np.float32) for n in sizes]
    compare16(grads, res, rho=0.001, mode=mode, label=f"resnet50 mode={mode}")


def test_shard_sparsify_hitopk():
    """The per-GPU share of the hierarchical scheme (Sec. 3.2, Alg. 2): one node of
    n = 8 GPUs splits the 25,557,032-element ResNet-50 gradient into eight
    contiguous shards; each GPU selects k~ = ceil(rho d / n) of its shard.
    Checks the first and the last (ragged) shard, fp32 and fp16 values."""
    d, n = gen.RESNET50_D, 8
    g = gen.flat_normal(d, config=2, std=1e-2)
    shard = -(-d // n)
    for s in (0, n - 1):
        lo, hi = s * shard, min(d, (s + 1) * shard)
        gs = np.ascontiguousarray(g[lo:hi])
        rs = (gen.flat_normal(hi - lo, config=2, step=1, std=1e-3))
        k = int(np.ceil(0.001 * d / n))
        announce(f"shard {s} size={hi - lo} k={k}")
        import test_gpu_sparsify as ts
        ts.compare_with_oracle([gs], [rs], k=k, label=f"shard {s}")
        compare16([gs], [rs], k=k, label=f"shard {s}")


def test_fp16_update_and_aggregate():
    """Lists with binary16 values: the kernels widen each value exactly and
    accumulate in binary32, so the results equal the binary32 path fed the
    widened values."""
    import torch
    rng = np.random.default_rng(52)
    sizes = [50_000, 333, 8192]
    d = sum(sizes)
    P, k = 12, 2000
    idx, val32 = _lists(rng, d, P, k, std=1e-1)
    val16 = oracle.f16_rne(val32)
    compare_aggregate(sizes, idx, val16, label="fp16 values")
    dev = need_gpu()
    w0 = (rng.standard_normal(d) * 0.1).astype(np.float32)
    b0 = np.zeros(d, np.float32)
    announce("update fp16 values momentum")
    w = [torch.from_numpy(a.copy()).to(dev) for a in np.split(w0, np.cumsum(sizes)[:-1])]
    b = [torch.from_numpy(a.copy()).to(dev) for a in np.split(b0, np.cumsum(sizes)[:-1])]
    plan = tk.UpdatePlan(sizes, P=P, stride=k, val_dtype=torch.float16)
    plan.bind(w, b)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    plan.execute(torch.from_numpy(idx).to(dev), torch.from_numpy(val16).to(dev),
                 lr=0.1, mu=0.9, wd=5e-5, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    w_ref, b_ref = orc().update(w0, b0, idx, val16.astype(np.float32), lr=0.1, mu=0.9, wd=5e-5)
    wg, bg = gen.concat(to_host(w)), gen.concat(to_host(b))
    cnt = np.bincount(idx.ravel(), minlength=d)
    le2 = cnt <= 2
    assert_bitwise(wg[le2], w_ref[le2], "w (<= 2 contributions)")
    assert_bitwise(bg[le2], b_ref[le2], "b (<= 2 contributions)")
    A = np.zeros(d)
    np.add.at(A, idx.ravel(), np.abs(val16.astype(np.float64).ravel()))
    S = 0.1 * (A + 5e-5 * np.abs(w0))
    assert np.all(np.abs(wg.astype(np.float64) - w_ref) <= 1e-6 * (np.abs(w_ref) + S))
    assert np.all(np.abs(bg.astype(np.float64) - b_ref) <= 1e-6 * (np.abs(b_ref) + S / 0.1))


def test_fp16_plan_rejects_mismatched_dtype():
    import torch
    dev = need_gpu()
    plan = tk.UpdatePlan([100], P=1, stride=4, val_dtype=torch.float16)
    plan.bind([torch.zeros(100, device=dev)])
    with pytest.raises(ValueError):
        plan.aggregate(torch.zeros((1, 4), dtype=torch.int32, device=dev),
                       torch.zeros((1, 4), dtype=torch.float32, device=dev))
