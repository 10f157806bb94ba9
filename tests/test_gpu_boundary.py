"""GPU parity of the one-shot C entry points, each through its Python
binding of the same name, against the oracle:

  tkef_sparsify          (tensor list; modes GLOBAL, PER_TENSOR, APPROX;
                          binary32 / binary16 values; counts_out)
  tkef_sparsify1         (one flat tensor, explicit k: Alg. 1's (x, k)
                          interface, Sec. 3.1)
  tkef_aggregate_update  (P separate worker lists, host counts: the lists
                          Alg. 2 gathers, Sec. 3.2, then the Eq. (1) update)

and the status handling of the one-shot calls (they raise TkefStatusError
when the device reports a problem). Selections are compared bit for bit;
updates with the tolerance of tests/test_gpu_update.py (bit for bit where a
position has at most two contributions, and on dyadic inputs everywhere).
"""
import zlib

import numpy as np
import pytest

import gen
import oracle
import oracle.mstopk as ms
import paper_2010_10458_amd as tk
from gpu_common import announce, assert_bitwise, need_gpu, to_dev, to_host
from test_gpu_update import compare

pytestmark = pytest.mark.gpu

ORC = None


def orc():
    global ORC
    if ORC is None:
        ORC = oracle.Oracle()
    return ORC


def _inputs(sizes, seed, scale=0.3):
    rng = np.random.default_rng(seed)
    g = [rng.standard_normal(n).astype(np.float32) for n in sizes]
    r = [(rng.standard_normal(n) * scale).astype(np.float32) for n in sizes]
    return g, r


@pytest.mark.parametrize("mode", ["global", "per_tensor", "approx"])
@pytest.mark.parametrize("val16", [False, True])
def test_sparsify_one_shot(mode, val16):
    import torch
    dev = need_gpu()
    sizes = [1, 4095, 8192 * 3 + 7, 0, 100_000, 33]
    grads, res = _inputs(sizes, zlib.crc32(f"{mode}/{val16}".encode()))
    m = {"global": tk.GLOBAL, "per_tensor": tk.PER_TENSOR, "approx": tk.APPROX}[mode]
    announce(f"tkef_sparsify one-shot mode={mode} val16={val16}")
    g, r = to_dev(grads, dev), to_dev(res, dev)
    idx, val, counts = tk.sparsify(g, r, rho=0.01, mode=m,
                                   val_dtype=torch.float16 if val16 else torch.float32,
                                   return_counts=True)
    rg = gen.concat(to_host(r))
    if mode == "approx":
        k = tk.k_from_rho(sum(sizes), 0.01)
        oi, ov, orr, _ = ms.mstopk_sparsify(gen.concat(grads), gen.concat(res), k, 30, 0)
        ks = [k]
    else:
        oi, ov, orr, ks = orc().sparsify(
            grads, res, rho=0.01,
            mode=oracle.PER_TENSOR if mode == "per_tensor" else oracle.GLOBAL)
        orr = gen.concat(orr)
    assert counts == list(ks)
    assert_bitwise(idx.cpu().numpy(), oi, "idx")
    if val16:
        assert np.array_equal(val.cpu().numpy().view(np.uint16),
                              oracle.f16_rne(ov).view(np.uint16)), "val (binary16)"
    else:
        assert_bitwise(val.cpu().numpy(), ov, "val")
    assert_bitwise(rg, orr, "residual")


@pytest.mark.parametrize("d,k", [(1, 1), (7, 7), (1000, 1), (8193, 100), (300_001, 3000),
                                 (1 << 20, 1049)])
def test_sparsify1(d, k):
    dev = need_gpu()
    rng = np.random.default_rng(d * 31 + k)
    g = rng.standard_normal(d).astype(np.float32)
    g[rng.random(d) < 0.05] = 1.5          # a tie class
    r = (rng.standard_normal(d) * 0.1).astype(np.float32)
    announce(f"tkef_sparsify1 d={d} k={k}")
    gt, rt = to_dev([g], dev), to_dev([r], dev)
    idx, val = tk.sparsify1(gt[0], rt[0], k)
    oi, ov, orr, _ = orc().sparsify([g], [r], k=k)
    assert_bitwise(idx.cpu().numpy(), oi, "idx")
    assert_bitwise(val.cpu().numpy(), ov, "val")
    assert_bitwise(to_host(rt)[0], orr[0], "residual")


def run_per_worker(sizes, w_host, b_host, idx, val, lr, mu, wd, nnz=None):
    """tkef_aggregate_update: worker p's list as its own pair of device
    tensors (its first nnz[p] entries), counts from the host."""
    import torch
    dev = need_gpu()
    w = to_dev(w_host, dev)
    b = to_dev(b_host, dev) if b_host is not None else None
    P, stride = idx.shape
    nn = [stride] * P if nnz is None else [int(np.clip(c, 0, stride)) for c in nnz]
    lists = [(torch.from_numpy(np.ascontiguousarray(idx[p, :nn[p]], np.int32)).to(dev),
              torch.from_numpy(np.ascontiguousarray(val[p, :nn[p]], np.float32)).to(dev))
             for p in range(P)]
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    tk.aggregate_update(w, lists, lr, momentum=b, mu=mu, wd=wd, status=status)
    torch.cuda.synchronize()
    return to_host(w), (to_host(b) if b is not None else None), int(status.item())


@pytest.mark.parametrize("mode", ["plain", "momentum"])
def test_aggregate_update_per_worker_lists(mode):
    rng = np.random.default_rng(700 + (mode == "momentum"))
    sizes = [1, 5, 64, 8193, 100, 30_000, 0, 17, 16_384, 3]
    d = sum(sizes)
    w0 = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    b0 = [(rng.standard_normal(n) * 0.01).astype(np.float32) for n in sizes] \
        if mode == "momentum" else None
    mu, wd = (0.9, 5e-5) if mode == "momentum" else (0.0, 0.0)
    for P in (1, 9, 300):                   # 300: more workers than a batch of 256
        k = 600
        idx = np.stack([np.sort(rng.choice(d, k, replace=False)) for _ in range(P)]).astype(np.int32)
        val = (rng.standard_normal((P, k)) * 1e-2).astype(np.float32)
        nnz = rng.integers(0, k + 1, P)
        nnz[0] = 0                          # an empty list (null pointers)
        if P > 1:
            nnz[1] = k
        compare(sizes, w0, b0, idx, val, 0.1, mu, wd, nnz=nnz, label=f"per-worker P={P}",
                runner=run_per_worker)


def test_aggregate_update_per_worker_dyadic_bit_exact():
    rng = np.random.default_rng(702)
    sizes = [8192 * 3 + 11, 517, 4096]
    d = sum(sizes)
    w0 = [(rng.integers(-4095, 4096, n) / 256.0).astype(np.float32) for n in sizes]
    b0 = [np.zeros(n, np.float32) for n in sizes]
    P, k = 24, 3000
    pool = rng.choice(d, 4000, replace=False)
    idx = np.stack([np.sort(rng.choice(pool, k, replace=False)) for _ in range(P)]).astype(np.int32)
    e = rng.integers(-8, -3, (P, k)).astype(np.float64)
    val = (np.exp2(e) * np.where(rng.random((P, k)) < 0.5, -1, 1)).astype(np.float32)
    compare(sizes, w0, b0, idx, val, 0.25, 0.5, 0.0625, exact=True, label="per-worker dyadic",
            runner=run_per_worker)


def run_gathered_one_shot(sizes, w_host, b_host, idx, val, lr, mu, wd, nnz=None):
    """tkef_sparse_aggregate_update: the (P, stride) gathered layout."""
    import torch
    dev = need_gpu()
    w = to_dev(w_host, dev)
    b = to_dev(b_host, dev) if b_host is not None else None
    nt = torch.from_numpy(np.asarray(nnz, np.int32)).to(dev) if nnz is not None else None
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    tk.sparse_aggregate_update(w, torch.from_numpy(np.ascontiguousarray(idx, np.int32)).to(dev),
                               torch.from_numpy(np.ascontiguousarray(val, np.float32)).to(dev),
                               lr, momentum=b, mu=mu, wd=wd, nnz=nt, status=status)
    torch.cuda.synchronize()
    return to_host(w), (to_host(b) if b is not None else None), int(status.item())


@pytest.mark.parametrize("form", ["per_worker", "gathered"])
def test_aggregate_update_one_shots_c5(form):
    """The aggregate-update workload (P = 128 lists of 25,600 pairs into the
    ResNet-50-shaped parameters, momentum 0.9, wd 5e-5, lr 0.1) through each
    one-shot entry point, against the oracle."""
    sizes = gen.numels(gen.resnet50_shapes())
    d = sum(sizes)
    w_host = gen.params_like(sizes, config=5)
    b_host = [np.zeros(n, np.float32) for n in sizes]
    idx, val = gen.sparse_lists(d, 128, 25_600, step=0)
    compare(sizes, w_host, b_host, idx, val, 0.1, 0.9, 5e-5, label=f"c5 {form} one-shot",
            runner=run_per_worker if form == "per_worker" else run_gathered_one_shot)


def test_one_shots_raise_on_device_status():
    import torch
    dev = need_gpu()
    g = np.ones(5000, np.float32)
    g[17] = np.nan
    announce("one-shot status: NaN")
    gt, rt = to_dev([g], dev), to_dev([np.zeros(5000, np.float32)], dev)
    with pytest.raises(tk.TkefStatusError) as ei:
        tk.sparsify1(gt[0], rt[0], 10)
    assert ei.value.bits & tk.STATUS_NAN
    # with a caller status word the call does not raise; the bit is there
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    tk.sparsify(gt, rt, k=10, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) & tk.STATUS_NAN
    announce("one-shot status: unsorted list")
    w = to_dev([np.ones(1000, np.float32)], dev)
    bad = torch.tensor([5, 3, 9], dtype=torch.int32, device=dev)
    with pytest.raises(tk.TkefStatusError) as ei:
        tk.aggregate_update(w, [(bad, torch.ones(3, device=dev))], 0.1)
    assert ei.value.bits & tk.STATUS_UNSORTED
    plan = tk.UpdatePlan([1000], P=1, stride=3, check=True)
    plan.bind(w)
    with pytest.raises(tk.TkefStatusError):
        plan.execute(bad.view(1, 3), torch.ones(1, 3, device=dev), lr=0.1)
