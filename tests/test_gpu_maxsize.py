"""GPU parity at the largest size the library takes: one tensor of
2^31 - 1 elements (int32 positions up to the last one, 2^18 tiles, every
selection workgroup the grid allows).

The oracle's full sort cannot finish at this size in a test, so the
selection is checked through the properties that fix it exactly at any size
(see check_selection in gpu_common): |S| = k, ascending positions, val =
x[idx] bitwise, residual = x outside S and +0 inside, no unselected magnitude
above a selected one, and the tie class at the threshold split toward lower
positions. The checks run as torch operations on the device (8 GiB per
array; a host copy would dominate the test). x itself is the device's
binary32 add of g and r, checked against the oracle's add on a sample of
positions (the planted ties, both ends and 4 M drawn at random). The update that follows is
checked bit-exactly against its definition: with at most two summands per
position, the sum does not depend on the order of addition.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2010_10458_amd as tk
from gpu_common import announce, assert_bitwise, need_gpu

pytestmark = pytest.mark.gpu

D_MAX = 2**31 - 1
RHO = 0.001
N_TIES = 20_000


def _i32(t):
    return t.view(torch.int32)


def _planted_input(dev):
    """g ~ N(0, 1) and r ~ N(0, 1e-3) over 2^31 - 1 positions (torch's seeded
    device generator), with N_TIES positions, the last eight among them, set
    to x = +-q exactly. q is the magnitude whose expected count above it among
    d standard normals is k - 10,000 (seven standard deviations below k), so
    the planted tie class straddles the k-th place and the index rule splits
    it."""
    from scipy.special import erfcinv

    d = D_MAX
    k = int(tk.k_from_rho(d, RHO))
    q = float(np.float32(np.sqrt(2.0) * erfcinv((k - 10_000) / d)))
    rng = np.random.default_rng(2_010_104_580)
    planted = rng.choice(d - 8, size=N_TIES - 8, replace=False)
    planted = np.concatenate([planted, np.arange(d - 8, d)])
    signs = np.where(rng.integers(0, 2, size=N_TIES) == 1, 1.0, -1.0).astype(np.float32)
    tg = torch.Generator(device=dev)
    tg.manual_seed(2_010_104_581)
    g = torch.randn(d, generator=tg, device=dev)
    r = torch.randn(d, generator=tg, device=dev).mul_(1e-3)
    pos = torch.from_numpy(planted.astype(np.int64)).to(dev)
    g[pos] = torch.from_numpy(signs * np.float32(q)).to(dev)
    r[pos] = 0.0
    x = g + r  # one binary32 add, the definition of x
    xa = x.abs()
    above = int((xa > q).sum())
    ties = int((xa == q).sum())
    del xa
    assert above < k < above + ties, (above, ties, k)
    check_x_against_oracle(g, r, x, planted)
    return g, r, x, k, q, above, ties


def check_x_against_oracle(g, r, x, planted):
    """x = fl32(g + r) at sampled positions, by the oracle's add."""
    rng = np.random.default_rng(77)
    d = x.numel()
    samp = np.unique(np.concatenate([planted, np.arange(1000), np.arange(d - 1000, d),
                                     rng.integers(0, d, 4_000_000)]))
    pos = torch.from_numpy(samp.astype(np.int64)).to(x.device)
    gs, rs, xs = g[pos].cpu().numpy(), r[pos].cpu().numpy(), x[pos].cpu().numpy()
    assert_bitwise(xs, oracle.Oracle().ef_add(gs, rs), "x = g + r (sampled)")


@pytest.mark.parametrize("mode", [tk.GLOBAL, tk.PER_TENSOR])
def test_max_size_sparsify(mode):
    dev = need_gpu()
    d = D_MAX
    announce(f"max size d={d} mode={mode}: generate")
    g, r, x, k, q, above, ties = _planted_input(dev)
    assert k == 2_147_484

    announce(f"max size d={d} mode={mode}: sparsify k={k}")
    plan = tk.SparsifyPlan([d], mode=mode, rho=RHO)
    plan.bind([g], [r])
    idx, val = plan.execute()
    torch.cuda.synchronize()
    del plan, g
    torch.cuda.empty_cache()

    li = idx.long()
    assert idx.numel() == k
    assert int(li[0]) >= 0 and int(li[-1]) < d
    assert bool((li[1:] > li[:-1]).all()), "indices not strictly ascending"
    assert torch.equal(_i32(val), _i32(x[li])), "val != x[idx]"
    assert bool((_i32(r[li]) == 0).all()), "selected residual entries must be +0.0"
    va = val.abs()
    T = float(va.min())
    assert T == q
    sel_tie = va == T
    assert int(sel_tie.sum()) == k - above
    last_sel_tie = int(li[sel_tie].max())
    x[li] = 0.0
    assert torch.equal(_i32(r), _i32(x)), "unselected residual != x"
    x.abs_()
    assert float(x.max()) <= T, "an unselected magnitude exceeds a selected one"
    unsel_tie = x == T
    assert int(unsel_tie.sum()) == ties - (k - above)
    first_unsel_tie = int(torch.argmax(unsel_tie.to(torch.uint8)))
    assert last_sel_tie < first_unsel_tie, "ties not broken toward lower positions"
    del x, r, unsel_tie, sel_tie, va, li, idx, val
    torch.cuda.empty_cache()


def test_max_size_plain_update():
    """Plain update (mu = wd = 0) of 2^31 - 1 parameters with two seeded
    ascending lists (2.1 M and 5 K entries) that both include the first and
    the last positions."""
    dev = need_gpu()
    d = D_MAX
    rng = np.random.default_rng(2_010_104_582)
    ends = [0, d - 2, d - 1]
    lists = [np.unique(np.concatenate([rng.integers(0, d, size=n), ends])).astype(np.int32)
             for n in (2_150_000, 5_000)]
    vals = [(rng.standard_normal(a.size) * 0.01).astype(np.float32) for a in lists]
    stride = max(a.size for a in lists)
    idx_all = torch.zeros((2, stride), dtype=torch.int32, device=dev)
    val_all = torch.zeros((2, stride), dtype=torch.float32, device=dev)
    for p, (a, v) in enumerate(zip(lists, vals)):
        idx_all[p, :a.size] = torch.from_numpy(a).to(dev)
        val_all[p, :a.size] = torch.from_numpy(v).to(dev)
    nnz = torch.tensor([a.size for a in lists], dtype=torch.int32, device=dev)
    announce(f"max size d={d}: plain update P=2")
    tg = torch.Generator(device=dev)
    tg.manual_seed(2_010_104_583)
    w = torch.randn(d, generator=tg, device=dev).mul_(0.1)
    w0 = w.clone()
    up = tk.UpdatePlan([d], P=2, stride=stride)
    up.bind([w])
    lr = 0.5
    up.execute(idx_all, val_all, lr=lr, nnz=nnz)
    torch.cuda.synchronize()
    del up

    G = torch.zeros(d, device=dev)
    for p, a in enumerate(lists):
        G.index_add_(0, idx_all[p, :a.size].long(), val_all[p, :a.size])
    step = G.mul_(lr)                # fl32(lr * G)
    w_ref = w0.sub_(step)            # fl32(w - fl32(lr * G)); untouched: w - 0 = w
    assert torch.equal(_i32(w), _i32(w_ref)), "plain update differs from its definition"
    del w, w0, G, idx_all, val_all
    torch.cuda.empty_cache()


def test_max_size_mstopk():
    """MSTopK (Alg. 1, N = 30) over 2^31 - 1 positions, through its
    invariants: the k1 positions at or above thres1 are all selected, the
    band {thres2 <= |x| < thres1} holds k2 - k1 positions, and the selection
    takes k - k1 consecutive band members (in position order) from the drawn
    offset; idx, val and the residual obey the sparsify contract."""
    dev = need_gpu()
    d = D_MAX
    announce(f"max size d={d}: MSTopK generate")
    g, r, x, k, q, above, ties = _planted_input(dev)
    del q, above, ties
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    announce(f"max size d={d}: MSTopK k={k}")
    plan = tk.SparsifyPlan([d], mode=tk.APPROX, rho=RHO, n_search=30)
    plan.bind([g], [r])
    idx, val = plan.execute(status=status, window_word=0x9E3779B97F4A7C15)
    torch.cuda.synchronize()
    res = plan.approx_result()
    del plan, g
    torch.cuda.empty_cache()
    assert int(status.item()) == 0

    k1, k2, off, take = res["k1"], res["k2"], res["offset"], res["take"]
    assert 0 <= k1 <= k <= k2 and take == k - k1 and 0 <= off <= k2 - k1 - take, res
    li = idx.long()
    assert idx.numel() == k
    assert bool((li[1:] > li[:-1]).all()), "indices not strictly ascending"
    assert torch.equal(_i32(val), _i32(x[li])), "val != x[idx]"
    assert bool((_i32(r[li]) == 0).all()), "selected residual entries must be +0.0"
    keys = _i32(x) & 0x7FFFFFFF
    ks = keys[li]
    assert int((ks >= res["key1"]).sum()) == k1
    assert int((keys >= res["key1"]).sum()) == k1, "a position above thres1 left out"
    in_band = (keys >= res["key2"]) & (keys < res["key1"])
    assert int(in_band.sum()) == k2 - k1
    band = torch.nonzero(in_band).squeeze(1)
    del in_band, keys
    sel_band = li[(ks >= res["key2"]) & (ks < res["key1"])]
    assert torch.equal(sel_band, band[off:off + take]), "band window is not consecutive"
    x[li] = 0.0
    assert torch.equal(_i32(r), _i32(x)), "unselected residual != x"
    del x, r, band, sel_band, li, idx, val
    torch.cuda.empty_cache()
