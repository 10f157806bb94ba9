"""GPU parity: tkef sparsify (through the C ABI) against the CPU oracle.

Bit-exact on idx, val and the updated residual. Small cases are compared
element by element with the oracle; the ResNet-50-shaped workload runs the
full oracle on its first and last error-feedback steps and the exact
selection properties on every step; the 110 M and 340 M workloads use the
exact selection properties plus ranks of sampled positions computed one by
one by the oracle.
"""
import numpy as np
import pytest

import gen
import oracle
import paper_2010_10458_amd as tk
from gpu_common import (announce, assert_bitwise, bits, check_selection, need_gpu, to_dev,
                        to_host)

pytestmark = pytest.mark.gpu

ORC = None


def orc():
    global ORC
    if ORC is None:
        ORC = oracle.Oracle()
    return ORC


def run_gpu(grads, residuals, rho=None, k=None, mode=tk.GLOBAL):
    import torch
    dev = need_gpu()
    g = to_dev(grads, dev)
    r = to_dev(residuals, dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    plan = tk.SparsifyPlan([a.size for a in grads], mode=mode, rho=rho, k=k)
    plan.bind(g, r)
    idx, val = plan.execute(status=status)
    torch.cuda.synchronize()
    return (idx.cpu().numpy(), val.cpu().numpy(), to_host(r), int(status.item()), plan)


def compare_with_oracle(grads, residuals, rho=None, k=None, mode=tk.GLOBAL, label=""):
    announce(f"sparsify {label} sizes={[a.size for a in grads][:6]} rho={rho} k={k} mode={mode}")
    idx, val, r, status, plan = run_gpu(grads, residuals, rho=rho, k=k, mode=mode)
    oi, ov, orr, ks = orc().sparsify(grads, residuals, rho=rho, k=k,
                                     mode=oracle.GLOBAL if mode == tk.GLOBAL else oracle.PER_TENSOR)
    assert plan.k_total == sum(ks)
    assert_bitwise(idx, oi, "idx")
    assert_bitwise(val, ov, "val")
    for t, (a, b) in enumerate(zip(r, orr)):
        assert_bitwise(a, b.ravel(), f"residual[{t}]")
    assert status == 0
    return idx, val, r


SIZES = [1, 2, 7, 31, 32, 33, 1000, 8191, 8192, 8193, 3 * 8192 + 5, 100_003]


@pytest.mark.parametrize("n", SIZES)
def test_flat_normal_sizes(n):
    rng = np.random.default_rng(100 + n)
    g = rng.standard_normal(n).astype(np.float32)
    r = (rng.standard_normal(n) * 0.3).astype(np.float32)
    for k in sorted({1, max(1, n // 1000), max(1, n // 10), max(1, n - 1), n}):
        compare_with_oracle([g], [r], k=k, label=f"normal n={n}")


@pytest.mark.parametrize("levels", [2, 5, 64])
def test_ties(levels):
    rng = np.random.default_rng(200 + levels)
    n = 50_001
    mags = rng.integers(0, levels, n).astype(np.float32) * np.float32(0.5)
    g = np.where(rng.random(n) < 0.5, -mags, mags).astype(np.float32)
    r = np.zeros(n, np.float32)
    for k in (1, 17, 5000, 25_000, n - 3, n):
        compare_with_oracle([g], [r], k=k, label=f"ties levels={levels}")


def test_special_values():
    tiny = np.float32(np.finfo(np.float32).smallest_subnormal)
    rng = np.random.default_rng(7)
    n = 20_000
    g = (rng.standard_normal(n) * 1e-38).astype(np.float32)   # subnormal-range sums
    g[::97] = np.inf
    g[5::97] = -np.inf
    g[7::13] = -0.0
    g[9::31] = tiny
    g[11::31] = -3 * tiny
    r = np.zeros(n, np.float32)
    r[::2] = -0.0
    r[1::7] = (rng.standard_normal(n)[1::7] * 1e-39).astype(np.float32)
    r[::97] = 0.0
    r[5::97] = 0.0
    for k in (1, 50, 300, 5000, n):
        compare_with_oracle([g], [r], k=k, label="special values")


def test_all_zero_and_all_equal():
    n = 70_000
    z = np.zeros(n, np.float32)
    zm = np.full(n, -0.0, np.float32)
    compare_with_oracle([zm], [zm.copy()], k=123, label="all -0")
    compare_with_oracle([z], [zm], k=n, label="all zero k=d")
    c = np.where(np.arange(n) % 3 == 0, np.float32(-2.5), np.float32(2.5))
    compare_with_oracle([c], [z], k=40_000, label="all equal magnitude")


def test_multi_tensor_global_and_per_tensor():
    rng = np.random.default_rng(300)
    sizes = [1, 5, 64, 8193, 100, 30_000, 0, 17, 16_384, 3]
    grads = [(rng.standard_normal(n) * (1 + t)).astype(np.float32) for t, n in enumerate(sizes)]
    res = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    compare_with_oracle(grads, res, rho=0.001, label="multi global 0.001")
    compare_with_oracle(grads, res, rho=0.05, label="multi global 0.05")
    compare_with_oracle(grads, res, k=1, label="multi global k=1")
    compare_with_oracle(grads, res, rho=0.01, mode=tk.PER_TENSOR, label="multi per-tensor 0.01")
    compare_with_oracle(grads, res, rho=0.3, mode=tk.PER_TENSOR, label="multi per-tensor 0.3")


def test_per_tensor_candidate_overflow_and_dense_threads():
    """Per tensor: a 300 K tensor of one magnitude (every element a candidate
    of its group: more than the candidate list holds, 4 k_total + 65,536, so
    hist3 and emit walk the lines instead) next to ordinary tensors; and a
    dense selection where threads hold more candidates than gather stages."""
    rng = np.random.default_rng(310)
    n0 = 300_000
    flat = np.where(np.arange(n0) % 5 == 0, np.float32(-0.75), np.float32(0.75))
    grads = [flat, (rng.standard_normal(50_000)).astype(np.float32),
             (rng.standard_normal(8_193) * 3).astype(np.float32)]
    res = [np.zeros(a.size, np.float32) for a in grads]
    compare_with_oracle(grads, res, rho=0.001, mode=tk.PER_TENSOR, label="per-tensor overflow")
    dense = [(rng.standard_normal(n) * (1 + t)).astype(np.float32)
             for t, n in enumerate([200_000, 70_001, 5])]
    res = [(rng.standard_normal(a.size) * 0.1).astype(np.float32) for a in dense]
    compare_with_oracle(dense, res, rho=0.4, mode=tk.PER_TENSOR, label="per-tensor rho 0.4")


def test_per_tensor_many_groups():
    """1,100 small tensors per tensor (more groups than emit forms bases for
    itself: the group-scan kernel runs), 5,000 (more groups than the
    selection grids have workgroups, and several rounds of the group scan) and
    1,000 (emit forms them)."""
    rng = np.random.default_rng(311)
    for T in (1100, 5000, 1000):
        sizes = [int(n) for n in rng.integers(0, 300, T)]
        grads = [(rng.standard_normal(n) * (1 + (t % 7))).astype(np.float32)
                 for t, n in enumerate(sizes)]
        res = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
        compare_with_oracle(grads, res, rho=0.05, mode=tk.PER_TENSOR, label=f"{T} groups")


def test_unaligned_views():
    """Tensors that start off a 16-byte boundary take the scalar path."""
    import torch
    dev = need_gpu()
    rng = np.random.default_rng(400)
    sizes = [8192 * 2 + 3, 777, 12_000]
    grads = [rng.standard_normal(n).astype(np.float32) for n in sizes]
    res = [(rng.standard_normal(n) * 0.5).astype(np.float32) for n in sizes]
    announce("sparsify unaligned views")
    gbig = [torch.zeros(n + 1, device=dev) for n in sizes]
    rbig = [torch.zeros(n + 3, device=dev) for n in sizes]
    g = [b[1:] for b in gbig]
    r = [b[3:] for b in rbig]
    for t, a in zip(g + r, grads + res):
        t.copy_(torch.from_numpy(a))
    for t in g + r:
        assert t.data_ptr() % 16 != 0
    plan = tk.SparsifyPlan(sizes, rho=0.01)
    plan.bind(g, r)
    idx, val = plan.execute()
    torch.cuda.synchronize()
    oi, ov, orr, _ = orc().sparsify(grads, res, rho=0.01)
    assert_bitwise(idx.cpu().numpy(), oi, "idx")
    assert_bitwise(val.cpu().numpy(), ov, "val")
    for a, b in zip(to_host(r), orr):
        assert_bitwise(a, b, "residual")


def test_repeated_execution_is_deterministic():
    import torch
    dev = need_gpu()
    rng = np.random.default_rng(500)
    n = 300_007
    g = (np.round(rng.standard_normal(n) * 16) / 16).astype(np.float32)
    announce("sparsify repeat x100")
    out = None
    for it in range(100):
        gt = to_dev([g], dev)
        rt = to_dev([np.zeros(n, np.float32)], dev)
        plan = tk.SparsifyPlan([n], rho=0.01)
        plan.bind(gt, rt)
        idx, val = plan.execute()
        cur = (idx.cpu().numpy().copy(), val.cpu().numpy().copy(), rt[0].cpu().numpy().copy())
        if out is None:
            out = cur
        else:
            for a, b, w in zip(cur, out, ("idx", "val", "r")):
                assert_bitwise(a, b, w)


def test_nan_sets_status():
    n = 10_000
    g = np.ones(n, np.float32)
    g[1234] = np.nan
    announce("sparsify NaN status")
    idx, val, r, status, plan = run_gpu([g], [np.zeros(n, np.float32)], k=10)
    assert status & tk.STATUS_NAN
    assert idx.size == 10 and np.all((idx >= 0) & (idx < n))


def test_one_shot_entry_point():
    import torch
    dev = need_gpu()
    rng = np.random.default_rng(600)
    sizes = [4000, 9000]
    grads = [rng.standard_normal(n).astype(np.float32) for n in sizes]
    res = [np.zeros(n, np.float32) for n in sizes]
    announce("sparsify one-shot")
    g, r = to_dev(grads, dev), to_dev(res, dev)
    idx, val = tk.sparsify(g, r, rho=0.001)
    torch.cuda.synchronize()
    oi, ov, _, _ = orc().sparsify(grads, res, rho=0.001)
    assert_bitwise(idx.cpu().numpy(), oi, "idx")
    assert_bitwise(val.cpu().numpy(), ov, "val")


# ---------------------------------------------------------------- workloads

def test_c1_single_tensor_1m():
    g = gen.flat_normal(gen.C1_D, config=1)
    r = np.zeros_like(g)
    idx, val, rr = compare_with_oracle([g], [r], rho=0.001, label="1M N(0,1) rho=0.001")
    assert idx.size == 1049


def test_resnet50_residual_carry_10_steps():
    """161 tensors, 25,557,032 elements, rho = 0.001 global, 10 error-feedback
    steps with a fresh gradient each step and the residual carried on the GPU."""
    import torch
    dev = need_gpu()
    sizes = gen.numels(gen.resnet50_shapes())
    plan = tk.SparsifyPlan(sizes, rho=0.001)
    assert plan.k_total == 25_558
    gdev = [torch.empty(n, device=dev) for n in sizes]
    rdev = [torch.zeros(n, device=dev) for n in sizes]
    plan.bind(gdev, rdev)
    r_host = [np.zeros(n, np.float32) for n in sizes]
    for step in range(10):
        announce(f"resnet50 carry step {step}")
        grads = gen.resnet_grads(step)
        for t, a in zip(gdev, grads):
            t.copy_(torch.from_numpy(a))
        idx, val = plan.execute()
        torch.cuda.synchronize()
        idx, val = idx.cpu().numpy(), val.cpu().numpy()
        r_new = [t.cpu().numpy() for t in rdev]
        x = orc().ef_add(gen.concat(grads), gen.concat(r_host))
        check_selection(x, idx, val, gen.concat(r_new), 25_558)
        if step in (0, 9):
            oi, ov, orr, _ = orc().sparsify(grads, r_host, rho=0.001)
            assert_bitwise(idx, oi, "idx")
            assert_bitwise(val, ov, "val")
            assert_bitwise(gen.concat(r_new), gen.concat(orr), "residual")
        r_host = r_new


def _sampled_ranks(x, idx, k, rng, nsamp=6):
    """The oracle's rank of sampled positions: selected ones rank below k,
    unselected ones at or above it."""
    sel = rng.choice(idx, size=min(nsamp, idx.size), replace=False)
    mask = np.ones(x.size, bool)
    mask[idx] = False
    a = np.abs(x)
    top = a[mask].max()
    boundary = np.nonzero(mask & (a == top))[0][:nsamp]   # largest unselected
    for i in sel:
        assert orc().rank(x, int(i)) < k
    for i in boundary:
        assert orc().rank(x, int(i)) >= k


def test_transformer_110m_global_and_per_tensor():
    import torch
    dev = need_gpu()
    sizes = gen.numels(gen.transformer_shapes())
    grads = gen.laplace_grads(0, sizes)
    x = orc().ef_add(gen.concat(grads), np.zeros(sum(sizes), np.float32))
    rng = np.random.default_rng(700)
    for rho in (0.001, 0.01):
        announce(f"transformer 110M global rho={rho}")
        g, r = to_dev(grads, dev), [torch.zeros(n, device=dev) for n in sizes]
        plan = tk.SparsifyPlan(sizes, rho=rho)
        plan.bind(g, r)
        idx, val = plan.execute()
        torch.cuda.synchronize()
        idx, val = idx.cpu().numpy(), val.cpu().numpy()
        check_selection(x, idx, val, gen.concat(to_host(r)), plan.k_total)
        _sampled_ranks(x, idx, plan.k_total, rng)
        del g, r
    for rho in (0.001, 0.01):
        announce(f"transformer 110M per-tensor rho={rho}")
        g, r = to_dev(grads, dev), [torch.zeros(n, device=dev) for n in sizes]
        plan = tk.SparsifyPlan(sizes, mode=tk.PER_TENSOR, rho=rho)
        plan.bind(g, r)
        idx, val = plan.execute()
        torch.cuda.synchronize()
        idx, val = idx.cpu().numpy(), val.cpu().numpy()
        rr = to_host(r)
        ks = plan.group_k()
        assert ks == [tk.k_from_rho(n, rho) for n in sizes]
        off, pos = 0, 0
        for t, n in enumerate(sizes):
            check_selection(x[off:off + n], idx[pos:pos + ks[t]], val[pos:pos + ks[t]], rr[t],
                            ks[t], base=off)
            off += n
            pos += ks[t]
        assert pos == idx.size
        del g, r


def test_bert_large_340m_tie_stressed():
    import torch
    dev = need_gpu()
    n = gen.BERT_LARGE_D
    announce("bert-large 340M tie-stressed: generate")
    x = gen.tie_stressed(n)
    k = 340_000
    a32 = np.float32(gen.NORMAL_TAIL_0P001)
    above = int(np.count_nonzero(np.abs(x) > a32))
    ties = int(np.count_nonzero(np.abs(x) == a32))
    assert above < k < above + ties, (above, ties)   # the tie class straddles k
    announce("bert-large 340M tie-stressed: run")
    g = to_dev([x], dev)
    r = [torch.zeros(n, device=dev)]
    plan = tk.SparsifyPlan([n], rho=0.001)
    plan.bind(g, r)
    idx, val = plan.execute()
    torch.cuda.synchronize()
    del g
    idx, val = idx.cpu().numpy(), val.cpu().numpy()
    rr = r[0].cpu().numpy()
    del r
    xs = orc().ef_add(x, np.zeros(n, np.float32))
    del x
    check_selection(xs, idx, val, rr, k)
    assert np.abs(val).min() == a32
    x = xs
    rng = np.random.default_rng(800)
    _sampled_ranks(x, idx, k, rng, nsamp=3)


@pytest.mark.parametrize("mode", [tk.GLOBAL, tk.PER_TENSOR])
def test_ragged_list_between_one_and_two_units_per_workgroup(mode):
    """A ragged list of 2.8 M elements (1,025 to 2,048 stream units: some
    workgroups of the stream take two units, others one), global and per
    tensor, where a workgroup's units can belong to different tensors."""
    rng = np.random.default_rng(700 + mode)
    sizes = [2_500_000, 777, 8193, 1, 300_000]
    grads = [rng.standard_normal(n).astype(np.float32) for n in sizes]
    res = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    units = sum(-(-n // 8192) for n in sizes) * 4
    assert 1024 < units <= 2048
    compare_with_oracle(grads, res, rho=0.001, mode=mode, label="2.8 M ragged")
    if mode == tk.GLOBAL:
        compare_with_oracle(grads, res, k=250_000, label="2.8 M ragged, large k")


@pytest.mark.parametrize("rho", [0.01, 0.05])
def test_dense_selection_band_beyond_lds(rho):
    """A dense selection on 10 M N(0, 1) elements: at rho = 0.05 a region of
    the global selection holds about 8 K members of the threshold's level-1
    bin, more than its workgroup keeps in LDS, so they are placed from a
    second read of its lines."""
    rng = np.random.default_rng(int(rho * 1000))
    n = 10_000_000
    g = rng.standard_normal(n).astype(np.float32)
    r = (rng.standard_normal(n) * 0.01).astype(np.float32)
    compare_with_oracle([g], [r], rho=rho, label=f"dense rho={rho}")


@pytest.mark.parametrize("case", ["one_region", "two_regions_ties", "every_region"])
def test_band_beyond_region_capacity(case):
    """One exact selection over 2^20 elements (16 regions of 65,536 for the
    selection kernels, each storing at most 4,608 candidates at k = 1,000 or
    3,500) where one or two regions hold 6,000-10,000 members of the
    threshold's level-1 bin: those regions store neither their candidates nor
    their band, and every later step reads their lines instead. With ties:
    the band takes its magnitudes from 700 values, so the threshold class is
    split by position. Every region: all sixteen hold 6,000 band members."""
    rng = np.random.default_rng({"one_region": 4242, "two_regions_ties": 4343}.get(case, 4444))
    n = 1 << 20
    g = (rng.standard_normal(n) * 0.1).astype(np.float32)
    top = rng.choice(n, 500, replace=False)
    g[top] = (10 + rng.random(500)).astype(np.float32) * rng.choice([-1, 1], 500)
    if case == "one_region":
        pos = 3 * 65536 + rng.choice(65536, 10_000, replace=False)
        g[pos] = (5 + 0.5 * rng.random(pos.size)).astype(np.float32) * rng.choice([-1, 1], pos.size)
        k = 1000
    elif case == "every_region":
        pos = np.concatenate([q * 65536 + rng.choice(65536, 6000, replace=False)
                              for q in range(16)])
        g[pos] = (5 + 0.5 * rng.random(pos.size)).astype(np.float32) * rng.choice([-1, 1], pos.size)
        k = 1000
    else:
        vals = (5 + 0.5 * rng.random(700)).astype(np.float32)
        pos = np.concatenate([3 * 65536 + rng.choice(65536, 6000, replace=False),
                              9 * 65536 + rng.choice(65536, 6000, replace=False)])
        g[pos] = rng.choice(vals, pos.size) * rng.choice([-1, 1], pos.size).astype(np.float32)
        k = 3500
    r = np.zeros(n, np.float32)
    compare_with_oracle([g], [r], k=k, label=f"band beyond region capacity ({case})")


@pytest.mark.parametrize("levels", [3, 50])
def test_dense_regions_with_ties_across_rounds(levels):
    """2^21 elements whose magnitudes take only `levels` values, k = 150,000:
    each of the 32 selection regions stores several thousand candidates,
    taken by the finish kernel in rounds of one candidate per thread, and the
    threshold class (tens of thousands of equal magnitudes, split by
    position) runs through many rounds of every region."""
    rng = np.random.default_rng(9100 + levels)
    n = 1 << 21
    mags = np.sort(rng.random(levels).astype(np.float32) + np.float32(0.5))
    g = (mags[rng.integers(0, levels, n)] * rng.choice([-1, 1], n)).astype(np.float32)
    r = np.zeros(n, np.float32)
    idx, val, _ = compare_with_oracle([g], [r], k=150_000,
                                      label=f"dense ties across rounds ({levels} levels)")
    # the threshold class is split: some of its members are taken, some not
    T = np.abs(val).min()
    taken = np.count_nonzero(np.abs(val) == T)
    assert 0 < taken < np.count_nonzero(np.abs(g) == T)


def test_large_regions_with_ties_across_rounds():
    """40 M elements, k = 200,000, values N(0, 1) rounded to multiples of
    1/64: above 2^20 summary lines and with k < d / 160 the selection runs
    1,024-thread workgroups (153 regions), each storing about 1,500
    candidates, which the finish kernel takes in two rounds; the threshold
    class (thousands of equal magnitudes) is split by position. Checked
    through the exact selection properties against the oracle's x."""
    import torch
    dev = need_gpu()
    rng = np.random.default_rng(9200)
    n = 40_000_000
    g = (np.round(rng.standard_normal(n) * 64) / 64).astype(np.float32)
    announce("sparsify 40M quantized k=200000")
    gd, rd = torch.from_numpy(g).to(dev), torch.zeros(n, device=dev)
    plan = tk.SparsifyPlan([n], k=200_000).bind([gd], [rd])
    idx, val = plan.execute()
    torch.cuda.synchronize()
    idx, val = idx.cpu().numpy(), val.cpu().numpy()
    x = orc().ef_add(g, np.zeros(n, np.float32))
    check_selection(x, idx, val, rd.cpu().numpy(), 200_000)
    T = np.abs(val).min()
    assert 0 < np.count_nonzero(np.abs(val) == T) < np.count_nonzero(np.abs(x) == T)
