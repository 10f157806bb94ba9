"""GPU parity: MSTopK (Alg. 1, TKEF_APPROX plans) through the C ABI against
the float64 oracle in oracle/mstopk.py.

Both sides take the mean as the exact sum of |x| rounded once to double and
divided by d, form every trial threshold with the same double operations and
compare magnitudes exactly, so for the same window word the index list, the
values and the residual match bit for bit, and so do the recorded counts k1,
k2, the window offset and the threshold keys.
"""
import numpy as np
import pytest

import gen
import oracle.mstopk as ms
import paper_2010_10458_amd as tk
from gpu_common import announce, assert_bitwise, need_gpu, to_dev, to_host

pytestmark = pytest.mark.gpu


def key_ceil(t: float) -> int:
    """Bits (sign cleared) of the smallest binary32 >= t, t >= 0."""
    if t == np.inf:
        return 1 << 31
    if t <= 0:
        return 0
    f = np.float32(t)
    if float(f) < t:
        f = np.nextafter(f, np.float32(np.inf))
    return int(np.array(f, np.float32).view(np.uint32))


def run_gpu(grads, residuals, k, n_search, word, val_dtype=None, rho=None):
    import torch
    dev = need_gpu()
    g = to_dev(grads, dev)
    r = to_dev(residuals, dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    plan = tk.SparsifyPlan([a.size for a in grads], mode=tk.APPROX, k=k, rho=rho,
                           n_search=n_search, val_dtype=val_dtype or torch.float32)
    plan.bind(g, r)
    idx, val = plan.execute(status=status, window_word=word)
    torch.cuda.synchronize()
    res = plan.approx_result()
    return idx.cpu().numpy(), val.cpu().numpy(), to_host(r), int(status.item()), res, plan


def compare(grads, residuals, k, n_search=30, word=0, label="", rho=None):
    sizes = [a.size for a in grads]
    announce(f"mstopk {label} sizes={sizes[:6]} k={k} rho={rho} N={n_search} word={word}")
    idx, val, r, status, res, plan = run_gpu(grads, residuals, k, n_search, word, rho=rho)
    kk = plan.k_total
    g = gen.concat(grads) if len(grads) > 1 else grads[0].ravel()
    rr = gen.concat(residuals) if len(residuals) > 1 else residuals[0].ravel()
    oi, ov, orr, tr = ms.mstopk_sparsify(g, rr, kk, n_search, word)
    assert status == 0
    assert res["mean"] == tr.abar and res["u"] == tr.u, (res, tr.abar, tr.u)
    assert (res["k1"], res["k2"], res["offset"], res["take"]) == (tr.k1, tr.k2, tr.rand,
                                                                 kk - tr.k1), (res, tr)
    assert res["key1"] == key_ceil(tr.thres1) and res["key2"] == key_ceil(tr.thres2), (res, tr)
    assert_bitwise(idx, oi, "idx")
    assert_bitwise(val, ov, "val")
    assert_bitwise(gen.concat(r), orr, "residual")
    return idx, tr


SIZES = [1, 2, 7, 33, 1000, 8191, 8193, 3 * 8192 + 5, 100_003, 1_000_001]


@pytest.mark.parametrize("n", SIZES)
def test_flat_sizes(n):
    rng = np.random.default_rng(300 + n)
    g = rng.standard_normal(n).astype(np.float32)
    r = (rng.standard_normal(n) * 0.3).astype(np.float32)
    for k in sorted({1, max(1, n // 1000), max(1, n // 10), n}):
        compare([g], [r], k, word=int(rng.integers(0, 2**63)), label=f"normal n={n}")


@pytest.mark.parametrize("n_search", [1, 5, 6, 7, 12, 13, 18, 19, 30, 31, 42, 48])
def test_rounds(n_search):
    rng = np.random.default_rng(400 + n_search)
    n = 200_003
    g = rng.standard_normal(n).astype(np.float32)
    g[rng.random(n) < 0.01] *= 50
    compare([g], [np.zeros(n, np.float32)], 211, n_search=n_search, word=12345,
            label=f"rounds {n_search}")


def test_ragged_tensor_list_and_window_words():
    rng = np.random.default_rng(41)
    sizes = [1, 5, 64, 8193, 100, 30_000, 0, 17, 16_384, 3]
    grads = [rng.standard_normal(s).astype(np.float32) for s in sizes]
    res = [(rng.standard_normal(s) * 0.1).astype(np.float32) for s in sizes]
    for word in (0, 1, 2**63 - 1, 2**64 - 1):
        compare(grads, res, 55, word=word, label="ragged list")


def test_hand_worked_cases():
    import json
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "mstopk_worked.json")
    for c in json.load(open(path))["cases"]:
        x = np.array(c["x"], np.float32)
        idx, tr = compare([x], [np.zeros_like(x)], c["k"], n_search=c["n_search"],
                          word=c["window_word"], label=c["name"])
        assert idx.tolist() == c["iota"]


def test_ties_equal_magnitudes_and_k_equals_d():
    rng = np.random.default_rng(42)
    n = 70_001
    x = np.where(rng.random(n) < 0.5, -0.75, 0.75).astype(np.float32)
    for word in (0, 5, 2**40 + 3):
        compare([x], [np.zeros(n, np.float32)], 1234, word=word, label="all equal")
    levels = rng.integers(0, 6, n).astype(np.float32) * 0.5
    compare([levels], [np.zeros(n, np.float32)], 9000, word=77, label="few levels")
    compare([levels], [np.zeros(n, np.float32)], n, word=77, label="k = d")
    z = np.zeros(n, np.float32)
    compare([z], [z.copy()], 10, word=3, label="all zero")


def test_denormal_and_huge_magnitudes():
    rng = np.random.default_rng(43)
    n = 50_000
    x = (rng.standard_normal(n) * 1e-40).astype(np.float32)   # subnormal range
    compare([x], [np.zeros(n, np.float32)], 50, word=9, label="subnormal")
    y = (rng.standard_normal(n) * 1e37).astype(np.float32)
    y[:3] = [3.4e38, -3.3e38, 3.0e38]
    compare([y], [np.zeros(n, np.float32)], 50, word=9, label="near FLT_MAX")


def test_nonfinite_sets_status_and_takes_first_k():
    import torch
    n = 10_000
    x = np.ones(n, np.float32)
    x[17] = np.inf
    announce("mstopk non-finite")
    idx, val, r, status, res, _ = run_gpu([x], [np.zeros(n, np.float32)], 5, 30, 1)
    assert status & tk.STATUS_NONFINITE
    assert idx.tolist() == [0, 1, 2, 3, 4]


def test_resnet50_step_with_residual_carry():
    """The ResNet-50-shaped gradient set (161 tensors, 25,557,032 elements),
    rho = 0.001, N = 30, two steps with the residual carried on each side."""
    import torch
    dev = need_gpu()
    sizes = gen.numels(gen.resnet50_shapes())
    res_h = [np.zeros(n, np.float32) for n in sizes]
    res_d = to_dev(res_h, dev)
    plan = tk.SparsifyPlan(sizes, mode=tk.APPROX, rho=0.001)
    r_or = gen.concat(res_h)
    for step in range(2):
        grads = gen.resnet_grads(step)
        announce(f"mstopk resnet50 step {step}")
        g_d = to_dev(grads, dev)
        plan.bind(g_d, res_d)
        status = torch.zeros(1, dtype=torch.int32, device=dev)
        word = 1000 + step
        idx, val = plan.execute(status=status, window_word=word)
        torch.cuda.synchronize()
        oi, ov, r_or, tr = ms.mstopk_sparsify(gen.concat(grads), r_or, plan.k_total, 30, word)
        assert int(status.item()) == 0
        assert_bitwise(idx.cpu().numpy(), oi, "idx")
        assert_bitwise(val.cpu().numpy(), ov, "val")
        assert_bitwise(gen.concat(to_host(res_d)), r_or, "residual")


def test_fp16_values_and_shard_shape():
    """One shard of the eight-way split of the ResNet-50 gradient (k~ = 3,195)
    with binary16 values."""
    import torch
    from oracle import f16_rne
    d, n = gen.RESNET50_D, 8
    shard = -(-d // n)
    g = gen.flat_normal(shard, config=2, std=1e-2)
    r = gen.flat_normal(shard, config=2, step=1, std=1e-3)
    k = -(-d // (n * 1000))
    announce(f"mstopk shard fp16 d={shard} k={k}")
    idx, val, rr, status, res, _ = run_gpu([g], [r], k, 30, 99, val_dtype=torch.float16)
    oi, ov, orr, tr = ms.mstopk_sparsify(g, r, k, 30, 99)
    assert status == 0
    assert_bitwise(idx, oi, "idx")
    assert np.array_equal(val.view(np.uint16), f16_rne(ov).view(np.uint16))
    assert_bitwise(rr[0], orr, "residual")
