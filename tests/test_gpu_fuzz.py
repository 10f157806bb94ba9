"""GPU parity on seeded random configurations: ragged tensor lists (sizes
around tile and line boundaries, empty tensors), several value distributions
(normal, heavy ties, zeros and signed zeros, subnormals, wide exponent
spread), random residuals, every selection mode and both value formats,
each compared bit for bit with the oracle (exact selection) or the MSTopK
oracle (TKEF_APPROX)."""
import numpy as np
import pytest

import gen
import oracle
import oracle.mstopk as ms
import paper_2010_10458_amd as tk
from gpu_common import announce, assert_bitwise, need_gpu, to_dev, to_host

pytestmark = pytest.mark.gpu

EDGE_SIZES = [0, 1, 2, 31, 32, 33, 1023, 4096, 8191, 8192, 8193, 16_385, 40_000, 131_072]


def draw_values(rng, n, kind):
    if kind == "normal":
        return rng.standard_normal(n).astype(np.float32)
    if kind == "ties":
        return (rng.integers(-6, 7, n) * 0.25).astype(np.float32)
    if kind == "zeros":
        z = np.zeros(n, np.float32)
        z[rng.random(n) < 0.5] = -0.0
        z[rng.random(n) < 0.01] = 1.5
        return z
    if kind == "subnormal":
        return (rng.standard_normal(n) * 1e-41).astype(np.float32)
    # wide: magnitudes spread over most of the binary32 exponent range
    return (rng.standard_normal(n) * np.exp2(rng.integers(-120, 120, n))).astype(np.float32)


def case(seed):
    rng = np.random.default_rng(9000 + seed)
    T = int(rng.integers(1, 9))
    sizes = [int(rng.choice(EDGE_SIZES)) if rng.random() < 0.6 else int(rng.integers(1, 300_000))
             for _ in range(T)]
    if sum(sizes) == 0:
        sizes[0] = 1
    kind = ["normal", "ties", "zeros", "subnormal", "wide"][seed % 5]
    grads = [draw_values(rng, n, kind) for n in sizes]
    res = [(draw_values(rng, n, "normal") * np.float32(rng.choice([0.0, 0.1, 10.0])))
           .astype(np.float32) for n in sizes]
    mode = [tk.GLOBAL, tk.PER_TENSOR, tk.APPROX][seed % 3]
    rho = float(rng.choice([0.0005, 0.001, 0.01, 0.1, 0.5, 1.0]))
    f16 = seed % 4 == 3
    return sizes, grads, res, mode, rho, f16, int(rng.integers(0, 2**63)), int(rng.integers(1, 49))


@pytest.mark.parametrize("seed", range(96))
def test_fuzz(seed):
    import torch
    from oracle import f16_rne
    sizes, grads, res, mode, rho, f16, word, n_search = case(seed)
    announce(f"fuzz seed={seed} sizes={sizes} mode={mode} rho={rho} f16={f16} N={n_search}")
    dev = need_gpu()
    g_d, r_d = to_dev(grads, dev), to_dev(res, dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    vdt = torch.float16 if f16 else torch.float32
    if mode == tk.APPROX:
        plan = tk.SparsifyPlan(sizes, mode=mode, rho=rho, n_search=n_search, val_dtype=vdt)
        plan.bind(g_d, r_d)
        idx, val = plan.execute(status=status, window_word=word)
    else:
        plan = tk.SparsifyPlan(sizes, mode=mode, rho=rho, val_dtype=vdt)
        plan.bind(g_d, r_d)
        idx, val = plan.execute(status=status)
    torch.cuda.synchronize()
    idx, val = idx.cpu().numpy(), val.cpu().numpy()
    r_out = gen.concat(to_host(r_d))
    g, r = gen.concat(grads), gen.concat(res)
    if mode == tk.APPROX:
        oi, ov, orr, tr = ms.mstopk_sparsify(g, r, plan.k_total, n_search, word)
        assert int(status.item()) == 0
    else:
        oi, ov, orr_t, ks = oracle.Oracle().sparsify(
            grads, res, rho=rho,
            mode=oracle.GLOBAL if mode == tk.GLOBAL else oracle.PER_TENSOR)
        orr = gen.concat([a.ravel() for a in orr_t])
        assert plan.k_total == sum(ks)
        assert int(status.item()) == 0
    assert_bitwise(idx, oi, "idx")
    if f16:
        assert np.array_equal(val.view(np.uint16), f16_rne(ov).view(np.uint16)), "val (f16)"
    else:
        assert_bitwise(val, ov, "val")
    assert_bitwise(r_out, orr, "residual")


@pytest.mark.parametrize("seed", range(24))
def test_fuzz_update(seed):
    """Random sparse aggregate + update: ragged parameter lists (tensors that
    do not fill a tile, sizes not a multiple of four), P workers with ragged
    ascending lists (repeated indices within and across workers, empty
    lists), plain SGD or momentum with weight decay."""
    from test_gpu_update import compare
    rng = np.random.default_rng(9500 + seed)
    T = int(rng.integers(1, 7))
    sizes = [int(rng.choice([1, 3, 4095, 4096, 4097, 10_001])) if rng.random() < 0.5
             else int(rng.integers(1, 120_000)) for _ in range(T)]
    d = sum(sizes)
    P = int(rng.integers(1, 200))
    stride = int(rng.integers(1, 3000))
    idx = np.sort(rng.integers(0, d, (P, stride)), axis=1).astype(np.int32)
    val = (rng.standard_normal((P, stride)) * 1e-2).astype(np.float32)
    nnz = rng.integers(0, stride + 1, P).astype(np.int32)
    nnz[rng.random(P) < 0.1] = 0
    w0 = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    mom = seed % 2 == 1
    b0 = [(rng.standard_normal(n) * 0.01).astype(np.float32) for n in sizes] if mom else None
    lr = float(rng.choice([0.1, 0.5, 1.0]))
    mu, wd = (0.9, 5e-5) if mom else (0.0, 0.0)
    compare(sizes, w0, b0, idx, val, lr, mu, wd, nnz=nnz, label=f"fuzz seed={seed} d={d}")
