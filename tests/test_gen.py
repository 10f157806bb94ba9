"""Seeded input generators: determinism and the workload shape recipes."""
import numpy as np

import gen


def test_shape_recipes():
    rn = gen.numels(gen.resnet50_shapes())
    assert len(rn) == 161 and sum(rn) == gen.RESNET50_D == 25_557_032
    assert max(rn) == 512 * 512 * 3 * 3 and min(rn) == 64
    tr = gen.numels(gen.transformer_shapes())
    assert sum(tr) == gen.TRANSFORMER_D == 109_708_544


def test_determinism_and_independence():
    a = gen.resnet_grads(step=3, sizes=[1000, 37])
    b = gen.resnet_grads(step=3, sizes=[1000, 37])
    c = gen.resnet_grads(step=4, sizes=[1000, 37])
    assert all(np.array_equal(x.view(np.uint32), y.view(np.uint32)) for x, y in zip(a, b))
    assert not np.array_equal(a[0], c[0])
    f1 = gen.flat_normal(3 << 20, config=1, chunk=1 << 20)
    f2 = gen.flat_normal(3 << 20, config=1, chunk=1 << 20)
    assert np.array_equal(f1, f2) and f1.dtype == np.float32


def test_outlier_mix():
    (g,) = gen.resnet_grads(step=0, sizes=[400_000])
    big = np.abs(g) > 0.2  # far beyond N(0, 1e-2), essentially only outliers
    frac = big.mean()
    assert 0.006 < frac < 0.0105
    assert abs(np.std(g[np.abs(g) < 0.05]) - 1e-2) < 1e-3


def test_tie_stressed_structure():
    n = 2_000_000
    x = gen.tie_stressed(n, band=0.05)
    a32 = np.float32(gen.NORMAL_TAIL_0P001)
    snapped = np.abs(x) == a32
    assert snapped.sum() > 100
    low16_zero = (x.view(np.uint32) & 0xFFFF) == 0
    assert 0.09 < low16_zero.mean() < 0.11


def test_sparse_lists_layout():
    idx, val = gen.sparse_lists(d=100_000, P=4, k=500)
    assert idx.shape == (4, 500) and idx.dtype == np.int32 and val.dtype == np.float32
    for p in range(4):
        assert np.all(np.diff(idx[p]) > 0) and idx[p].min() >= 0 and idx[p].max() < 100_000
