"""GPU parity: LARS (Eq. lars rates and the cited method's step) through the
C ABI against the oracle in oracle/lars.py (rates in double, step in
binary32) and the C oracle's worker-ordered aggregate for the gradient.

Rates: both sides sum the squares of binary32 values in double; the oracle
rounds the exact sum once, the GPU adds a few hundred terms per partial in a
fixed order, which accounts for well under 1e-12 relative. The gradient
itself may differ where a position has three or more contributions (the GPU
sums them in another order): |dG_i| <= 2 (c_i - 1) 2^-24 sum|v|_i, so
||g|| moves by at most ||dG||, and the rate (inversely proportional to
||g|| + eps ||w||) by the factor ||dG|| / (||g|| + eps ||w||). The bound is
the sum of the two. Step: where the binary32 rates agree (always when no
position has three contributions), positions with at most two contributions
match bit for bit (same argument as the plain update); every position lies
within 1e-6 (|w_ref| + S), S = rate (sum |v| + eps |w|) + mu |b|. Dyadic
layers built so that the rate is exactly 2 match bit for bit everywhere.
"""
import numpy as np
import pytest

import gen
import oracle
import oracle.lars as lars
import paper_2010_10458_amd as tk
from gpu_common import announce, assert_bitwise, need_gpu, to_dev, to_host

pytestmark = pytest.mark.gpu

ORC = None


def orc():
    global ORC
    if ORC is None:
        ORC = oracle.Oracle()
    return ORC


def split(flat, sizes):
    return np.split(np.asarray(flat), np.cumsum(sizes)[:-1])


def check_rates(got, ref, what, extra=None):
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    assert got.shape == ref.shape
    rel = 1e-12 + (0.0 if extra is None else np.asarray(extra))
    bad = np.abs(got - ref) > rel * np.abs(ref)
    assert not bad.any(), f"{what}: rates differ at {np.nonzero(bad)[0][:5]}: {got[bad][:3]} vs {ref[bad][:3]}"


def run_lars(sizes, w_host, b_host, idx, val, gamma, eta, eps, mu, nnz=None, val_dtype=None):
    import torch
    dev = need_gpu()
    w = to_dev(w_host, dev)
    b = to_dev(b_host, dev) if b_host is not None else None
    P, stride = idx.shape
    plan = tk.UpdatePlan(sizes, P=P, stride=stride, val_dtype=val_dtype or torch.float32)
    plan.bind(w, b)
    it = torch.from_numpy(np.ascontiguousarray(idx, np.int32)).to(dev)
    vt = torch.from_numpy(np.ascontiguousarray(val)).to(dev)
    nt = torch.from_numpy(np.asarray(nnz, np.int32)).to(dev) if nnz is not None else None
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    rates = plan.lars_execute(it, vt, gamma, eta, eps, mu=mu, nnz=nt, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    return to_host(w), (to_host(b) if b is not None else None), rates.cpu().numpy()


def compare_lars(sizes, w0, b0, idx, val, gamma, eta, eps, mu, nnz=None, exact=False, label="",
                 val_dtype=None):
    announce(f"lars {label} T={len(sizes)} P={idx.shape[0]} stride={idx.shape[1]} mu={mu}")
    wg, bg, rg = run_lars(sizes, w0, b0, idx, val, gamma, eta, eps, mu, nnz, val_dtype)
    d = sum(sizes)
    G = orc().aggregate(d, idx, np.asarray(val).astype(np.float32),
                        None if nnz is None else np.asarray(nnz, np.int64))
    Gs = split(G, sizes)
    w_ref, b_ref, r_ref = lars.lars_update(w0, b0, Gs, gamma, eta, eps, mu)
    P, stride = idx.shape
    nn = np.full(P, stride) if nnz is None else np.clip(np.asarray(nnz), 0, stride)
    flat_i = np.concatenate([idx[p, :nn[p]] for p in range(P)]).astype(np.int64)
    flat_v = np.concatenate([np.asarray(val)[p, :nn[p]] for p in range(P)]).astype(np.float64)
    cnt = np.bincount(flat_i, minlength=d)
    A = np.zeros(d)
    np.add.at(A, flat_i, np.abs(flat_v))
    dG = 2 * np.maximum(cnt - 1, 0) * 2.0 ** -24 * A
    extra = []
    for t, Gt in enumerate(Gs):
        lo = int(np.sum(sizes[:t]))
        den = lars.layer_norm(Gt) + eps * lars.layer_norm(w0[t])
        nd = float(np.sqrt(np.sum(dG[lo:lo + sizes[t]] ** 2)))
        extra.append(1.01 * nd / den if den > 0 else 0.0)
    check_rates(rg, r_ref, "rates", extra)
    same32 = np.float32(rg) == np.float32(r_ref)
    for t, n in enumerate(sizes):
        if n == 0:
            continue
        lo = int(np.sum(sizes[:t]))
        sl = slice(lo, lo + n)
        wt, rt = wg[t], w_ref[t]
        if exact:
            assert_bitwise(wt, rt, f"w[{t}]")
            if b_ref is not None:
                assert_bitwise(bg[t], b_ref[t], f"b[{t}]")
            continue
        rate = float(r_ref[t])
        S = rate * (A[sl] + eps * np.abs(w0[t])) + (mu * np.abs(b0[t]) if b0 is not None else 0.0)
        assert np.all(np.abs(wt.astype(np.float64) - rt) <= 1e-6 * (np.abs(rt) + S)), f"w[{t}]"
        if b_ref is not None:
            assert np.all(np.abs(bg[t].astype(np.float64) - b_ref[t]) <= 1e-6 * (np.abs(b_ref[t]) + S)), f"b[{t}]"
        if same32[t]:
            le2 = cnt[sl] <= 2
            assert_bitwise(wt[le2], rt[le2], f"w[{t}] (<= 2 contributions)")
            if b_ref is not None:
                assert_bitwise(bg[t][le2], b_ref[t][le2], f"b[{t}] (<= 2 contributions)")
    return rg


def _lists(rng, d, P, k, std=1e-2):
    idx = np.stack([np.sort(rng.choice(d, size=k, replace=False)) for _ in range(P)]).astype(np.int32)
    val = (rng.standard_normal((P, k)) * std).astype(np.float32)
    return idx, val


@pytest.mark.parametrize("mom", [False, True])
def test_lars_ragged_sizes(mom):
    rng = np.random.default_rng(81 + mom)
    sizes = [1, 5, 64, 8193, 100, 30_000, 0, 17, 16_384, 3, 4096, 4097]
    d = sum(sizes)
    w0 = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    b0 = [(rng.standard_normal(n) * 0.01).astype(np.float32) for n in sizes] if mom else None
    for P in (1, 7):
        idx, val = _lists(rng, d, P, d // 20)
        compare_lars(sizes, w0, b0, idx, val, 0.001, 0.1, 5e-5, 0.9 if mom else 0.0,
                     label=f"ragged P={P}")


def test_lars_zero_layers_and_ragged_nnz():
    """Eq. (lars) at zero norms: tensor 1 has w = 0 and a gradient (rate 0),
    tensor 2 gets no gradient (rate gamma eta / eps), tensor 4 has neither
    (a zero denominator: rate 0); ragged list lengths."""
    rng = np.random.default_rng(83)
    sizes = [300, 5000, 77, 4096, 64]
    off = np.concatenate([[0], np.cumsum(sizes)])
    d = sum(sizes)
    w0 = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    w0[1][:] = 0.0
    w0[4][:] = 0.0
    idx, val = _lists(rng, d, 4, 400)
    in_t = lambda t: (idx >= off[t]) & (idx < off[t + 1])  # noqa: E731
    val = np.where(in_t(2) | in_t(4), 0.0, val).astype(np.float32)
    nnz = [400, 0, 123, 399]
    rates = compare_lars(sizes, w0, None, idx, val, 0.01, 0.5, 1e-4, 0.0, nnz=nnz,
                         label="zero layers")
    got_g1 = any(np.any(in_t(1)[p, :nnz[p]] & (val[p, :nnz[p]] != 0)) for p in range(4))
    assert got_g1
    assert rates[1] == 0.0 and rates[4] == 0.0
    assert abs(rates[2] - 0.01 * 0.5 / 1e-4) <= 1e-12 * rates[2]


def test_lars_dyadic_rate_two_bit_exact():
    """Layers of 16, 4096 and 16384 positions with w = +-2 and a summed
    gradient of +-1/2 (two workers of +-1/4): ||w|| = 2 sqrt(n), ||g|| =
    sqrt(n) / 2, eps = 1/4, gamma = eta = 1, so the rate is exactly 2 and
    every binary32 operation of the step is exact."""
    sizes = [16, 4096, 16384]
    d = sum(sizes)
    sgn = np.where(np.arange(d) % 3 == 0, -1.0, 1.0)
    w0 = split((2.0 * sgn).astype(np.float32), sizes)
    b0 = split(np.where(np.arange(d) % 5 == 0, 0.5, -0.25).astype(np.float32), sizes)
    idx = np.stack([np.arange(d), np.arange(d)]).astype(np.int32)
    val = np.stack([0.25 * sgn, 0.25 * sgn]).astype(np.float32)
    rates = compare_lars(sizes, w0, None, idx, val, 1.0, 1.0, 0.25, 0.0, exact=True,
                         label="dyadic plain")
    assert np.all(rates == 2.0)
    compare_lars(sizes, w0, b0, idx, val, 1.0, 1.0, 0.25, 0.5, exact=True, label="dyadic momentum")


def test_lars_resnet50_p128_momentum():
    """The update workload (P = 128 lists of 25,600 pairs into ResNet-50-
    shaped parameters) with the LARS step: gamma 0.001, eta 0.1 (the global
    rate), eps 5e-5, momentum 0.9."""
    sizes = gen.numels(gen.resnet50_shapes())
    d = sum(sizes)
    w0 = gen.params_like(sizes, config=5)
    b0 = [np.zeros(n, np.float32) for n in sizes]
    idx, val = gen.sparse_lists(d, 128, 25_600, step=0)
    compare_lars(sizes, w0, b0, idx, val, 0.001, 0.1, 5e-5, 0.9, label="resnet50 P=128")


@pytest.mark.parametrize("mom", [False, True])
def test_lars_binary16_values(mom):
    """binary16 values on the wire, widened exactly and summed in binary32:
    the same tolerance (and bit-exact positions) as the binary32 lists."""
    import torch
    rng = np.random.default_rng(84 + mom)
    sizes = [50_000, 333, 8192]
    d = sum(sizes)
    idx, val = _lists(rng, d, 6, 3000, std=0.1)
    v16 = oracle.f16_rne(val)
    w0 = [(rng.standard_normal(n) * 0.1).astype(np.float32) for n in sizes]
    b0 = [(rng.standard_normal(n) * 0.01).astype(np.float32) for n in sizes] if mom else None
    compare_lars(sizes, w0, b0, idx, v16, 0.001, 0.1, 5e-5, 0.9 if mom else 0.0,
                 label="binary16 values", val_dtype=torch.float16)


@pytest.mark.parametrize("model", ["resnet50", "transformer"])
def test_lars_rates_dense(model):
    """The rates alone from dense w and g (random, as the paper measures them):
    the ResNet-50 list (161 layers) and the Transformer list (261 layers)."""
    import torch
    dev = need_gpu()
    shapes = gen.resnet50_shapes() if model == "resnet50" else gen.transformer_shapes()
    sizes = gen.numels(shapes)
    rng = np.random.default_rng(85)
    w = [(rng.standard_normal(n) * 0.05).astype(np.float32) for n in sizes]
    g = [(rng.standard_normal(n) * 1e-3).astype(np.float32) for n in sizes]
    w[3][:] = 0.0
    announce(f"lars rates dense {model}")
    plan = tk.UpdatePlan(sizes, P=1, stride=0)
    wt, gt = to_dev(w, dev), to_dev(g, dev)
    plan.bind(wt)
    plan.bind_grads(gt)
    rates = plan.lars_rates(0.001, 0.1, 5e-5)
    torch.cuda.synchronize()
    check_rates(rates.cpu().numpy(), lars.lars_rates(w, g, 0.001, 0.1, 5e-5), model)
    # the parameters are only read
    assert all(np.array_equal(a, b) for a, b in zip(to_host(wt), w))
    # same inputs, same rates, bit for bit (fixed summation order)
    again = plan.lars_rates(0.001, 0.1, 5e-5)
    torch.cuda.synchronize()
    assert np.array_equal(again.cpu().numpy(), rates.cpu().numpy())
