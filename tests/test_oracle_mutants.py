"""Pin strength: plant plausible mistakes in a copy of the oracle source
(on the CPU) and require every such broken oracle to fail at least one pin.

Each mutant replaces one exact snippet of ``oracle/tkef_oracle.c``; the test
first checks that the snippet is present, so an edit of the oracle that
removes it fails loudly here instead of silently weakening the check.
"""
import os

import pytest

import oracle
from oracle_pins import ALL_PINS

MUTANTS = {
    "tie_break_higher_index": ("return (a < b) ? -1 : (a > b) ? 1 : 0;",
                               "return (a > b) ? -1 : (a < b) ? 1 : 0;"),
    "ascending_magnitude": ("if (ma > mb) return -1;\n    if (ma < mb) return 1;",
                            "if (ma < mb) return -1;\n    if (ma > mb) return 1;"),
    "signed_instead_of_magnitude": ("float ma = fabsf(x[a]), mb = fabsf(x[b]);",
                                    "float ma = x[a], mb = x[b];"),
    "no_residual_add": ("x[i] = g[i] + r[i];", "x[i] = g[i];"),
    "value_from_gradient": ("val_out[j] = x[sel[j]];", "val_out[j] = g[sel[j]];"),
    "residual_not_cleared": ("r_out[sel[j]] = +0.0f;", "(void)0;"),
    "residual_keeps_old": ("for (int64_t i = 0; i < n; ++i) r_out[i] = x[i];",
                           "for (int64_t i = 0; i < n; ++i) r_out[i] = r[i];"),
    "k_floor": ("double kd = ceil(rho * (double)d);", "double kd = floor(rho * (double)d);"),
    "k_round": ("double kd = ceil(rho * (double)d);", "double kd = round(rho * (double)d);"),
    "output_not_sorted": ("qsort(sel, (size_t)k, sizeof(int64_t), by_index);", "(void)by_index;"),
    "update_sign": ("w[i] = w[i] - step;\n        }\n    } else {",
                    "w[i] = w[i] + step;\n        }\n    } else {"),
    "mean_not_sum": ("G[i] = G[i] + val[(int64_t)p * stride + j];",
                     "G[i] = G[i] + val[(int64_t)p * stride + j] / (float)P;"),
    "first_worker_dropped": ("for (int32_t p = 0; p < P; ++p) {\n        for (int64_t j = 0; j < nnz[p]; ++j) {\n            int32_t i = idx[(int64_t)p * stride + j];\n            G[i]",
                             "for (int32_t p = 1; p < P; ++p) {\n        for (int64_t j = 0; j < nnz[p]; ++j) {\n            int32_t i = idx[(int64_t)p * stride + j];\n            G[i]"),
    "duplicate_overwrites": ("G[i] = G[i] + val[(int64_t)p * stride + j];",
                             "G[i] = val[(int64_t)p * stride + j];"),
    "momentum_mu_dropped": ("float keep = mu * b[i];", "float keep = b[i];"),
    "momentum_dampened": ("b[i] = keep + D;", "b[i] = keep + (1.0f - mu) * D;"),
    "weight_decay_dropped": ("float D = G[i] + decay;", "float D = G[i];"),
    "weight_decay_sign": ("float D = G[i] + decay;", "float D = G[i] - decay;"),
    "dense_lr_twice": ("float step = lr * U;", "float step = lr * lr * U;"),
    "plain_lr_dropped": ("float step = lr * G[i];", "float step = G[i];"),
    "nesterov": ("U = b[i];", "U = D + mu * b[i];"),
    "aggregate_overwrites": ("out[iq[j]] += vq[j];", "out[iq[j]] = vq[j];"),
    "aggregate_mean": ("out[iq[j]] += vq[j];", "out[iq[j]] += vq[j] / (float)P;"),
    "aggregate_not_zeroed": ("for (int64_t i = 0; i < d; ++i) out[i] = 0.0f;", "(void)0;"),
    "aggregate_first_worker_dropped": ("for (int32_t q = 0; q < P; ++q) {\n        const int32_t *iq",
                                       "for (int32_t q = 1; q < P; ++q) {\n        const int32_t *iq"),
    "aggregate_reverse_workers": ("for (int32_t q = 0; q < P; ++q) {\n        const int32_t *iq",
                                  "for (int32_t q = P - 1; q >= 0; --q) {\n        const int32_t *iq"),
    "aggregate_nnz_ignored": ("for (int64_t j = 0; j < nnz[q]; ++j) out", "for (int64_t j = 0; j < stride; ++j) out"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(oracle.SRC).read()
    assert src.count(old) >= 1, f"snippet for {name} not found in the oracle source"
    mutated = src.replace(old, new, 1)
    path = tmp_path / "mutant.c"
    path.write_text(mutated)
    lib = oracle.build(str(path), str(tmp_path / "libmutant.so"))
    orc = oracle.Oracle(oracle.load(lib))
    caught = []
    for pin in ALL_PINS:
        try:
            pin(orc)
        except Exception as exc:  # noqa: BLE001 - any failure counts as caught
            caught.append((pin.__name__, type(exc).__name__))
            break
    assert caught, f"mutant {name} passed every pin"
