"""The MSTopK oracle (Alg. 1) against its pins, and pin strength: plausible
mistakes planted in a copy of the oracle source (on the CPU) must each fail
at least one pin. Each mutant replaces one exact snippet of
``oracle/mstopk.py``; the snippet's presence is checked first."""
import importlib.util

import pytest

import oracle.mstopk as ms
from mstopk_pins import ALL_MS_PINS


@pytest.mark.parametrize("pin", ALL_MS_PINS, ids=[p.__name__ for p in ALL_MS_PINS])
def test_ms_pin(pin):
    pin(ms)


MUTANTS = {
    "thres1_starts_at_zero": ("thres1, thres2 = math.inf, 0.0", "thres1, thres2 = 0.0, 0.0"),
    "mean_of_signed_x": ("abar = math.fsum(a.tolist()) / d",
                         "abar = math.fsum(x.astype(np.float64).tolist()) / d"),
    "mean_float32_sum": ("abar = math.fsum(a.tolist()) / d",
                         "abar = float(np.sum(np.abs(x), dtype=np.float32)) / d"),
    "ratio_drops_l": ("ratio = l + (r - l) / 2", "ratio = (r - l) / 2"),
    "thres_from_zero": ("thres = abar + ratio * (u - abar)", "thres = ratio * u"),
    "strict_count": ("nnz = int(np.count_nonzero(a >= thres))",
                     "nnz = int(np.count_nonzero(a > thres))"),
    "k1_always_updated": ("if nnz > k1:\n                k1 = nnz",
                          "if True:\n                k1 = nnz"),
    "k2_kept_largest": ("if nnz < k2:", "if nnz > k2 or k2 == d:"),
    "bounds_swapped": ("r = ratio\n", "l = ratio\n"),
    "band_includes_top": ("iota2 = np.flatnonzero((a < thres1) & (a >= thres2))",
                          "iota2 = np.flatnonzero(a >= thres2)"),
    "offset_ignored": ("rand = int(window_word) % (len(iota2) - take + 1)", "rand = 0"),
    "offset_closed_interval": ("rand = int(window_word) % (len(iota2) - take + 1)",
                               "rand = int(window_word) % max(1, len(iota2) - take)"),
    "window_from_end": ("iota2[rand:rand + take]", "iota2[len(iota2) - take:]"),
    "unsorted_output": ("iota = np.sort(np.concatenate([iota1, iota2[rand:rand + take]]))",
                        "iota = (np.concatenate([iota1, iota2[rand:rand + take]]))"),
    "residual_kept": ("r_out[iota] = np.float32(0.0)", "pass"),
    "value_from_gradient": ("return (iota + index_base).astype(np.int32), val, r_out, trace",
                            "return (iota + index_base).astype(np.int32), g[iota], r_out, trace"),
    "one_round_less": ("for _ in range(n_search):", "for _ in range(n_search - 1):"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_ms_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(ms.__file__).read()
    assert src.count(old) >= 1, f"snippet for {name} not found in the oracle source"
    path = tmp_path / f"ms_{name}.py"
    path.write_text(src.replace(old, new, 1))
    spec = importlib.util.spec_from_file_location(f"ms_mutant_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    for pin in ALL_MS_PINS:
        try:
            pin(mod)
        except Exception:  # noqa: BLE001 - any failure counts as caught
            return
    raise AssertionError(f"mutant {name} passed every pin")
