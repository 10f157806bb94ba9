"""The MSTopK oracle (Alg. 1) against its pins, and pin strength: plausible
mistakes planted in a copy of the oracle source (on the CPU) must each fail
at least one pin. Each mutant replaces exact snippets of
``oracle/mstopk.py``; each snippet's presence is checked first."""
import importlib.util

import pytest

import oracle.mstopk as ms
from mstopk_pins import ALL_MS_PINS


@pytest.mark.parametrize("pin", ALL_MS_PINS, ids=[p.__name__ for p in ALL_MS_PINS])
def test_ms_pin(pin):
    pin(ms)


MUTANTS = {
    "thres1_starts_at_zero": [("k1, thres1 = 0, math.inf", "k1, thres1 = 0, 0.0")],
    "mean_of_signed_x": [("abar = math.fsum(a.tolist()) / d",
                          "abar = math.fsum(x.astype(np.float64).tolist()) / d")],
    "mean_float32_sum": [("abar = math.fsum(a.tolist()) / d",
                          "abar = float(np.sum(np.abs(x), dtype=np.float32)) / d")],
    "ratio_endpoint": [("ratio = math.ldexp(2 * path + 1, -n)",
                        "ratio = math.ldexp(2 * path, -n)")],
    "thres_from_zero": [("thres = abar + ratio * (u - abar)", "thres = ratio * u")],
    "strict_count": [('side="left"', 'side="right"')],
    "count_equal_to_k_not_low": [("if 0 < c <= k]", "if 0 < c < k]"),
                                 ("if k < c < d]", "if k <= c < d]")],
    "k1_record_last_trial": [("thres1 = next(t for c, t in low if c == k1)",
                              "thres1 = [t for c, t in low if c == k1][-1]")],
    "k2_kept_largest": [("k2 = min(c for c, _ in high)", "k2 = max(c for c, _ in high)")],
    "bounds_swapped": [("(1 if count > k else 0)", "(0 if count > k else 1)")],
    "band_includes_top": [("band = (a >= thres2) & ~top", "band = a >= thres2")],
    "offset_ignored": [("offset = int(window_word) % (nband - take + 1)", "offset = 0")],
    "offset_closed_interval": [("offset = int(window_word) % (nband - take + 1)",
                                "offset = int(window_word) % max(1, nband - take)")],
    "window_from_end": [("(rank >= offset) & (rank < offset + take)", "(rank >= nband - take)")],
    "band_listed_first": [("iota = np.flatnonzero(top | window).astype(np.int64)",
                           "iota = np.concatenate([np.flatnonzero(window), np.flatnonzero(top)]).astype(np.int64)")],
    "residual_kept": [("r_out[iota] = np.float32(0.0)", "pass")],
    "value_from_gradient": [("return (iota + index_base).astype(np.int32), val, r_out, trace",
                             "return (iota + index_base).astype(np.int32), g[iota], r_out, trace")],
    "one_round_less": [("for n in range(1, n_search + 1):", "for n in range(1, n_search):")],
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_ms_mutant_is_caught(name, tmp_path):
    src = open(ms.__file__).read()
    for old, new in MUTANTS[name]:
        assert src.count(old) >= 1, f"snippet for {name} not found in the oracle source"
        src = src.replace(old, new, 1)
    path = tmp_path / f"ms_{name}.py"
    path.write_text(src)
    spec = importlib.util.spec_from_file_location(f"ms_mutant_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    for pin in ALL_MS_PINS:
        try:
            pin(mod)
        except Exception:  # noqa: BLE001 - any failure counts as caught
            return
    raise AssertionError(f"mutant {name} passed every pin")
