"""The LARS oracle (Eq. lars) against its pins, and pin strength: plausible
mistakes planted in a copy of ``oracle/lars.py`` (on the CPU) must each fail
at least one pin. The snippet of each mutant is checked to be present."""
import importlib.util

import pytest

import oracle.lars as lars
from lars_pins import ALL_LARS_PINS


@pytest.mark.parametrize("pin", ALL_LARS_PINS, ids=[p.__name__ for p in ALL_LARS_PINS])
def test_lars_pin(pin):
    pin(lars)


RATE = "return (gamma * eta * nw) / den"
DEN = "den = ng + eps * nw"
MUTANTS = {
    "norms_swapped": [(DEN, "den = nw + eps * ng"),
                      (RATE, "return (gamma * eta * ng) / den")],
    "eps_on_gradient": [(DEN, "den = nw + eps * ng")],
    "eps_dropped": [(DEN, "den = ng")],
    "gamma_dropped": [(RATE, "return (eta * nw) / den")],
    "no_sqrt": [("return math.sqrt(math.fsum((v * v).tolist()))",
                 "return math.fsum((v * v).tolist())")],
    "l1_norm": [("return math.sqrt(math.fsum((v * v).tolist()))",
                 "return math.fsum(np.abs(v).tolist())")],
    # the trust ratio taken as 1 whenever a norm is zero (a convention of
    # LARS implementations, not Eq. lars)
    "zero_norm_trust_ratio_one": [("    if den > 0.0:\n", "    if nw > 0.0 and ng > 0.0:\n"),
                                  ("    return 0.0\n", "    return gamma * eta\n")],
    "zero_gradient_gives_zero": [("    if den > 0.0:\n", "    if ng > 0.0:\n")],
    "zero_weight_gives_gamma_eta": [("    if den > 0.0:\n", "    if nw > 0.0 and den > 0.0:\n"),
                                    ("    return 0.0\n", "    return gamma * eta\n")],
    "zero_denominator_gamma_eta": [("    return 0.0\n", "    return gamma * eta\n")],
    "decay_sign": [("D = g + e32 * w", "D = g - e32 * w")],
    "decay_dropped": [("D = g + e32 * w", "D = g + 0 * w")],
    "rate_outside_momentum": [("b = m32 * b + U\n            w = w - b",
                               "b = m32 * b + D\n            w = w - lam * b")],
    "momentum_dropped": [("b = m32 * b + U", "b = U")],
    "dampened": [("b = m32 * b + U", "b = m32 * b + (1 - m32) * U")],
    "rate_not_rounded": [("lam = np.float32(rates[t])", "lam = rates[t]")],
    "global_norm": [("return np.array([lars_rate(layer_norm(w), layer_norm(g), gamma, eta, eps)\n                     for w, g in zip(ws, gs)], dtype=np.float64)",
                     "return np.array([lars_rate(layer_norm(np.concatenate(ws)), layer_norm(np.concatenate(gs)), gamma, eta, eps)\n                     for w, g in zip(ws, gs)], dtype=np.float64)")],
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_lars_mutant_is_caught(name, tmp_path):
    src = open(lars.__file__).read()
    for old, new in MUTANTS[name]:
        assert src.count(old) >= 1, f"snippet for {name} not found in the oracle source"
        src = src.replace(old, new, 1)
    path = tmp_path / f"lars_{name}.py"
    path.write_text(src)
    spec = importlib.util.spec_from_file_location(f"lars_mutant_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    for pin in ALL_LARS_PINS:
        try:
            pin(mod)
        except Exception:  # noqa: BLE001 - any failure counts as caught
            return
    raise AssertionError(f"mutant {name} passed every pin")
