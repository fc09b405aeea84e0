"""Pins of the cost-model oracle (oracle/costmodel.py).

  tables_eq2   the paper's printed step times (Tables 1 and 2, in
               tests/golden/sd_speedup_tables.csv): Eq. 2 built from the
               printed gamma*T_D, T_V and Omega reproduces the printed T^SD to
               within 3% (never above it: the measured step carries overheads
               the model leaves out) and the printed speedup x from T^AR;
  eq1_values   Eq. 1 at alpha = 0, 1 and a hand-summed geometric series;
  eq2_cases    Eq. 2 / Eq. 3 special cases: perfect acceptance with free drafts
               and free verification gives 1 / (gamma + 1); zero acceptance
               gives the plain cost ratio; selection time adds gamma * T_select;
  alpha_inverse  the inverse of Eq. 1 returns alpha values Eq. 1 maps back,
               and recovers known alphas;
  best_gamma   Eq. 4 over gamma on a worked example with an interior optimum,
               monotone cases at both ends, and ties to the smaller gamma.
"""
import csv
import math
import os

import oracle.costmodel as real

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "sd_speedup_tables.csv")


def _m(mod):
    return real if mod is None else mod


def golden_rows():
    with open(GOLDEN) as f:
        lines = [l for l in f if not l.startswith("#")]
    rows = []
    for r in csv.DictReader(lines):
        rows.append({k: (v if k in ("source", "setting") else float(v)) for k, v in r.items()})
    return rows


def pin_tables_eq2(mod=None):
    s = _m(mod)
    rows = golden_rows()
    assert len(rows) == 12
    for r in rows:
        g = int(r["gamma"])
        t_d = r["gamma_td"] / g
        model = s.step_time(g, t_d, r["tv"]) / r["omega"]
        dev = model / r["t_sd"] - 1
        assert -0.03 <= dev <= 0.0, (r["setting"], model, r["t_sd"])
        alpha = s.alpha_from_omega(g, r["omega"])
        x_model = 1.0 / s.latency_ratio(g, alpha, r["t_ar"], t_d, r["tv"])
        assert 1.0 <= x_model / r["x"] <= 1.035, (r["setting"], x_model, r["x"])
        assert abs(r["t_ar"] / r["t_sd"] - r["x"]) <= 0.006  # the table's own x column


def pin_eq1_values(mod=None):
    s = _m(mod)
    assert s.expected_tokens(5, 0.0) == 1.0
    assert s.expected_tokens(5, 1.0) == 6.0
    assert abs(s.expected_tokens(2, 0.5) - 1.75) < 1e-15
    assert abs(s.expected_tokens(3, 0.9) - (1 + 0.9 + 0.81 + 0.729)) < 1e-12
    assert s.expected_tokens(0, 0.7) == 1.0


def pin_eq2_cases(mod=None):
    s = _m(mod)
    for g in (1, 3, 8):
        assert abs(s.latency_ratio(g, 1.0, 2.0, 0.0, 2.0) - 1.0 / (g + 1)) < 1e-15
        assert abs(s.latency_ratio(g, 0.0, 2.0, 0.5, 3.0) - (g * 0.5 + 3.0) / 2.0) < 1e-15
        with_sel = s.latency_ratio(g, 0.6, 2.0, 0.5, 3.0, t_select=0.25)
        without = s.latency_ratio(g, 0.6, 2.0, 0.5, 3.0)
        assert abs((with_sel - without) * 2.0 * s.expected_tokens(g, 0.6) - g * 0.25) < 1e-12
    assert s.draft_time(0.5, 0.25) == 0.75


def pin_alpha_inverse(mod=None):
    s = _m(mod)
    for g in (1, 4, 11):
        for a in (0.05, 0.5, 0.93, 0.999):
            om = 1.0
            for k in range(1, g + 1):       # Omega as a plain sum, not Eq. 1's closed form
                om += a ** k
            assert abs(s.alpha_from_omega(g, om) - a) < 1e-9, (g, a)
    assert s.alpha_from_omega(4, 1.0) < 1e-12
    # Omega = gamma + 1 means alpha = 1, where Eq. 1's closed form cancels
    # (1 - a^5 and 1 - a both vanish): only ~1e-8 of alpha is resolvable there.
    assert abs(s.alpha_from_omega(4, 5.0) - 1.0) < 1e-6
    assert math.isnan(s.alpha_from_omega(4, 5.5)) and math.isnan(s.alpha_from_omega(4, 0.5))


def pin_best_gamma(mod=None):
    s = _m(mod)
    # alpha 0.8, T_T 1, T_D 0.1, T_V(g) = 1 + 0.05 g.  Eq. 2 by hand:
    # g=4: (0.4 + 1.20) / 3.3616 = 0.47596; g=5: (0.5 + 1.25) / 3.68928 = 0.47435;
    # g=6: (0.6 + 1.30) / 3.951424 = 0.48084.
    tv = [1 + 0.05 * g for g in range(1, 11)]
    g, r = s.best_gamma(0.8, 1.0, 0.1, tv)
    assert g == 5 and abs(r - 1.75 / 3.68928) < 1e-9, (g, r)
    # free drafts and flat verification: longer is always better
    assert s.best_gamma(0.9, 1.0, 0.0, [1.0] * 7)[0] == 7
    # drafts as costly as the target: the shortest speculation wins
    assert s.best_gamma(0.5, 1.0, 1.0, [1.0] * 7)[0] == 1
    # alpha = 0 with free drafts and flat verification: every gamma ties at 1
    g, r = s.best_gamma(0.0, 1.0, 0.0, [1.0] * 5)
    assert g == 1 and r == 1.0


ALL_COSTMODEL_PINS = [pin_tables_eq2, pin_eq1_values, pin_eq2_cases, pin_alpha_inverse,
                      pin_best_gamma]
