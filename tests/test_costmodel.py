"""The library's cost model (md_sd_*, host arithmetic of Eq. 1-4) against the
oracle, on the paper's printed rows and on seeded random inputs (CPU only)."""
import math
import os

import numpy as np
import pytest

import oracle.costmodel as ref
import paper_2408_11049_amd as md
from costmodel_pins import golden_rows


@pytest.fixture(scope="module", autouse=True)
def lib():
    if not os.path.exists(md.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return md.load_library()


def rel(a, b):
    return abs(a - b) / max(abs(b), 1e-300)


def test_expected_tokens_matches_oracle():
    rng = np.random.default_rng(1)
    for _ in range(500):
        g = int(rng.integers(0, 40))
        a = float(rng.uniform(0, 0.999))
        assert rel(md.md_sd_expected_tokens(g, a), ref.expected_tokens(g, a)) < 1e-12
    for g in (0, 3, 17):
        assert md.md_sd_expected_tokens(g, 0.0) == 1.0
        assert md.md_sd_expected_tokens(g, 1.0) == g + 1
    assert math.isnan(md.md_sd_expected_tokens(-1, 0.5))
    assert math.isnan(md.md_sd_expected_tokens(3, 1.5))
    assert math.isnan(md.md_sd_expected_tokens(3, -0.1))


def test_latency_ratio_matches_oracle():
    rng = np.random.default_rng(2)
    for _ in range(500):
        g = int(rng.integers(1, 16))
        a = float(rng.uniform(0, 0.99))
        tt, td, ts, tv = (float(x) for x in rng.uniform(0.01, 10, size=4))
        got = md.md_sd_latency_ratio(g, a, tt, td, tv, t_select=ts)
        assert rel(got, ref.latency_ratio(g, a, tt, td, tv, t_select=ts)) < 1e-12
    assert math.isnan(md.md_sd_latency_ratio(3, 0.5, 0.0, 1.0, 1.0))
    assert math.isnan(md.md_sd_latency_ratio(3, 0.5, 1.0, -1.0, 1.0))
    assert math.isnan(md.md_sd_latency_ratio(3, 0.5, 1.0, 1.0, float("nan")))


def test_best_gamma_matches_oracle():
    rng = np.random.default_rng(3)
    for _ in range(300):
        n = int(rng.integers(1, 20))
        a = float(rng.uniform(0, 0.99))
        tt, td, ts = float(rng.uniform(0.5, 2)), float(rng.uniform(0, 0.5)), float(rng.uniform(0, 0.1))
        tv = list(tt * (1 + np.cumsum(rng.uniform(0, 0.3, size=n))))
        g, r = md.md_sd_best_gamma(a, tt, td, tv, t_select=ts)
        rg, rr = ref.best_gamma(a, tt, td, tv, t_select=ts)
        assert g == rg and rel(r, rr) < 1e-12
    with pytest.raises(ValueError):
        md.md_sd_best_gamma(0.5, 1.0, 0.1, [])
    with pytest.raises(ValueError):
        md.md_sd_best_gamma(0.5, 1.0, 0.1, [1.0, -2.0])


def test_alpha_from_omega_matches_oracle():
    for g in (1, 4, 11):
        for a in (0.1, 0.5, 0.9, 0.93):
            om = ref.expected_tokens(g, a)
            assert abs(md.md_sd_alpha_from_omega(g, om) - ref.alpha_from_omega(g, om)) < 1e-10
    # near alpha = 1 the library's summed form stays resolvable
    om = sum(0.999999 ** k for k in range(12))
    assert abs(md.md_sd_alpha_from_omega(11, om) - 0.999999) < 1e-12
    assert math.isnan(md.md_sd_alpha_from_omega(4, 5.5))
    assert math.isnan(md.md_sd_alpha_from_omega(4, 0.9))


def test_paper_rows_through_the_library():
    """The printed rows of Tables 1 and 2 evaluated by the library agree with
    the oracle and, like it, reproduce the printed speedups to within 3.5%."""
    for r in golden_rows():
        g = int(r["gamma"])
        a = md.md_sd_alpha_from_omega(g, r["omega"])
        assert abs(a - ref.alpha_from_omega(g, r["omega"])) < 1e-9
        x = 1.0 / md.md_sd_latency_ratio(g, a, r["t_ar"], r["gamma_td"] / g, r["tv"])
        assert 1.0 <= x / r["x"] <= 1.035, (r["setting"], x, r["x"])
