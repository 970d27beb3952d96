"""The cost-model fit (t = t0 + T_exp |U|, R^2, MAPE) on data with a known
answer; no GPU."""

import numpy as np
import pytest

from paper_2608_15018_amd.calibrate import calibrate, fit_linear


def test_exact_line_recovered():
    u = np.array([2, 3, 5, 8, 13])
    fit = fit_linear(u, 12.5 + 51.25 * u)
    assert fit["t0_us"] == pytest.approx(12.5, abs=1e-9)
    assert fit["T_exp_us"] == pytest.approx(51.25, abs=1e-9)
    assert fit["r2"] == pytest.approx(1.0)
    assert fit["mape_pct"] == pytest.approx(0.0, abs=1e-9)


def test_r2_and_mape_match_their_definitions():
    rng = np.random.default_rng(0)
    u = rng.integers(1, 60, size=40).astype(float)
    t = 20.0 + 1.4 * u + rng.normal(0, 2.0, size=u.size)
    fit = fit_linear(u, t)
    slope, icpt = np.polyfit(u, t, 1)
    assert fit["T_exp_us"] == pytest.approx(slope)
    assert fit["t0_us"] == pytest.approx(icpt)
    r = np.corrcoef(u, t)[0, 1]
    assert fit["r2"] == pytest.approx(r * r)  # simple regression: R^2 = Pearson r^2
    pred = icpt + slope * u
    assert fit["mape_pct"] == pytest.approx(100 * np.mean(np.abs(t - pred) / t))


def test_degenerate_inputs_rejected():
    with pytest.raises(ValueError):
        fit_linear([4, 4, 4], [1.0, 2.0, 3.0])
    with pytest.raises(ValueError):
        fit_linear([4], [1.0])


def test_calibrate_fits_both_latencies():
    s = [{"n_uniq": n, "t_step_us": 10 + 2 * n, "t_ffn_us": 3 * n} for n in (1, 2, 4)]
    fit = calibrate(s)
    assert fit["step"]["T_exp_us"] == pytest.approx(2.0)
    assert fit["ffn"]["t0_us"] == pytest.approx(0.0, abs=1e-9)
