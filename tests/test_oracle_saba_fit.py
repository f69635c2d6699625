"""Pins of the oracle's SABA fit by same-prefix budget replay (CPU, fp64).

What fixes it independently of its own code: recovery of the parameters a
noise-free replay log was generated from (gain eq. saba-gain and cost eq.
saba-cost, from starts far away); a hand-worked three-point cost fit; the
scale of each round cancelling (the budget rule only compares budgets within a
round); rounds that accept nothing or whose tau is clamped; and optimality of
the fitted phi on a noisy log."""
import numpy as np
import pytest

import synthetic as S
from oracle import saba_fit as F


def _log(T=400, noise=0.0, seed=0, **kw):
    r = S.gen_replay(T, noise=noise, seed=seed, **kw)
    r["state64"] = r["state"].astype(np.float64)
    return r


@pytest.mark.parametrize("phi0", [(10.0, 10.0, 10.0, 10.0), (1.0, 80.0, 5.0, 30.0)])
def test_recovers_the_generating_parameters(phi0):
    r = _log()
    out = F.fit(r["budgets"], r["state64"], r["prefix"], r["accepted"], r["latency"],
                r["tau_min"], phi0)
    np.testing.assert_allclose(out["phi"], [6.0, 40.0, 30.0, 12.0], rtol=1e-5)
    np.testing.assert_allclose(out["c"], [20.0, 0.05, 2e-5], rtol=1e-5)
    assert out["gain_sse"] < 1e-8 and out["cost_sse"] < 1e-6


def test_cost_fit_by_hand():
    """Three rounds, two budgets, latencies on the plane 5 + 0.5 B + 0.01 B p."""
    B = np.array([10, 20], np.int32)
    prefix = np.array([0, 100, 300], np.int32)
    lat = np.array([[5 + 0.5 * b + 0.01 * b * p for b in (10, 20)] for p in (0, 100, 300)])
    c, sse = F.fit_cost(B, prefix, lat)
    np.testing.assert_allclose(c, [5.0, 0.5, 0.01], rtol=1e-12, atol=1e-12)
    assert sse < 1e-20


def test_round_scales_cancel():
    """A common scale leaves the fit unchanged on a noisy log; per-round
    scales leave it unchanged on an exact one (each round's scale is
    eliminated, and an exact log fits with zero residual either way)."""
    phi0 = (10.0, 10.0, 10.0, 10.0)
    r = _log(T=200, noise=0.02, seed=3)
    a = F.fit_gain(r["budgets"], r["state64"], r["accepted"], r["tau_min"], phi0)[0]
    b = F.fit_gain(r["budgets"], r["state64"], r["accepted"].astype(np.float64) * 3.7,
                   r["tau_min"], phi0)[0]
    np.testing.assert_allclose(a, b, rtol=1e-5)
    r = _log(T=200)
    scaled = r["accepted"].astype(np.float64) * np.linspace(0.1, 7.0, 200)[:, None]
    c = F.fit_gain(r["budgets"], r["state64"], scaled, r["tau_min"], phi0)[0]
    np.testing.assert_allclose(c, [6.0, 40.0, 30.0, 12.0], rtol=1e-5)


def test_empty_rounds_and_clamped_tau_contribute_nothing():
    r = _log(T=100)
    acc = r["accepted"].astype(np.float64).copy()
    acc[:10] = 0.0
    res = F.gain_residuals((6.0, 40.0, 30.0, 12.0), r["budgets"], r["state64"], acc, r["tau_min"])
    assert not res.reshape(100, -1)[:10].any()
    # every tau clamped: the residuals do not depend on phi
    lo = F.gain_residuals((-500.0, 1.0, 1.0, 1.0), r["budgets"], r["state64"], acc, r["tau_min"])
    lo2 = F.gain_residuals((-900.0, 2.0, 0.0, 3.0), r["budgets"], r["state64"], acc, r["tau_min"])
    np.testing.assert_array_equal(lo, lo2)
    G, tau = F.gain_model((-500.0, 1.0, 1.0, 1.0), r["budgets"], r["state64"], r["tau_min"])
    assert (tau == r["tau_min"]).all()


def test_noisy_fit_is_a_minimum():
    r = _log(T=300, noise=0.05, seed=7)
    phi, sse = F.fit_gain(r["budgets"], r["state64"], r["accepted"], r["tau_min"],
                          (10.0, 10.0, 10.0, 10.0))
    f = lambda p: float(np.sum(F.gain_residuals(p, r["budgets"], r["state64"], r["accepted"],
                                                r["tau_min"]) ** 2))
    assert sse == pytest.approx(f(phi), rel=1e-12)
    assert sse <= f((6.0, 40.0, 30.0, 12.0))
    for k in range(4):
        for h in (-1e-3, 1e-3):
            p = np.array(phi)
            p[k] *= 1 + h
            assert f(p) >= sse
