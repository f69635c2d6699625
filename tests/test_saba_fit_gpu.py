"""Parity of SABA's replay fit (HIP sums + host Levenberg-Marquardt through the
C ABI) with the CPU oracle.

Tolerances.  The sums are fp64 on both sides (fixed order here, numpy's
there).  The cost fit is linear least squares on the columns [1, B,
B * prefix]; scaled to unit columns their condition number is about 5.7 on
these logs, so the library's fp64 normal equations and the oracle's SVD solve
agree to about 1e-12 relative.  The library returns c in fp32, which adds at
most 2**-24 (6e-8) relative: c is compared at 1e-7 relative.  Both gain fits stop at the optimum of the same objective; on a
noisy log that optimum is flat to about 1e-6 relative in phi (the oracle pins
measure convergence agreement at that level), so phi is compared at 1e-4
relative and the objective at 1e-7 relative.  On an exact log both recover
the generating parameters (inputs rounded to fp32: 1e-5 relative)."""
import numpy as np
import pytest

import synthetic as S
from oracle import saba_fit as F

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _gpu(r):
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return T(r["state"]), T(r["prefix"]), T(r["accepted"]), T(r["latency"])


@pytest.mark.parametrize("T,noise,seed", [(3046, 0.0, 0), (3046, 0.05, 1), (37, 0.02, 2),
                                          (20000, 0.03, 3)])
def test_fit_matches_oracle(T, noise, seed):
    import paper_2608_20375_amd as G
    r = S.gen_replay(T, noise=noise, seed=seed)
    phi0 = (10.0, 10.0, 10.0, 10.0)
    got = G.saba_fit(r["budgets"], *_gpu(r), r["tau_min"], phi0, max_iter=500)
    ref = F.fit(r["budgets"], r["state"].astype(np.float64), r["prefix"], r["accepted"],
                r["latency"], r["tau_min"], phi0)
    assert got["converged"]
    np.testing.assert_allclose(got["c"], ref["c"], rtol=1e-7)
    assert got["cost_sse"] == pytest.approx(ref["cost_sse"], rel=1e-6, abs=1e-9)
    np.testing.assert_allclose(got["phi"], ref["phi"], rtol=1e-4)
    assert got["gain_sse"] == pytest.approx(ref["gain_sse"], rel=1e-7, abs=1e-12)
    if noise == 0.0:
        np.testing.assert_allclose(got["phi"], [6.0, 40.0, 30.0, 12.0], rtol=1e-5)
        np.testing.assert_allclose(got["c"], [20.0, 0.05, 2e-5], rtol=1e-5)


def test_empty_rounds_and_a_short_grid():
    import paper_2608_20375_amd as G
    r = S.gen_replay(500, grid=(16, 32, 64, 128, 256), noise=0.02, seed=4)
    r["accepted"][:50] = 0.0
    phi0 = (10.0, 10.0, 10.0, 10.0)
    got = G.saba_fit(r["budgets"], *_gpu(r), r["tau_min"], phi0, max_iter=500)
    ref = F.fit(r["budgets"], r["state"].astype(np.float64), r["prefix"], r["accepted"],
                r["latency"], r["tau_min"], phi0)
    np.testing.assert_allclose(got["phi"], ref["phi"], rtol=1e-4)
    assert got["gain_sse"] == pytest.approx(ref["gain_sse"], rel=1e-7)


def test_every_tau_clamped_returns_the_start():
    """phi . [1, s] below tau_min for every round: the objective does not
    depend on phi, the step system is singular, phi_init comes back."""
    import paper_2608_20375_amd as G
    r = S.gen_replay(200, seed=5)
    phi0 = (-500.0, 1.0, 1.0, 1.0)
    got = G.saba_fit(r["budgets"], *_gpu(r), r["tau_min"], phi0, max_iter=50)
    assert got["phi"] == [np.float32(v) for v in phi0]
    assert not got["converged"]
    ref = float(np.sum(F.gain_residuals(phi0, r["budgets"], r["state"].astype(np.float64),
                                        r["accepted"], r["tau_min"]) ** 2))
    assert got["gain_sse"] == pytest.approx(ref, rel=1e-9)


def test_deterministic_and_argument_errors():
    import paper_2608_20375_amd as G
    r = S.gen_replay(1000, noise=0.05, seed=6)
    a = G.saba_fit(r["budgets"], *_gpu(r), r["tau_min"], (10.0,) * 4)
    b = G.saba_fit(r["budgets"], *_gpu(r), r["tau_min"], (10.0,) * 4)
    assert a == b
    st, pre, acc, lat = _gpu(r)
    with pytest.raises(G.GraftError):
        G.saba_fit(list(r["budgets"]) + [0] * 40, st, pre,
                   torch.zeros(1000, 71, device="cuda"), torch.zeros(1000, 71, device="cuda"),
                   r["tau_min"], (10.0,) * 4)                       # more than 64 budgets
    with pytest.raises(G.GraftError):
        G.saba_fit(r["budgets"], st, pre, acc, lat, 0.0, (10.0,) * 4)   # tau_min <= 0
