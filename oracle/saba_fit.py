"""CPU oracle of SABA's parameter fit by same-prefix budget replay -- TEST
INFRASTRUCTURE.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this module; the HIP library never does.  numpy/scipy in fp64, written from the
paper's State-Aware Budget Allocation section (gain eq. saba-gain, cost eq.
saba-cost, "fit the parameters of G_t(B) and C_t(B) on a small held-out
validation set") and the experimental setup (the fit uses same-prefix budget
replay).

Replay log: round t of the validation set was decoded from one prefix with
every budget B_j of the grid, giving its accepted length a_t(B_j) and its
round latency l_t(B_j); s_t = [conf, degen, hist] is the round's state.

Readings (the paper gives the models, not the fitting procedure):
  * cost: ordinary least squares of l_t(B_j) on [1, B_j, B_j prefix_t];
  * gain: the accepted length is modelled as A_t G_t(B) with
    G_t(B) = 1 - exp(-B / tau_t), tau_t = max(phi . [1, s_t], tau_min) (the
    state weights with a bias term, as the budget rule uses them).  The
    round's scale A_t cancels in argmax_B G_t(B) / C_t(B), so it is a nuisance
    parameter, eliminated per round in closed form (A_t = sum_j a G / sum_j G^2,
    variable projection); a round that accepts nothing contributes nothing;
  * phi minimises sum_{t,j} (A_t G_t(B_j) - a_t(B_j))^2, found by
    Levenberg-Marquardt from a given start (scipy's MINPACK implementation
    here, a step of this oracle).
"""
from __future__ import annotations

import numpy as np

__all__ = ["fit_cost", "gain_model", "gain_residuals", "fit_gain", "fit"]

f64 = np.float64


def fit_cost(budgets, prefix, latency):
    """(c0, c1, c2, sse) of the affine cost model (eq. saba-cost)."""
    B = np.asarray(budgets, f64)
    pre = np.asarray(prefix, f64)
    lat = np.asarray(latency, f64)
    T, nb = lat.shape
    X = np.stack([np.ones(T * nb), np.tile(B, T), (pre[:, None] * B[None, :]).ravel()], axis=1)
    c, *_ = np.linalg.lstsq(X, lat.ravel(), rcond=None)
    r = X @ c - lat.ravel()
    return c, float(r @ r)


def gain_model(phi, budgets, state, tau_min):
    """G_t(B_j) [T, nb] (eq. saba-gain) and tau_t."""
    B = np.asarray(budgets, f64)
    s = np.concatenate([np.ones((len(state), 1)), np.asarray(state, f64)], axis=1)
    tau = np.maximum(s @ np.asarray(phi, f64), tau_min)
    return 1.0 - np.exp(-B[None, :] / tau[:, None]), tau


def gain_residuals(phi, budgets, state, accepted, tau_min):
    """A_t G_t(B_j) - a_t(B_j) with the best scale A_t of each round, flattened."""
    G, _ = gain_model(phi, budgets, state, tau_min)
    a = np.asarray(accepted, f64)
    den = (G * G).sum(axis=1)
    A = np.where(den > 0, (G * a).sum(axis=1) / np.where(den > 0, den, 1.0), 0.0)
    return (A[:, None] * G - a).ravel()


def fit_gain(budgets, state, accepted, tau_min, phi0):
    """(phi, sse) by Levenberg-Marquardt from phi0."""
    from scipy.optimize import least_squares
    res = least_squares(gain_residuals, np.asarray(phi0, f64), method="lm",
                        args=(budgets, state, accepted, tau_min), xtol=1e-15, ftol=1e-15,
                        gtol=1e-15, max_nfev=20000)
    r = res.fun
    return res.x, float(r @ r)


def fit(budgets, state, prefix, accepted, latency, tau_min, phi0):
    c, cost_sse = fit_cost(budgets, prefix, latency)
    phi, gain_sse = fit_gain(budgets, state, accepted, tau_min, phi0)
    return dict(phi=phi, c=c, gain_sse=gain_sse, cost_sse=cost_sse)
