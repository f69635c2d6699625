"""Pins of the oracle's TDES training step (CPU, fp64).

What fixes each piece independently of the oracle's own code:
  * the scorer f: the C inference oracle's edge scorer on the same parameters
    (a separate implementation of eq. tdes-bitower, itself pinned by the
    golden fixtures);
  * the three objectives: library routines (scipy's rel_entr for the KL, torch's
    BCE-with-logits with pos_weight, torch's softplus), closed forms (KL = 0 when
    the two distributions agree, the margin loss at f+ - f- = gamma is log 2)
    and invariances (shifting a group's logits leaves the KL unchanged);
  * the gradient: central finite differences of the losses, per objective;
  * AdamW: torch.optim.AdamW over several steps.
"""
import math

import numpy as np
import pytest

import oracle
import synthetic as S
from oracle import tdes_train as T

torch = pytest.importorskip("torch")


def _case(seed, E=8, m=4, L=3, K=4, G=5, P=4, V=40, target_hits=True):
    g = np.random.default_rng(seed)
    emb = g.standard_normal((V, E)) * 0.5
    theta = np.concatenate([g.standard_normal(2 * E * m) * 0.4, g.standard_normal(L * m) * 0.3,
                            [1.25]])
    child = np.stack([g.choice(V, K, replace=False) for _ in range(G)]).astype(np.int32)
    target = np.where(g.random(G) < 0.7, child[np.arange(G), g.integers(0, K, G)],
                      V + 1).astype(np.int32) if target_hits else np.full(G, -1, np.int32)
    batch = dict(parent=g.integers(0, V, G).astype(np.int32),
                 depth=g.integers(1, L + 1, G).astype(np.int32), child=child,
                 logq=np.sort(-g.exponential(1.0, (G, K)), axis=1)[:, ::-1].copy(),
                 z=g.standard_normal((G, K)) * 2.0, target=target,
                 pairs=np.stack([np.array([g.integers(0, V), g.integers(0, V), g.integers(1, L + 1),
                                           g.integers(0, V), g.integers(0, V), g.integers(1, L + 1)])
                                 for _ in range(P)]).astype(np.int32).reshape(P, 6))
    return emb, theta, batch, (E, m, L)


def test_edge_f_matches_the_inference_scorer():
    """f of the training oracle equals f of the C inference oracle (eq.
    tdes-bitower) for parents at depth 1 (the root) and deeper (candidates)."""
    L, K, E, m, V = 3, 4, 8, 4, 60
    g = np.random.default_rng(3)
    emb = (g.standard_normal((V, E)) * 0.5).astype(np.float32)
    gp = (g.standard_normal((E, m)) * 0.4).astype(np.float32)
    gc = (g.standard_normal((E, m)) * 0.4).astype(np.float32)
    u = (g.standard_normal((L, m)) * 0.3).astype(np.float32)
    scorer = dict(emb=emb, g_parent=gp, g_child=gc, depth_emb=u, scale=1.5, beta=1.0, center=0)
    P = oracle.make_params(L, K, 16, V, scorer)
    cand = np.stack([g.choice(V, K, replace=False) for _ in range(L)]).astype(np.int32)
    root = 7
    _, f = oracle.edge_scores(P, cand, np.zeros((L, K)), root)
    theta = np.concatenate([gp.ravel(), gc.ravel(), u.ravel(), [1.5]]).astype(np.float64)
    for l in range(L):
        parents = [root] if l == 0 else list(cand[l - 1])
        for pi, p in enumerate(parents):
            got = T.edge_f(theta, emb, np.full(K, p), cand[l], np.full(K, l + 1), E, m, L)
            np.testing.assert_allclose(got, f[l, pi], rtol=1e-12, atol=1e-14)


def test_kl_is_relative_entropy_and_vanishes_on_agreement():
    from scipy.special import rel_entr, softmax
    emb, theta, batch, (E, m, L) = _case(1)
    h = T.Hyper(lambda_kl=1.0, lambda_pair=0.0, lambda_bce=0.0)
    _, l_kl, _, _ = T.losses(theta, emb, batch, h, E, m, L)
    G, K = batch["child"].shape
    f = T.edge_f(theta, emb, np.repeat(batch["parent"], K), batch["child"].ravel(),
                 np.repeat(batch["depth"], K), E, m, L).reshape(G, K)
    want = np.mean([rel_entr(softmax(batch["z"][i]), softmax(batch["logq"][i] + f[i])).sum()
                    for i in range(G)])
    assert l_kl == pytest.approx(want, rel=1e-12)
    assert l_kl > 0
    same = dict(batch, z=batch["logq"] + f + 3.0)       # pi_tgt == pi_theta
    assert abs(T.losses(theta, emb, same, h, E, m, L)[1]) < 1e-14


def test_kl_ignores_a_per_group_shift():
    emb, theta, batch, (E, m, L) = _case(2)
    h = T.Hyper()
    g = np.random.default_rng(0)
    sh = dict(batch, z=batch["z"] + g.standard_normal((len(batch["z"]), 1)) * 5,
              logq=batch["logq"] + g.standard_normal((len(batch["z"]), 1)) * 5)
    assert T.losses(theta, emb, sh, h, E, m, L)[1] == pytest.approx(
        T.losses(theta, emb, batch, h, E, m, L)[1], rel=1e-11)


@pytest.mark.parametrize("w1", [1.0, 7.5])
def test_bce_is_bce_with_logits_and_pos_weight(w1):
    emb, theta, batch, (E, m, L) = _case(4)
    h = T.Hyper(w1=w1)
    G, K = batch["child"].shape
    f = T.edge_f(theta, emb, np.repeat(batch["parent"], K), batch["child"].ravel(),
                 np.repeat(batch["depth"], K), E, m, L)
    y = (batch["child"] == batch["target"][:, None]).ravel().astype(np.float64)
    assert y.sum() > 0
    want = torch.nn.functional.binary_cross_entropy_with_logits(
        torch.tensor(f), torch.tensor(y), pos_weight=torch.tensor(w1, dtype=torch.float64)).item()
    assert T.losses(theta, emb, batch, h, E, m, L)[3] == pytest.approx(want, rel=1e-12)


def test_pair_loss_is_softplus_of_the_margin():
    emb, theta, batch, (E, m, L) = _case(5)
    h = T.Hyper(gamma=0.7)
    pr = batch["pairs"]
    fp = T.edge_f(theta, emb, pr[:, 0], pr[:, 1], pr[:, 2], E, m, L)
    fn = T.edge_f(theta, emb, pr[:, 3], pr[:, 4], pr[:, 5], E, m, L)
    want = torch.nn.functional.softplus(torch.tensor(0.7 - fp + fn)).mean().item()
    assert T.losses(theta, emb, batch, h, E, m, L)[2] == pytest.approx(want, rel=1e-12)
    # v+ and v- the same edge: every pair sits exactly at the margin
    tie = dict(batch, pairs=np.concatenate([pr[:, :3], pr[:, :3]], axis=1))
    assert T.losses(theta, emb, tie, T.Hyper(gamma=0.0), E, m, L)[2] == pytest.approx(math.log(2),
                                                                                       rel=1e-14)


def test_total_is_the_weighted_sum():
    emb, theta, batch, (E, m, L) = _case(6)
    h = T.Hyper(lambda_kl=0.5, lambda_pair=2.0, lambda_bce=0.25)
    tot, a, b, c = T.losses(theta, emb, batch, h, E, m, L)
    assert tot == pytest.approx(0.5 * a + 2.0 * b + 0.25 * c, rel=1e-14)


def _fd(fun, theta, eps=1e-5):
    out = np.empty(theta.size)
    for i in range(theta.size):
        tp, tm = theta.copy(), theta.copy()
        tp[i] += eps
        tm[i] -= eps
        out[i] = (fun(tp) - fun(tm)) / (2 * eps)
    return out


@pytest.mark.parametrize("lam", [(1, 0, 0), (0, 1, 0), (0, 0, 1), (1, 1, 0.25)])
@pytest.mark.parametrize("seed", [7, 8])
def test_gradient_matches_finite_differences(lam, seed):
    emb, theta, batch, (E, m, L) = _case(seed)
    h = T.Hyper(lambda_kl=lam[0], lambda_pair=lam[1], lambda_bce=lam[2], gamma=0.6, w1=3.0)
    g, scale = T.gradient(theta, emb, batch, h, E, m, L)
    fd = _fd(lambda t: T.losses(t, emb, batch, h, E, m, L)[0], theta)
    np.testing.assert_allclose(g, fd, rtol=1e-6, atol=1e-9)
    assert (scale >= np.abs(g) * (1 - 1e-12)).all()
    assert np.abs(g).max() > 1e-3


def test_gradient_without_positives_and_with_k1():
    emb, theta, batch, (E, m, L) = _case(9, K=1, target_hits=False)
    h = T.Hyper(w1=2.0)
    g, _ = T.gradient(theta, emb, batch, h, E, m, L)
    fd = _fd(lambda t: T.losses(t, emb, batch, h, E, m, L)[0], theta)
    np.testing.assert_allclose(g, fd, rtol=1e-6, atol=1e-9)
    # one child per group: the KL is identically zero
    assert T.losses(theta, emb, batch, h, E, m, L)[1] == pytest.approx(0.0, abs=1e-15)


def test_empty_batch():
    E, m, L = 8, 4, 3
    theta = np.linspace(-1, 1, T.param_count(E, m, L))
    batch = dict(parent=np.zeros(0, np.int32), depth=np.zeros(0, np.int32),
                 child=np.zeros((0, 4), np.int32), logq=np.zeros((0, 4)), z=np.zeros((0, 4)),
                 target=np.zeros(0, np.int32), pairs=np.zeros((0, 6), np.int32))
    emb = np.ones((10, E))
    assert T.losses(theta, emb, batch, T.Hyper(), E, m, L) == (0.0, 0.0, 0.0, 0.0)
    g, _ = T.gradient(theta, emb, batch, T.Hyper(), E, m, L)
    assert not g.any()


def test_adamw_matches_torch():
    g = np.random.default_rng(11)
    h = T.Hyper(lr=2e-3, weight_decay=1e-4)
    theta = g.standard_normal(23)
    m1 = np.zeros(23)
    m2 = np.zeros(23)
    p = torch.nn.Parameter(torch.tensor(theta))
    opt = torch.optim.AdamW([p], lr=h.lr, betas=(h.beta1, h.beta2), eps=h.eps,
                            weight_decay=h.weight_decay)
    for step in range(1, 6):
        grad = g.standard_normal(23) * 10.0 ** g.integers(-6, 1)
        theta, m1, m2 = T.adamw(theta, grad, m1, m2, step, h)
        p.grad = torch.tensor(grad)
        opt.step()
        np.testing.assert_allclose(theta, p.detach().numpy(), rtol=1e-13, atol=1e-15)


def test_train_step_lowers_the_loss_on_synthetic_traces():
    """A few oracle steps on a small synthetic batch reduce the objective."""
    w = S.workload(0, V=300, L=4, K=4, emb_dim=16, rank=8)
    tr = S.gen_traces(w, 24, 16)
    sc = S.gen_scorer(w, "paper")
    E, m, L = w.emb_dim, w.rank, w.L
    theta = np.concatenate([sc["g_parent"].ravel(), sc["g_child"].ravel(),
                            sc["depth_emb"].ravel(), [sc["scale"]]]).astype(np.float64)
    h = T.Hyper(lr=2e-2, w1=3.0)
    m1 = np.zeros_like(theta)
    m2 = np.zeros_like(theta)
    first = None
    for step in range(1, 21):
        r = T.train_step(theta, m1, m2, step, sc["emb"], tr, h, E, m, L)
        theta, m1, m2 = r["theta"], r["m1"], r["m2"]
        first = r["loss"][0] if first is None else first
    assert T.losses(theta, sc["emb"], tr, h, E, m, L)[0] < 0.9 * first
