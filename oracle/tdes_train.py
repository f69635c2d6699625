"""CPU oracle of one TDES training step -- TEST INFRASTRUCTURE.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this module; the HIP library never does.  Plain numpy in fp64, written from the
paper's Target-Distilled Edge Scoring section (scorer eq. tdes-bitower, the
three training objectives and their sum eq. tdes-training) and the training
paragraph of the experimental setup (AdamW, learning rate 2e-3, weight decay
1e-4, loss weights 1 / 1 / 0.25).

Parameter vector theta (fp32 in the library, fp64 here), in this order:
  g_parent [E, m] row-major | g_child [E, m] | depth_emb [L, m] (u_d at row d-1) | scale s
Batch of target-model traces:
  groups g < G:  parent[g], depth[g] in 1..L, child[g, K] (the candidate set
                 C_{p,d}), logq[g, K] (draft log-probabilities), z[g, K] (target
                 logits of the children), target[g] (the target's next token
                 under the parent; -1 if unknown)
  pairs i < P:   pairs[i] = (p+, c+, d+, p-, c-, d-): a target-compatible edge and
                 an incompatible alternative

Readings (the paper leaves these open):
  * every child of every group is a verified edge of the class-balanced BCE,
    labelled 1 where it is the group's target token;
  * each expectation is the plain mean over its items (groups, pairs, edges);
    an empty set contributes 0;
  * gamma (margin) and w1 (positive weight) are inputs; AdamW uses the common
    beta1 = 0.9, beta2 = 0.999, eps = 1e-8 unless told otherwise and decays
    every parameter, the scale and the depth embeddings included;
  * the KL objective uses f itself (no beta, no centering): both would only
    rescale or shift the softmax logits of a group, and the shift cancels.

The gradient is the chain rule written out by hand; tests pin it against
central finite differences of `losses` and pin the losses against library
routines and closed forms.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

__all__ = ["Hyper", "param_count", "unpack", "edge_f", "losses", "gradient", "adamw",
           "train_step"]

f64 = np.float64


@dataclass
class Hyper:
    """Loss weights (eq. tdes-training) and AdamW settings."""
    lambda_kl: float = 1.0
    lambda_pair: float = 1.0
    lambda_bce: float = 0.25
    gamma: float = 1.0
    w1: float = 1.0
    lr: float = 2e-3
    weight_decay: float = 1e-4
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8


def param_count(E: int, m: int, L: int) -> int:
    return 2 * E * m + L * m + 1


def unpack(theta, E: int, m: int, L: int):
    """Views (g_parent [E,m], g_child [E,m], depth_emb [L,m], s) of theta."""
    theta = np.asarray(theta)
    assert theta.size == param_count(E, m, L)
    n = E * m
    return (theta[:n].reshape(E, m), theta[n:2 * n].reshape(E, m),
            theta[2 * n:2 * n + L * m].reshape(L, m), theta[2 * n + L * m])


def _towers(theta, emb, p, c, d, E, m, L):
    """(g_p(e_p) + u_d, g_c(e_c) + u_d) for edges (p, c, d), eq. tdes-bitower."""
    gp, gc, u, _ = unpack(np.asarray(theta, f64), E, m, L)
    ud = u[np.asarray(d) - 1]
    a = np.asarray(emb, f64)[np.asarray(p)] @ gp + ud
    b = np.asarray(emb, f64)[np.asarray(c)] @ gc + ud
    return a, b


def edge_f(theta, emb, p, c, d, E, m, L):
    """f(p, c, d) = s (g_p(e_p) + u_d)^T (g_c(e_c) + u_d) / sqrt(m)."""
    a, b = _towers(theta, emb, p, c, d, E, m, L)
    s = float(unpack(np.asarray(theta, f64), E, m, L)[3])
    return s * (a * b).sum(-1) / math.sqrt(m)


def _log_softmax(x):
    mx = x.max(-1, keepdims=True)
    return x - mx - np.log(np.exp(x - mx).sum(-1, keepdims=True))


def _softplus(x):
    return np.logaddexp(0.0, x)


def _sigmoid(x):
    return np.exp(-_softplus(-x))


def _group_f(theta, emb, batch, E, m, L):
    G, K = np.asarray(batch["child"]).shape     # [G, K]
    if G == 0:
        return np.zeros((0, K))
    p = np.repeat(np.asarray(batch["parent"]), K)
    d = np.repeat(np.asarray(batch["depth"]), K)
    c = np.asarray(batch["child"]).reshape(-1)
    return edge_f(theta, emb, p, c, d, E, m, L).reshape(G, K)


def _pair_f(theta, emb, batch, E, m, L):
    pr = np.asarray(batch["pairs"]).reshape(-1, 6)
    if pr.shape[0] == 0:
        return np.zeros(0), np.zeros(0)
    fpos = edge_f(theta, emb, pr[:, 0], pr[:, 1], pr[:, 2], E, m, L)
    fneg = edge_f(theta, emb, pr[:, 3], pr[:, 4], pr[:, 5], E, m, L)
    return fpos, fneg


def losses(theta, emb, batch, h: Hyper, E, m, L):
    """(L, L_KL, L_pair, L_BCE) of eq. tdes-training on one batch."""
    G = len(batch["parent"])
    f = _group_f(theta, emb, batch, E, m, L)
    if G:
        K = f.shape[1]
        logq = np.asarray(batch["logq"], f64).reshape(G, K)
        z = np.asarray(batch["z"], f64).reshape(G, K)
        # distribution level: KL(pi_tgt || pi_theta) over the children of a group
        lpt = _log_softmax(z)
        lpth = _log_softmax(logq + f)
        l_kl = float((np.exp(lpt) * (lpt - lpth)).sum(-1).mean())
        # edge level: class-balanced BCE, positives weighted by w1
        y = (np.asarray(batch["child"]).reshape(G, K) ==
             np.asarray(batch["target"]).reshape(G, 1)).astype(f64)
        log_sig, log_one_minus = -_softplus(-f), -_softplus(f)
        l_bce = float(-(h.w1 * y * log_sig + (1.0 - y) * log_one_minus).mean())
    else:
        l_kl = l_bce = 0.0
    # pairwise level: margin loss on (v+, v-)
    fpos, fneg = _pair_f(theta, emb, batch, E, m, L)
    l_pair = float(_softplus(h.gamma - fpos + fneg).mean()) if fpos.size else 0.0
    total = h.lambda_kl * l_kl + h.lambda_pair * l_pair + h.lambda_bce * l_bce
    return total, l_kl, l_pair, l_bce


def _accumulate(theta, emb, p, c, d, delta, delta_abs, E, m, L, grad, agrad):
    """Adds the contribution of edges (p, c, d) with dL/df = delta; delta_abs
    is the sum of the magnitudes of delta's own terms (its cancellation scale)."""
    if len(delta) == 0:
        return
    gp, gc, u, s = unpack(np.asarray(theta, f64), E, m, L)
    Gp, Gc, U, _ = unpack(grad, E, m, L)
    aGp, aGc, aU, _ = unpack(agrad, E, m, L)
    a, b = _towers(theta, emb, p, c, d, E, m, L)
    ep = np.asarray(emb, f64)[np.asarray(p)]
    ec = np.asarray(emb, f64)[np.asarray(c)]
    k = s / math.sqrt(m)
    da = (delta * k)[:, None] * b            # dL/d(g_p(e_p) + u_d)
    db = (delta * k)[:, None] * a            # dL/d(g_c(e_c) + u_d)
    Gp += ep.T @ da
    Gc += ec.T @ db
    ada = (delta_abs * abs(k))[:, None] * np.abs(b)
    adb = (delta_abs * abs(k))[:, None] * np.abs(a)
    aGp += np.abs(ep).T @ ada
    aGc += np.abs(ec).T @ adb
    di = np.asarray(d) - 1
    np.add.at(U, di, da + db)
    np.add.at(aU, di, ada + adb)
    dot = (a * b).sum(-1) / math.sqrt(m)
    grad[-1] += float((delta * dot).sum())
    agrad[-1] += float((delta_abs * (np.abs(a) * np.abs(b)).sum(-1)).sum()) / math.sqrt(m)


def gradient(theta, emb, batch, h: Hyper, E, m, L):
    """(dL/dtheta, scale) of eq. tdes-training.  `scale` sums the magnitudes
    of every term of each component (and of the terms inside each dL/df), so a
    summation in any order with relative rounding u per operation stays within
    about (terms + depth) * u * scale of the exact value."""
    theta = np.asarray(theta, f64)
    grad = np.zeros(theta.size)
    agrad = np.zeros(theta.size)
    G = len(batch["parent"])
    if G:
        f = _group_f(theta, emb, batch, E, m, L)
        K = f.shape[1]
        logq = np.asarray(batch["logq"], f64).reshape(G, K)
        z = np.asarray(batch["z"], f64).reshape(G, K)
        y = (np.asarray(batch["child"]).reshape(G, K) ==
             np.asarray(batch["target"]).reshape(G, 1)).astype(f64)
        # d KL / d f_k = pi_theta(k) - pi_tgt(k)
        d_kl = np.exp(_log_softmax(logq + f)) - np.exp(_log_softmax(z))
        # d BCE / d f = -w1 y (1 - sigma(f)) + (1 - y) sigma(f)
        d_bce = -h.w1 * y * _sigmoid(-f) + (1.0 - y) * _sigmoid(f)
        delta = h.lambda_kl / G * d_kl + h.lambda_bce / (G * K) * d_bce
        delta_abs = (abs(h.lambda_kl) / G * (np.exp(_log_softmax(logq + f)) + np.exp(_log_softmax(z)))
                     + abs(h.lambda_bce) / (G * K) * np.abs(d_bce))
        _accumulate(theta, emb, np.repeat(batch["parent"], K), np.asarray(batch["child"]).reshape(-1),
                    np.repeat(batch["depth"], K), delta.reshape(-1), delta_abs.reshape(-1),
                    E, m, L, grad, agrad)
    pr = np.asarray(batch["pairs"]).reshape(-1, 6)
    P = pr.shape[0]
    if P:
        fpos, fneg = _pair_f(theta, emb, batch, E, m, L)
        t = _sigmoid(h.gamma - fpos + fneg) * (h.lambda_pair / P)
        _accumulate(theta, emb, pr[:, 0], pr[:, 1], pr[:, 2], -t, np.abs(t), E, m, L, grad, agrad)
        _accumulate(theta, emb, pr[:, 3], pr[:, 4], pr[:, 5], t, np.abs(t), E, m, L, grad, agrad)
    return grad, agrad


def adamw(theta, grad, m1, m2, step: int, h: Hyper):
    """Decoupled weight decay then the bias-corrected Adam step (Loshchilov and
    Hutter's AdamW; `step` counts from 1).  Returns new (theta, m1, m2)."""
    theta = np.asarray(theta, f64) * (1.0 - h.lr * h.weight_decay)
    m1 = h.beta1 * np.asarray(m1, f64) + (1.0 - h.beta1) * grad
    m2 = h.beta2 * np.asarray(m2, f64) + (1.0 - h.beta2) * grad * grad
    mhat = m1 / (1.0 - h.beta1 ** step)
    vhat = m2 / (1.0 - h.beta2 ** step)
    theta = theta - h.lr * mhat / (np.sqrt(vhat) + h.eps)
    return theta, m1, m2


def train_step(theta, m1, m2, step: int, emb, batch, h: Hyper, E, m, L):
    """One step: losses and gradient at theta, then AdamW.  Returns a dict."""
    loss = losses(theta, emb, batch, h, E, m, L)
    grad, agrad = gradient(theta, emb, batch, h, E, m, L)
    t2, n1, n2 = adamw(theta, grad, m1, m2, step, h)
    return dict(loss=loss, grad=grad, abs_grad=agrad, theta=t2, m1=n1, m2=n2)
