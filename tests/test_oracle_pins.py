"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle through a route other than its own code: closed
forms, library routines that compute the same quantity differently, brute-force
enumeration on tiny inputs, and invariants that a dropped term, a wrong sign,
a wrong index or a transposed operand would break.
"""
import itertools
import math

import numpy as np
import pytest

import oracle
import synthetic as S

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def bf16(vals):
    return S.bf16_from_f32(np.asarray(vals, dtype=np.float32))


# ---------------------------------------------------------------------------
# O2: row statistics (LSE, top-1 probability, entropy)
# ---------------------------------------------------------------------------

def test_row_stats_closed_forms():
    # V = 1: all mass on one token
    lse, mp, h = oracle.row_stats(bf16([3.0]))
    assert lse == 3.0 and mp == 1.0 and h == 0.0
    # uniform row: LSE = x + ln V, top-1 prob = 1/V, entropy = ln V
    for V in (2, 7, 1000):
        lse, mp, h = oracle.row_stats(bf16(np.full(V, -1.5)))
        assert lse == pytest.approx(-1.5 + math.log(V), abs=1e-14)
        assert mp == pytest.approx(1.0 / V, rel=1e-14)
        assert h == pytest.approx(math.log(V), abs=1e-13)
    # two tokens with logits 0 and ln-ish 2 (bf16 of 2.0 is exact)
    lse, mp, h = oracle.row_stats(bf16([0.0, 2.0]))
    p = 1.0 / (1.0 + math.exp(-2.0))
    assert lse == pytest.approx(2.0 + math.log1p(math.exp(-2.0)), abs=1e-15)
    assert mp == pytest.approx(p, rel=1e-15)
    assert h == pytest.approx(-(p * math.log(p) + (1 - p) * math.log(1 - p)), rel=1e-13)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_row_stats_vs_torch_float64(seed):
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(seed)
    x = g.standard_normal(5000).astype(np.float32) * 3
    x[g.choice(5000, 5, replace=False)] += 9.0
    h16 = bf16(x)
    xv = torch.from_numpy(S.f32_from_bf16(h16).astype(np.float64))
    lse, mp, h = oracle.row_stats(h16)
    ref_lse = torch.logsumexp(xv, 0).item()
    q = torch.softmax(xv, 0)
    ref_h = torch.distributions.Categorical(probs=q).entropy().item()
    assert lse == pytest.approx(ref_lse, abs=1e-12)
    assert mp == pytest.approx(q.max().item(), rel=1e-12)
    assert h == pytest.approx(ref_h, rel=1e-11)


# ---------------------------------------------------------------------------
# O3: top-K candidates, DFlash's argmax draft as K = 1 (eq. dflash-top1)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(4))
def test_topk_vs_numpy_lexsort(seed):
    g = np.random.default_rng(seed)
    V = int(g.integers(50, 3000))
    x = np.round(g.standard_normal(V) * 4) / 4        # many exact ties
    h16 = bf16(x)
    xv = S.f32_from_bf16(h16).astype(np.float64)
    for K in (1, 3, 8, min(V, 40)):
        ids, vals = oracle.topk(h16, K)
        ref = np.lexsort((np.arange(V), -xv))[:K]
        assert (ids == ref).all()
        assert (vals == xv[ref]).all()
    ids, _ = oracle.topk(h16, 1)
    assert ids[0] == int(np.argmax(xv))               # first maximum


def test_topk_constant_row_ties_by_id():
    ids, _ = oracle.topk(bf16(np.zeros(100)), 5)
    assert list(ids) == [0, 1, 2, 3, 4]


# ---------------------------------------------------------------------------
# O4: TDES edge scores
# ---------------------------------------------------------------------------

def _scorer(g, V, E, m, L, scale, beta, center, depth=True):
    return dict(emb=(g.standard_normal((V, E)) * 0.3).astype(np.float32),
                g_parent=(g.standard_normal((E, m)) * 0.2).astype(np.float32),
                g_child=(g.standard_normal((E, m)) * 0.2).astype(np.float32),
                depth_emb=(g.standard_normal((L, m)) * 0.2).astype(np.float32) if depth else None,
                scale=scale, beta=beta, center=center)


def _cands(g, V, L, K):
    cand = np.stack([g.choice(V, K, replace=False) for _ in range(L)]).astype(np.int32)
    logq = -np.sort(g.uniform(1, 9, size=(L, K)), axis=1)
    return cand, logq


def test_tdes_literal_equals_dense_W():
    """literal mode e_p^T (U V^T) e_c computed with the dense d x d matrix."""
    g = np.random.default_rng(5)
    V, E, m, L, K = 300, 12, 5, 4, 3
    sc = _scorer(g, V, E, m, L, float(np.float32(math.sqrt(m))), 1.0, 0, depth=False)
    P = oracle.make_params(L, K, 16, V, sc)
    cand, logq = _cands(g, V, L, K)
    root = 17
    edge, f = oracle.edge_scores(P, cand, logq, root)
    W = sc["g_parent"].astype(np.float64) @ sc["g_child"].astype(np.float64).T
    emb = sc["emb"].astype(np.float64)
    s_over = float(np.float32(math.sqrt(m))) / math.sqrt(m)
    for l in range(L):
        parents = [root] if l == 0 else list(cand[l - 1])
        for p, pt in enumerate(parents):
            for c in range(K):
                ref = s_over * emb[pt] @ W @ emb[cand[l, c]]
                assert f[l, p, c] == pytest.approx(ref, rel=1e-12, abs=1e-15)
                assert edge[l, p, c] == pytest.approx(logq[l, c] + ref, rel=1e-13, abs=1e-14)


def test_tdes_centering_and_beta():
    g = np.random.default_rng(6)
    V, E, m, L, K = 200, 8, 4, 3, 5
    sc = _scorer(g, V, E, m, L, 1.7, 0.3, 1)
    P = oracle.make_params(L, K, 16, V, sc)
    cand, logq = _cands(g, V, L, K)
    edge, f = oracle.edge_scores(P, cand, logq, 3)
    resid = edge - logq[:, None, :]
    for l in range(L):
        rows = 1 if l == 0 else K
        # centered residuals sum to zero over the children of each parent
        assert np.abs(resid[l, :rows].sum(axis=1)).max() < 1e-13
    # beta = 0 -> DDTree edge score log q (eq. ddtree-path-score)
    sc0 = dict(sc, beta=0.0)
    e0, _ = oracle.edge_scores(oracle.make_params(L, K, 16, V, sc0), cand, logq, 3)
    for l in range(L):
        rows = 1 if l == 0 else K
        assert (e0[l, :rows] == logq[l][None, :]).all()


def test_tdes_parent_only_terms_cancel_under_centering():
    """With g_c = 0 every term of f depends on the parent alone, so the centered
    residual vanishes; the depth embedding's parent-only part cancels too."""
    g = np.random.default_rng(7)
    V, E, m, L, K = 150, 6, 3, 3, 4
    sc = _scorer(g, V, E, m, L, 2.0, 0.5, 1)
    sc["g_child"] = np.zeros_like(sc["g_child"])
    cand, logq = _cands(g, V, L, K)
    edge, f = oracle.edge_scores(oracle.make_params(L, K, 16, V, sc), cand, logq, 9)
    for l in range(L):
        rows = 1 if l == 0 else K
        assert np.allclose(edge[l, :rows], logq[l][None, :], atol=1e-14)
        # uncentered f is the same for every child of a parent but not zero
        assert np.allclose(f[l, :rows], f[l, :rows, :1], atol=1e-14)
    assert np.abs(f[:, 0, 0]).max() > 1e-4


def test_tdes_depth_embedding_closed_forms():
    """Where u_d enters eq. tdes-bitower: it is added to both towers.
    (a) G_p = G_c = 0: f = s |u_d|^2 / sqrt(m) for every pair (a u_d on one
        tower only would give 0);
    (b) G_c = 0: f = s (e_p G_p + u_d) . u_d / sqrt(m), one value per parent
        (u_d on the child tower only would drop the |u_d|^2 term, on the parent
        tower only would give 0);
    (c) G_p = 0: f = s u_d . (e_c G_c + u_d) / sqrt(m), one value per child;
    with centering on, (a)'s constant cancels and the edge score is log q."""
    g = np.random.default_rng(17)
    V, E, m, L, K = 90, 5, 4, 4, 3
    sc = _scorer(g, V, E, m, L, 1.3, 0.7, 0)
    cand, logq = _cands(g, V, L, K)
    root = 11
    emb = sc["emb"].astype(np.float64)
    u = sc["depth_emb"].astype(np.float64)
    s_m = 1.3 / math.sqrt(m)
    zero = np.zeros_like(sc["g_parent"])

    # (a)
    sa = dict(sc, g_parent=zero, g_child=zero)
    edge, f = oracle.edge_scores(oracle.make_params(L, K, 16, V, sa), cand, logq, root)
    for l in range(L):
        rows = 1 if l == 0 else K
        want = s_m * float(u[l] @ u[l])
        assert want > 1e-3
        assert np.allclose(f[l, :rows], want, rtol=1e-12, atol=0)
        assert np.allclose(edge[l, :rows], logq[l][None, :] + 0.7 * want, rtol=1e-13, atol=1e-14)
    ec, _ = oracle.edge_scores(oracle.make_params(L, K, 16, V, dict(sa, center=1)), cand, logq,
                               root)
    for l in range(L):
        rows = 1 if l == 0 else K
        assert np.allclose(ec[l, :rows], logq[l][None, :], rtol=0, atol=1e-14)

    # (b) and (c)
    gp = sc["g_parent"].astype(np.float64)
    gc = sc["g_child"].astype(np.float64)
    _, fb = oracle.edge_scores(oracle.make_params(L, K, 16, V, dict(sc, g_child=zero)), cand,
                               logq, root)
    _, fc = oracle.edge_scores(oracle.make_params(L, K, 16, V, dict(sc, g_parent=zero)), cand,
                               logq, root)
    for l in range(L):
        parents = [root] if l == 0 else list(cand[l - 1])
        for p, pt in enumerate(parents):
            want_b = s_m * float((emb[pt] @ gp + u[l]) @ u[l])
            assert np.allclose(fb[l, p], want_b, rtol=1e-12, atol=1e-15)
            for c in range(K):
                want_c = s_m * float(u[l] @ (emb[cand[l, c]] @ gc + u[l]))
                assert fc[l, p, c] == pytest.approx(want_c, rel=1e-12, abs=1e-15)


def test_tdes_scale_and_dim_normalisation():
    """f scales linearly with s, and duplicating the scoring dimensions
    (m -> 2m, dot product doubles) scales f by sqrt(2): the 1/sqrt(m) factor."""
    g = np.random.default_rng(8)
    V, E, m, L, K = 120, 5, 3, 2, 3
    sc = _scorer(g, V, E, m, L, 1.0, 1.0, 0)
    cand, logq = _cands(g, V, L, K)
    _, f1 = oracle.edge_scores(oracle.make_params(L, K, 16, V, sc), cand, logq, 1)
    _, f3 = oracle.edge_scores(oracle.make_params(L, K, 16, V, dict(sc, scale=3.0)), cand, logq, 1)
    assert np.allclose(f3, 3 * f1, rtol=1e-13, atol=1e-15)
    sc2 = dict(sc, g_parent=np.concatenate([sc["g_parent"]] * 2, 1),
               g_child=np.concatenate([sc["g_child"]] * 2, 1),
               depth_emb=np.concatenate([sc["depth_emb"]] * 2, 1))
    _, f2 = oracle.edge_scores(oracle.make_params(L, K, 16, V, sc2), cand, logq, 1)
    assert np.allclose(f2[0, :1], math.sqrt(2) * f1[0, :1], rtol=1e-12)
    assert np.allclose(f2[1:], math.sqrt(2) * f1[1:], rtol=1e-12)


def test_tdes_depth1_parent_is_root():
    g = np.random.default_rng(9)
    V, E, m, L, K = 100, 4, 3, 3, 3
    sc = _scorer(g, V, E, m, L, 1.0, 1.0, 0)
    cand, logq = _cands(g, V, L, K)
    P = oracle.make_params(L, K, 16, V, sc)
    e1, _ = oracle.edge_scores(P, cand, logq, 5)
    e2, _ = oracle.edge_scores(P, cand, logq, 6)
    assert not np.allclose(e1[0, 0], e2[0, 0])
    assert (e1[1:] == e2[1:]).all()


# ---------------------------------------------------------------------------
# O5: SABA
# ---------------------------------------------------------------------------

def _saba_params(grid, phi, c0=1.0, c1=1 / 128, c2=0.0, tau_min=1.0):
    sc = dict(emb=np.zeros((2, 1), np.float32), g_parent=np.zeros((1, 1), np.float32),
              g_child=np.zeros((1, 1), np.float32), depth_emb=None, scale=1, beta=0, center=0)
    return oracle.make_params(1, 1, 2048, 2, sc, dict(grid=np.asarray(grid), phi=phi,
                                                      tau_min=tau_min, c0=c0, c1=c1, c2=c2))


def test_saba_matches_continuous_optimum():
    """U(B) = (1-e^{-B/tau})/(c0 + c B) is quasi-concave in B; its maximiser
    B* = tau x solves e^x = 1 + x + kappa, kappa = c0 / (c tau).  The grid argmax
    is one of the two grid points that bracket B*."""
    from scipy.optimize import brentq
    grid = list(range(16, 2049, 16))
    for tau in (3.0, 8.0, 32.0, 77.0, 128.0, 256.0):
        for c1, c2, prefix in ((1 / 128, 0.0, 0), (1 / 512, 2e-7, 3000)):
            P = _saba_params(grid, (tau, 0, 0, 0), c1=c1, c2=c2)
            b, t, rel, util = oracle.saba(P, 0.0, 0.0, 0.0, prefix)
            assert t == tau
            c = c1 + c2 * prefix
            kappa = 1.0 / (c * tau)
            x = brentq(lambda x: math.exp(x) - 1 - x - kappa, 1e-9, 60)
            bstar = tau * x
            lo = max([v for v in grid if v <= bstar], default=grid[0])
            hi = min([v for v in grid if v >= bstar], default=grid[-1])
            assert b in (lo, hi)
            # brute force over the grid with the definition
            U = [(1 - math.exp(-B / tau)) / (1 + c1 * B + c2 * B * prefix) for B in grid]
            assert b == grid[int(np.argmax(U))]
            assert np.allclose(util, U, rtol=1e-14)


def test_saba_limits_and_ties():
    grid = [32, 48, 64, 512]
    # huge tau with no per-node cost: gain grows with B -> largest budget
    assert oracle.saba(_saba_params(grid, (1e9, 0, 0, 0), c1=0.0), 0, 0, 0, 0)[0] == 512
    # tau at its floor with a per-node cost: smallest budget
    assert oracle.saba(_saba_params(grid, (-5.0, 0, 0, 0)), 0, 0, 0, 0)[0] == 32
    # exact ties (gain saturated to 1, no per-node cost) go to the smaller budget
    assert oracle.saba(_saba_params(grid, (1e-3, 0, 0, 0), c1=0.0, tau_min=1e-3), 0, 0, 0, 0)[0] == 32
    # tau = phi . [1, conf, ent, hist]: each feature enters with its own weight
    P = _saba_params(grid, (1.0, 10.0, 100.0, 1000.0), tau_min=0.0)
    assert oracle.saba(P, 0.5, 0.25, 0.125, 0)[1] == pytest.approx(1 + 5 + 25 + 125)


# ---------------------------------------------------------------------------
# O5a: representation degeneration (SABA decoding state)
# ---------------------------------------------------------------------------

def _hidden_with_cosines(H=16):
    """Hidden states built so that the adjacent cosines are known by
    construction (small integers, exact in bf16):
      h1 = 3 e0            h2 = 3 e0 + 4 e1   (3-4-5 triangle: cos = 3/5)
      h3 = 6 e0 + 8 e1     (a multiple of h2: cos = 1)
      h4 = 5 e2            (disjoint support: cos = 0)
      h5 = -10 e2          (opposite direction: cos = -1)"""
    h = np.zeros((5, H), np.float32)
    h[0, 0] = 3
    h[1, 0], h[1, 1] = 3, 4
    h[2, 0], h[2, 1] = 6, 8
    h[3, 2] = 5
    h[4, 2] = -10
    return h, [0.6, 1.0, 0.0, -1.0]


def test_degen_worked_example():
    h, r = _hidden_with_cosines()
    d, got = oracle.degen(bf16(h))
    assert np.allclose(got, r, atol=1e-15)
    # the paper's degen: mean adjacent similarity plus its late-minus-early rise
    # (r_4 - r_1 = -1.6 here), with the cosines above: 0.15 - 1.6
    assert d == pytest.approx(0.15 - 1.6, abs=1e-15)


def test_degen_special_cases_and_invariants():
    g = np.random.default_rng(7)
    # L = 1: no adjacent pair; L = 2: mean and rise collapse to r_1
    assert oracle.degen(bf16(g.standard_normal((1, 32))))[0] == 0.0
    h2 = bf16(g.standard_normal((2, 32)))
    d2, r2 = oracle.degen(h2)
    assert d2 == r2[0]
    # identical states: every r = 1, degen = 1; a zero state gives cosine 0
    same = bf16(np.tile(g.standard_normal(24), (6, 1)))
    assert oracle.degen(same)[0] == pytest.approx(1.0, abs=1e-14)
    z = np.asarray(S.f32_from_bf16(same)).copy()
    z[2] = 0
    dz, rz = oracle.degen(bf16(z))
    assert rz[1] == 0.0 and rz[2] == 0.0
    # scaling each state by a power of two (exact in bf16) changes nothing
    x = g.standard_normal((8, 64)).astype(np.float32)
    scale = (2.0 ** g.integers(-3, 4, size=8)).astype(np.float32)[:, None]
    d, r = oracle.degen(bf16(x))
    ds, rs = oracle.degen(bf16(x * scale))
    assert ds == pytest.approx(d, abs=1e-14) and np.allclose(rs, r, atol=1e-14)
    # cosines against numpy's normalised dot products of the bf16 values
    xv = S.f32_from_bf16(bf16(x)).astype(np.float64)
    u = xv / np.linalg.norm(xv, axis=1, keepdims=True)
    assert np.allclose(r, np.einsum("ij,ij->i", u[:-1], u[1:]), atol=1e-14)
    # reversing the depth order keeps the mean and negates the rise:
    # degen(h) + degen(reversed h) = 2 * mean(r)
    dr, _ = oracle.degen(bf16(x[::-1].copy()))
    assert d + dr == pytest.approx(2 * r.mean(), abs=1e-14)


def test_degen_drives_the_saba_state():
    """With hidden states the budget follows tau = phi . [1, conf, degen, hist]
    instead of the entropy stand-in."""
    w = S.workload(2, batch=2, V=4096)
    inp = S.gen_round(w, with_targets=False)
    sc = S.gen_scorer(w)
    sp = S.saba_params(w)
    h = S.gen_hidden(w, hidden_dim=64)
    P = oracle.make_params(w.L, w.K, w.n_max, w.V, sc, sp)
    b = 0
    res_h = oracle.build_sequence(P, inp["logits"][b], inp["root_token"][b], inp["base_pos"][b],
                                  inp["prefix_len"][b], 0, float(inp["hist"][b]), h[b])
    d, r = oracle.degen(h[b])
    assert res_h["degen"] == d and np.array_equal(res_h["adj_cos"], r)
    bud, tau, _, _ = oracle.saba(P, res_h["conf"], d, float(inp["hist"][b]), inp["prefix_len"][b])
    assert res_h["budget"] == bud and res_h["tau"] == tau
    phi = [float(v) for v in sp["phi"]]
    expect = phi[0] + phi[1] * res_h["conf"] + phi[2] * d + phi[3] * float(inp["hist"][b])
    assert tau == pytest.approx(max(expect, sp["tau_min"]), rel=1e-12)


# ---------------------------------------------------------------------------
# O6/O7: selection and emission against brute-force enumeration
# ---------------------------------------------------------------------------

def _all_prefixes(L, K, edge):
    """Every prefix (slot path) with its path score summed root to leaf."""
    out = []
    for l in range(1, L + 1):
        for path in itertools.product(range(K), repeat=l):
            s = 0.0
            prev = 0
            for d, c in enumerate(path):
                s = s + float(edge[d, prev if d else 0, c])
                prev = c
            out.append((path, s))
    return out


def _staged(L, K, n_max, cand, edge32, budget, base=100):
    sc = dict(emb=np.zeros((2, 1), np.float32), g_parent=np.zeros((1, 1), np.float32),
              g_child=np.zeros((1, 1), np.float32), depth_emb=None, scale=1, beta=0, center=0)
    P = oracle.make_params(L, K, n_max, 1 << 20, sc)
    return oracle.select_staged(P, cand, edge32, budget, base)


def _tok_path(cand, path):
    return tuple(int(cand[d, c]) for d, c in enumerate(path))


def _tree_paths(res, n):
    """token path of every emitted node, rebuilt from parents/tokens."""
    paths = []
    for i in range(n):
        p = res["parents"][i]
        paths.append((paths[p] if p >= 0 else ()) + (int(res["tokens"][i]),))
    return paths


def _random_case(g, L, K, monotone=True, lattice=False):
    cand = np.stack([g.choice(50, K, replace=False) for _ in range(L)]).astype(np.int32)
    if lattice:
        edge = -g.integers(0, 4, size=(L, K, K)).astype(np.float32) * 0.5   # many exact ties
    else:
        edge = -g.uniform(0.1, 5, size=(L, K, K)).astype(np.float32)
    if not monotone:
        edge = edge + g.uniform(-1.0, 2.5, size=edge.shape).astype(np.float32)
    return cand, edge


@pytest.mark.parametrize("seed", range(12))
def test_selection_equals_top_budget_prefixes_when_monotone(seed):
    """With every edge score <= 0 (DDTree's log-probability scores, i.e.
    beta = 0), best-first selection = the first N prefixes of the heap order over
    ALL prefixes: the top-budget product-of-probability tree."""
    g = np.random.default_rng(seed)
    L, K = int(g.integers(1, 5)), int(g.integers(1, 4))
    cand, edge = _random_case(g, L, K, lattice=seed % 2 == 0)
    total = sum(K ** l for l in range(1, L + 1))
    for budget in (0, 1, 5, total // 2, total, total + 7):
        res = _staged(L, K, 128, cand, edge, budget)
        n = res["n_nodes"]
        assert n == min(budget, total)
        allp = _all_prefixes(L, K, edge)
        key = lambda ps: (-ps[1], len(ps[0]), _tok_path(cand, ps[0]))
        top = sorted(allp, key=key)[:n]
        want = sorted((len(p), _tok_path(cand, p)) for p, _ in top)
        got = _tree_paths(res, n)
        assert [(len(p), p) for p in got] == want       # canonical order too
        assert res["node_scores"][:n].tolist() == [s for _, s in sorted(
            ((len(p), _tok_path(cand, p)), s) for p, s in top)]


def _py_best_first(L, K, cand, edge, budget):
    """Independent eager best-first with heapq and tuple keys."""
    import heapq
    h = []
    for c in range(K):
        s = float(edge[0, 0, c])
        heapq.heappush(h, (-s, 1, _tok_path(cand, (c,)), (c,), s))
    sel = []
    while len(sel) < budget and h:
        _, d, _, path, s = heapq.heappop(h)
        sel.append((path, s))
        if d < L:
            for c in range(K):
                s2 = s + float(edge[d, path[-1], c])
                p2 = path + (c,)
                heapq.heappush(h, (-s2, d + 1, _tok_path(cand, p2), p2, s2))
    return sel


@pytest.mark.parametrize("seed", range(12))
def test_selection_non_monotone_bottleneck_and_heapq(seed):
    """Positive edge scores: a child may outrank its parent.  The selected set
    is still prefix-closed, equals an independent heapq best-first, and obeys
    the bottleneck invariant min_sel b >= max_unsel b with
    b(u) = min over non-root prefixes of u of S."""
    g = np.random.default_rng(100 + seed)
    L, K = int(g.integers(2, 5)), int(g.integers(2, 4))
    cand, edge = _random_case(g, L, K, monotone=False, lattice=seed % 3 == 0)
    total = sum(K ** l for l in range(1, L + 1))
    budget = int(g.integers(1, total + 1))
    res = _staged(L, K, 128, cand, edge, budget)
    n = res["n_nodes"]
    got = set(_tree_paths(res, n))
    ref = _py_best_first(L, K, cand, edge, budget)
    assert got == {_tok_path(cand, p) for p, _ in ref}
    for p in got:                                      # prefix closed
        assert len(p) == 1 or p[:-1] in got
    allp = {_tok_path(cand, p): s for p, s in _all_prefixes(L, K, edge)}

    def bott(tp):
        return min(allp[tp[:i]] for i in range(1, len(tp) + 1))
    unsel = [tp for tp in allp if tp not in got]
    if unsel and got:
        assert min(bott(tp) for tp in got) >= max(bott(tp) for tp in unsel)


def test_selection_k1_is_dflash_chain():
    """K = 1: the tree is DFlash's argmax draft, a chain of min(N, L) nodes."""
    g = np.random.default_rng(3)
    L = 6
    cand = g.choice(1000, (L, 1), replace=False).astype(np.int32)
    edge = -g.uniform(0.1, 3, (L, 1, 1)).astype(np.float32)
    for budget in (0, 3, 6, 50):
        res = _staged(L, 1, 64, cand, edge, budget)
        n = res["n_nodes"]
        assert n == min(budget, L)
        assert list(res["tokens"][:n]) == list(cand[:n, 0])
        assert list(res["parents"][:n]) == ([-1] + list(range(n - 1)))[:n]


@pytest.mark.parametrize("seed", range(6))
def test_emission_invariants(seed):
    g = np.random.default_rng(200 + seed)
    L, K = 4, 3
    cand, edge = _random_case(g, L, K, monotone=seed % 2 == 0)
    n_max = 64
    budget = int(g.integers(1, n_max + 1))
    res = _staged(L, K, n_max, cand, edge, budget, base=1000)
    n = res["n_nodes"]
    par, dep, pos, mask = res["parents"], res["depth"], res["pos_ids"], res["mask"]
    paths = _tree_paths(res, n)
    # canonical order strictly increasing in (depth, token path)
    keys = [(len(p), p) for p in paths]
    assert all(a < b for a, b in zip(keys, keys[1:]))
    for i in range(n):
        assert par[i] < i
        assert dep[i] == len(paths[i]) and pos[i] == 1000 + dep[i]
        # mask row = ancestor-or-self set, recomputed as a closure of parents
        anc = set()
        j = i
        while j >= 0:
            anc.add(j)
            j = par[j]
        bits = {j for j in range(n_max) if (int(mask[i, j >> 6]) >> (j & 63)) & 1}
        assert bits == anc
        assert len(bits) == dep[i]                      # popcount = depth
    assert (mask[n:] == 0).all()
    assert (res["tokens"][n:] == -1).all() and (par[n:] == -1).all()


# ---------------------------------------------------------------------------
# O8: acceptance
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(8))
def test_acceptance_is_longest_target_consistent_path(seed):
    g = np.random.default_rng(300 + seed)
    L, K = 4, 3
    cand = np.stack([g.choice(6, K, replace=False) for _ in range(L)]).astype(np.int32)
    edge = -g.uniform(0.1, 2, (L, K, K)).astype(np.float32)
    res = _staged(L, K, 64, cand, edge, int(g.integers(1, 60)))
    n, tok, par = res["n_nodes"], res["tokens"], res["parents"]
    depth = res["depth"]
    # per-node targets over a tiny alphabet so matches are frequent
    troot = int(g.integers(0, 6))
    tnode = g.integers(0, 6, n_max := 64).astype(np.int32)
    a, nodes, bonus = oracle.accept(n, tok, par, L, troot, target_node=tnode)

    def target(j):
        return troot if j < 0 else int(tnode[j])

    ok = [i for i in range(n)]
    best = 0
    for i in range(n):
        j, good = i, True
        while j >= 0:
            if tok[j] != target(par[j]):
                good = False
            j = par[j]
        if good:
            best = max(best, int(depth[i]))
    assert a == best
    cur = -1
    for k in range(a):
        assert par[nodes[k]] == cur and tok[nodes[k]] == target(cur)
        cur = nodes[k]
    assert (nodes[a:] == -1).all()
    assert bonus == target(cur)
    # per-depth targets: all-equal targets reduce to following that token
    td = np.full(L + 1, int(cand[0, 0]), np.int32)
    a2, _, b2 = oracle.accept(n, tok, par, L, target_depth=td)
    assert b2 == td[a2]


def test_acceptance_empty_tree():
    a, nodes, bonus = oracle.accept(0, np.zeros(4, np.int32), np.zeros(4, np.int32), 4,
                                    target_root=42, target_node=np.zeros(4, np.int32))
    assert a == 0 and bonus == 42 and (nodes == -1).all()


# ---------------------------------------------------------------------------
# The parent-child mismatch example of the paper's motivation figure,
# rebuilt with numbers of our own: DDTree attaches "is" under the more probable
# parent "of"; a compatibility residual that prefers "fruits -> is" moves the
# child to the target-compatible parent.
# ---------------------------------------------------------------------------

def test_parent_child_mismatch_example():
    of, fruits, is_, are = 10, 11, 20, 21
    L, K = 2, 2
    cand = np.array([[of, fruits], [is_, are]], np.int32)
    logq = np.log(np.array([[0.6, 0.4], [0.7, 0.3]]))
    # DDTree: edge = log q; budget 3 keeps {of, fruits, of->is}
    edge_dd = np.zeros((L, K, K), np.float32)
    edge_dd[0, 0] = logq[0]
    edge_dd[1, :, :] = logq[1][None, :]
    res = _staged(L, K, 8, cand, edge_dd, 3)
    assert set(_tree_paths(res, 3)) == {(of,), (fruits,), (of, is_)}
    # TDES residual: +0.6 on fruits->is, -0.6 on of->is (centered per parent)
    f = np.array([[-0.6, 0.6], [0.6, -0.6]])           # rows: parent of / fruits
    edge_t = edge_dd.copy()
    edge_t[1] = logq[1][None, :] + 1.0 * (f - f.mean(1, keepdims=True))
    res = _staged(L, K, 8, cand, edge_t, 3)
    assert set(_tree_paths(res, 3)) == {(of,), (fruits,), (fruits, is_)}


# ---------------------------------------------------------------------------
# Whole-sequence pipeline on a synthetic workload: internal consistency
# ---------------------------------------------------------------------------

def test_build_sequence_consistency_small_workload():
    w = S.workload(2, batch=3, V=4000)
    inp = S.gen_round(w)
    sc = S.gen_scorer(w, "paper")
    sp = S.saba_params(w)
    res = oracle.build_round(w, inp, sc, sp)
    P = oracle.make_params(w.L, w.K, w.n_max, w.V, sc, sp)
    for b, r in enumerate(res):
        for l in range(w.L):
            lse, mp, h = oracle.row_stats(inp["logits"][b, l])
            assert r["row_lse"][l] == lse
            ids, x = oracle.topk(inp["logits"][b, l], w.K)
            assert (r["topk_ids"][l] == ids).all()
            assert np.allclose(r["topk_logq"][l], x - lse, atol=0)
        edge, _ = oracle.edge_scores(P, r["topk_ids"], r["topk_logq"], inp["root_token"][b])
        assert np.array_equal(edge, r["edge"])
        bud, *_ = oracle.saba(P, r["row_maxprob"].mean(), r["row_entropy"].mean(),
                              float(inp["hist"][b]), int(inp["prefix_len"][b]))
        assert bud == r["budget"] and r["n_nodes"] == min(bud, w.n_max)
        # staged selection on the oracle's own edges (as fp32) reaches the same tree
        st = oracle.select_staged(P, r["topk_ids"], r["edge"].astype(np.float32), r["budget"],
                                  int(inp["base_pos"][b]))
        if oracle.sequence_ok(r, w.L):
            assert np.array_equal(st["tokens"], r["tokens"])
            assert np.array_equal(st["parents"], r["parents"])
