"""Hand-worked examples under tests/golden/ (each fixture states the passage of
the paper it illustrates and its derivation): the CPU oracle must reproduce
them exactly (integers) or to 1e-12 (floating point), and the HIP path, where
the C ABI reaches the step, to its own bars."""
import os

import numpy as np
import pytest

import oracle
import synthetic as S

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name):
    """key: value lines; 'case:' starts a new case; '#' comments."""
    head, cases, cur = {}, [], None
    for line in open(os.path.join(GOLDEN, name)):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        k, v = (x.strip() for x in line.split(":", 1))
        if k == "case":
            cur = {"case": v}
            cases.append(cur)
        else:
            (cur if cur is not None else head)[k] = v
    return head, cases


def nums(v, dt=float):
    return np.array([dt(x) for x in v.replace("|", " ").split()])


def groups(v, dt=float):
    return [nums(g, dt) for g in v.split("|")]


def bf16(x):
    return S.bf16_from_f32(np.asarray(x, np.float32))


# ---------------------------------------------------------------------------
# oracle (CPU)
# ---------------------------------------------------------------------------

def test_golden_row_stats():
    _, cases = load("row_stats.txt")
    assert len(cases) == 3
    for c in cases:
        lse, mp, h = oracle.row_stats(bf16(nums(c["logits"])))
        assert lse == pytest.approx(float(c["lse"]), rel=1e-12, abs=1e-12), c["case"]
        assert mp == pytest.approx(float(c["maxprob"]), rel=1e-12), c["case"]
        assert h == pytest.approx(float(c["entropy"]), rel=1e-12, abs=1e-12), c["case"]


def _selection_inputs():
    head, cases = load("selection_tiebreak.txt")
    L, K = int(head["L"]), int(head["K"])
    cand = np.array(groups(head["cand"], int), np.int32)
    edge = np.array(groups(head["edge"]), np.float32).reshape(L, K, K)
    return L, K, int(head["base_pos"]), cand, edge, cases


def test_golden_selection_and_emission():
    L, K, base, cand, edge, cases = _selection_inputs()
    sc = dict(emb=np.zeros((2, 1), np.float32), g_parent=np.zeros((1, 1), np.float32),
              g_child=np.zeros((1, 1), np.float32), depth_emb=None, scale=1, beta=0, center=0)
    P = oracle.make_params(L, K, 64, 1 << 20, sc)
    for c in cases:
        n = int(c["budget"])
        r = oracle.select_staged(P, cand, edge, n, base)
        assert r["n_nodes"] == n
        assert r["tokens"][:n].tolist() == nums(c["tokens"], int).tolist(), c["case"]
        assert r["parents"][:n].tolist() == nums(c["parents"], int).tolist(), c["case"]
        assert r["pos_ids"][:n].tolist() == nums(c["pos_ids"], int).tolist(), c["case"]
        assert r["mask"][:n, 0].tolist() == nums(c["mask"], int).tolist(), c["case"]
        assert r["node_scores"][:n].tolist() == nums(c["scores"]).tolist(), c["case"]
        assert (r["tokens"][n:] == -1).all() and (r["mask"][n:] == 0).all()


def _acceptance():
    head, cases = load("acceptance.txt")
    return nums(head["tokens"], int), nums(head["parents"], int), int(head["L"]), cases


def test_golden_acceptance():
    tokens, parents, L, cases = _acceptance()
    for c in cases:
        a, nodes, bonus = oracle.accept(len(tokens), tokens, parents, L,
                                        target_depth=nums(c["target_depth"], int))
        assert a == int(c["acc_len"]), c["case"]
        assert nodes.tolist() == nums(c["acc_nodes"], int).tolist(), c["case"]
        assert bonus == int(c["bonus"]), c["case"]


def test_golden_degen():
    head, _ = load("degen.txt")
    H = int(head["H"])
    h = np.array(groups(head["hidden"]), np.float32).reshape(-1, H)
    d, r = oracle.degen(bf16(h))
    assert np.allclose(r, nums(head["adj_cos"]), rtol=0, atol=1e-15)
    assert d == pytest.approx(float(head["degen"]), abs=1e-14)


# ---------------------------------------------------------------------------
# HIP path (GPU), same fixtures
# ---------------------------------------------------------------------------

def _ctx(torch, batch, L, V, K, n_max):
    import paper_2608_20375_amd as G
    ctx = G.Context(batch, L, V, K, n_max)
    f = lambda *s: torch.zeros(*s, dtype=torch.float32, device="cuda")
    ctx.set_scorer(f(V, 1), f(1, 1), f(1, 1), None, 1.0, 0.0, 0)
    return ctx


@pytest.mark.gpu
def test_golden_row_stats_gpu():
    torch = pytest.importorskip("torch")
    _, cases = load("row_stats.txt")
    for c in cases:
        x = bf16(nums(c["logits"]))
        V = x.size
        ctx = _ctx(torch, 1, 1, V, 1, 8)
        logits = torch.from_numpy(x.view(np.int16).reshape(1, 1, V)).cuda()
        z = torch.zeros(1, dtype=torch.int32, device="cuda")
        out = ctx.build_tree(logits, z, z, fixed_budget=z + 1)
        torch.cuda.synchronize()
        for key, got in (("lse", out.row_lse), ("maxprob", out.row_maxprob),
                         ("entropy", out.row_entropy)):
            ref = float(c[key])
            assert abs(float(got.item()) - ref) <= 1e-6 + 1e-5 * abs(ref), (c["case"], key)
        ctx.close()


@pytest.mark.gpu
def test_golden_acceptance_gpu():
    torch = pytest.importorskip("torch")
    tokens, parents, L, cases = _acceptance()
    n_max = 8
    ctx = _ctx(torch, 1, L, 16, 2, n_max)
    pad = lambda a: np.concatenate([a, -np.ones(n_max - a.size, np.int64)]).astype(np.int32)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()
    n = T([len(tokens)])
    tk, pr = T(pad(tokens)[None]), T(pad(parents)[None])
    for c in cases:
        a, nodes, bonus = ctx.accept(n, tk, pr, target_depth=T(nums(c["target_depth"], int)[None]))
        assert int(a.item()) == int(c["acc_len"]), c["case"]
        assert nodes.cpu().numpy()[0].tolist() == nums(c["acc_nodes"], int).tolist(), c["case"]
        assert int(bonus.item()) == int(c["bonus"]), c["case"]
    ctx.close()


@pytest.mark.gpu
def test_golden_degen_gpu():
    torch = pytest.importorskip("torch")
    head, _ = load("degen.txt")
    H = int(head["H"])
    h = np.array(groups(head["hidden"]), np.float32).reshape(-1, H)
    L = h.shape[0]
    hp = np.zeros((L, 8), np.float32)          # widths are multiples of 8: zero padding
    hp[:, :H] = h
    ctx = _ctx(torch, 1, L, 64, 2, 8)
    logits = torch.zeros(1, L, 64, dtype=torch.int16, device="cuda")
    z = torch.zeros(1, dtype=torch.int32, device="cuda")
    hid = torch.from_numpy(bf16(hp).view(np.int16)[None]).cuda()
    out = ctx.build_tree(logits, z, z, fixed_budget=z + 1, hidden=hid, adj_cos=True)
    torch.cuda.synchronize()
    r = out.adj_cos.cpu().numpy()[0]
    assert np.allclose(r, nums(head["adj_cos"]), rtol=1e-6, atol=1e-6)
    assert abs(float(out.saba_state[0, 1].item()) - float(head["degen"])) <= 1e-5
    ctx.close()
