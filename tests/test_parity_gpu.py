"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Bars: candidate ids, trees, masks, position ids, budgets and acceptance are
bit-exact; log-probabilities, row statistics and edge scores agree with the
fp64 oracle within 1e-5 relative (absolute floor 1e-6 for values near zero).
End-to-end parity holds on sequences whose inputs were re-drawn until every
floating-point decision has a margin of L * 2**-17 (see tests/workload.py);
staged parity (the oracle selecting on the GPU's own fp32 edge scores and
budget) is bit-exact on every sequence.
"""
import os
import sys
import time

import numpy as np
import pytest

import oracle
import synthetic as S

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import workload as WL  # noqa: E402

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

RTOL, ATOL = 1e-5, 1e-6


def _say(*a):
    print(*a, flush=True)


def close(gpu, ref, rtol=RTOL, atol=ATOL):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    return np.abs(gpu - ref) <= atol + rtol * np.abs(ref)


def check_tree_equal(g, b, r, n_max, words):
    n = r["n_nodes"]
    assert g["n_nodes"][b] == n
    assert np.array_equal(g["tokens"][b], r["tokens"])
    assert np.array_equal(g["parents"][b], r["parents"])
    assert np.array_equal(g["pos_ids"][b], r["pos_ids"])
    gm = g["mask"][b].view(np.uint64).reshape(n_max, words)
    assert np.array_equal(gm, r["mask"])


def staged_check(w, g, sc, sp, inp, seqs):
    P = oracle.make_params(w.L, w.K, w.n_max, w.V, sc, sp)
    words = (w.n_max + 63) // 64
    for b in seqs:
        st = oracle.select_staged(P, g["topk_ids"][b], g["edge_scores"][b], int(g["budget"][b]),
                                  int(inp["base_pos"][b]))
        check_tree_equal(g, b, st, w.n_max, words)
        n = st["n_nodes"]
        assert np.array_equal(g["node_scores"][b][:n], st["node_scores"][:n])


def saba_check(w, g, sc, sp, inp, seqs):
    if sp is None:
        assert np.array_equal(g["budget"], inp["fixed_budget"])
        return
    P = oracle.make_params(w.L, w.K, w.n_max, w.V, sc, sp)
    for b in seqs:
        conf = sum(float(v) for v in g["row_maxprob"][b]) / w.L
        ent = sum(float(v) for v in g["row_entropy"][b]) / w.L
        bud, tau, rel, _ = oracle.saba(P, conf, ent, float(inp["hist"][b]), int(inp["prefix_len"][b]))
        if rel > 1e-12:
            assert bud == g["budget"][b], (b, bud, g["budget"][b], rel)


def end_to_end_check(w, g, inp, results):
    words = (w.n_max + 63) // 64
    for b, r in results.items():
        assert np.array_equal(g["topk_ids"][b], r["topk_ids"]), b
        assert close(g["topk_logq"][b], r["topk_logq"]).all(), b
        assert close(g["row_lse"][b], r["row_lse"]).all(), b
        assert close(g["row_maxprob"][b], r["row_maxprob"]).all(), b
        assert close(g["row_entropy"][b], r["row_entropy"]).all(), b
        for l in range(w.L):
            rows = 1 if l == 0 else w.K
            assert close(g["edge_scores"][b, l, :rows], r["edge"][l, :rows]).all(), (b, l)
        assert g["budget"][b] == r["budget"], b
        check_tree_equal(g, b, r, w.n_max, words)
        n = r["n_nodes"]
        # a node's path score is the sum of the edge scores along its path
        # (eq. tdes-path-score), each within the edge bound above, so it is
        # within depth * ATOL + RTOL * (sum of |edge score| on the path)
        sc_r = r["node_scores"][:n].astype(np.float64)
        par = r["parents"][:n]
        abs_path = np.zeros(n)
        for i in range(n):
            p = int(par[i])
            abs_path[i] = abs(sc_r[i]) if p < 0 else abs_path[p] + abs(sc_r[i] - sc_r[p])
        err = np.abs(g["node_scores"][b][:n] - sc_r)
        bound = r["depth"][:n] * ATOL + RTOL * abs_path
        assert (err <= bound).all(), (b, float((err / bound).max()))


# ---------------------------------------------------------------------------
# logits pass on shapes that exercise tiles, splits and ragged rows
# ---------------------------------------------------------------------------

SHAPES = [
    # batch, L, V, K
    (1, 3, 40, 32),        # a row shorter than one tile, K close to V
    (2, 4, 777, 8),        # V % 8 != 0: misaligned rows, scalar head/tail
    (1, 2, 5003, 16),      # several tiles + ragged tail, split rows
    (3, 5, 20000, 4),
    (2, 3, 70001, 64),     # K = 64 (the 256-entry buffer variant)
    (4, 2, 9, 1),          # K = 1: DFlash's argmax draft
]


@pytest.mark.parametrize("shape", SHAPES)
def test_logits_pass_topk_and_stats(shape):
    B, L, V, K = shape
    _say("logits pass", shape)
    w = S.workload(0, batch=B, L=L, V=V, K=K, n_max=64, fixed_budget=8)
    inp = S.gen_round(w, with_targets=False)
    # many exact ties among tail values: quantise part of the rows
    g = np.random.default_rng(V)
    x = S.f32_from_bf16(inp["logits"])
    q = np.round(x * 4) / 4
    x = np.where(g.random(x.shape) < 0.5, q, x)
    inp["logits"] = S.bf16_from_f32(x)
    sc = WL.scorer_inputs(w, "literal")
    ctx = WL.gpu_context(w, sc, None, torch)
    gr = WL.gpu_round(ctx, w, inp, torch)
    for b in range(B):
        for l in range(L):
            row = inp["logits"][b, l]
            ids, xv = oracle.topk(row, K)
            lse, mp, h = oracle.row_stats(row)
            assert np.array_equal(gr["topk_ids"][b, l], ids), (b, l)
            assert close(gr["topk_logq"][b, l], xv - lse).all()
            assert close(gr["row_lse"][b, l], lse)
            assert close(gr["row_maxprob"][b, l], mp)
            assert close(gr["row_entropy"][b, l], h)
    ctx.close()


# ---------------------------------------------------------------------------
# whole round, every workload (full sizes; the oracle on every sequence)
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("wid", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("mode", ["literal", "paper"])
def test_round_parity(wid, mode):
    w = S.workload(wid)
    _say("round parity workload", wid, mode)
    t0 = time.time()
    inp, sc, sp, results = WL.audited_round(w, 0, mode)
    assert len(results) == w.batch
    _say("  inputs ready in %.1fs (%d oracle threads); attempts per sequence: mean %.2f, max %d"
         % (time.time() - t0, WL.oracle_threads(), inp["attempts"].mean() + 1,
            inp["attempts"].max() + 1))
    ctx = WL.gpu_context(w, sc, sp, torch)
    g = WL.gpu_round(ctx, w, inp, torch)
    _say("  gpu done; budgets", g["budget"][:8].tolist(), "nodes", g["n_nodes"][:8].tolist())
    end_to_end_check(w, g, inp, results)
    seqs = range(w.batch)
    staged_check(w, g, sc, sp, inp, seqs)
    saba_check(w, g, sc, sp, inp, seqs)
    acc = accept_check(ctx, w, g, inp, results, w.seed)
    _say("  accepted nodes per sequence: mean %.2f, max %d" % (acc.mean(), acc.max()))
    assert ctx.device_status() == 0
    ctx.close()


def accept_check(ctx, w, g, inp, results, seed, update_history=False):
    """The acceptance walk on the GPU's trees against the oracle's walk, every
    sequence: per-depth targets from the inputs, or per-node targets drawn on
    the device (graft_synth_node_targets) and checked against their CPU twin on
    the oracle's trees.  Returns the accepted lengths."""
    out = g["_out"]
    if w.targets == "depth":
        acc = ctx.accept(out.n_nodes, out.tokens, out.parents,
                         target_depth=torch.from_numpy(inp["target_depth"]).cuda(),
                         update_history=update_history)
        acc = [a.cpu().numpy() for a in acc]
        for b in range(w.batch):
            a, nodes, bonus = oracle.accept(g["n_nodes"][b], g["tokens"][b], g["parents"][b],
                                            w.L, target_depth=inp["target_depth"][b])
            assert acc[0][b] == a and acc[2][b] == bonus, b
            assert np.array_equal(acc[1][b], nodes), b
        return acc[0]
    tr, tn = ctx.synth_node_targets(seed, torch.from_numpy(inp["root_token"]).cuda(),
                                    out.n_nodes, out.tokens, out.parents, out.topk_ids)
    acc = ctx.accept(out.n_nodes, out.tokens, out.parents, target_root=tr, target_node=tn,
                     update_history=update_history)
    acc = [a.cpu().numpy() for a in acc]
    tr, tn = tr.cpu().numpy(), tn.cpu().numpy()
    assert len(results) == w.batch
    for b, r in results.items():
        n = r["n_nodes"]
        par, tok, dep = r["parents"][:n], r["tokens"][:n], r["depth"][:n]
        ptok = np.where(par < 0, inp["root_token"][b], r["tokens"][np.maximum(par, 0)])
        ref_nodes = S.node_targets(seed, b, dep, ptok, tok, r["topk_ids"], w.V, w.L, w.K)
        ref_root = S.node_targets(seed, b, [0], [-1], [inp["root_token"][b]], r["topk_ids"],
                                  w.V, w.L, w.K)[0]
        assert tr[b] == ref_root, b
        assert np.array_equal(tn[b][:n], ref_nodes), b
        a, nodes, bonus = oracle.accept(n, r["tokens"], r["parents"], w.L, int(ref_root),
                                        target_node=np.concatenate(
                                            [ref_nodes, -np.ones(w.n_max - n, np.int32)]))
        assert acc[0][b] == a and acc[2][b] == bonus, b
        assert np.array_equal(acc[1][b], nodes), b
    return acc[0]


CHAIN_ROUNDS = 5


def test_chained_rounds_w4():
    """Five consecutive full-size rounds of workload 4 (batch 128, L 32, V
    151936, K 32), as its 50-round run chains them: each round's acceptance
    pushes acc_len into the device history ring (window 4, so the fifth push
    wraps to slot 0) and the next round's SABA reads the ring's mean as hist_t.
    Round r is audited with the oracle after round r-1's acceptance, with the
    oracle's hist equal to the ring mean; budgets, trees, masks, acceptance and
    the ring contents are compared every round."""
    w = S.workload(4)
    sc, sp = WL.scorer_inputs(w, "literal"), WL.saba_inputs(w)
    ctx = WL.gpu_context(w, sc, sp, torch)
    ring = S.hist_ring_init(w)
    ctx.set_history(torch.from_numpy(ring).cuda())
    pos = np.zeros(w.batch, np.int64)
    for rnd in range(CHAIN_ROUNDS):
        t0 = time.time()
        hist = ring.astype(np.float64).mean(axis=1)
        inp, _, _, results = WL.audited_round(w, rnd, "literal", hist=hist)
        _say("chained w4 round %d: audited in %.1fs, attempts mean %.2f" %
             (rnd, time.time() - t0, inp["attempts"].mean() + 1))
        g = WL.gpu_round(ctx, w, inp, torch, use_ring=True)
        assert (g["saba_state"][:, 2] == hist.astype(np.float32)).all()
        end_to_end_check(w, g, inp, results)
        staged_check(w, g, sc, sp, inp, range(w.batch))
        a = accept_check(ctx, w, g, inp, results, w.seed + rnd, update_history=True)
        for b in range(w.batch):
            ring[b, pos[b]] = a[b]
        pos = (pos + 1) % S.HIST_WINDOW
        dring, dpos = (x.cpu().numpy() for x in ctx.get_history(w.batch))
        assert np.array_equal(dring, ring)
        assert np.array_equal(dpos, pos)
        _say("  accepted mean %.2f; ring pos %d" % (a.mean(), pos[0]))
    assert ctx.device_status() == 0
    ctx.close()


def _peaked_chain(b, logits):
    """Even sequences: the rank-1 candidate of every depth gets +6.5 (log q
    about -0.2 to -1.5), so the chain of rank-1 candidates reaches depth L
    inside the budget while every edge score stays negative (a larger boost
    lets the interaction term push some above 0, and packs the near-free chain
    extensions of every sibling into score gaps below the audit's margin)."""
    if b % 2:
        return
    x = S.f32_from_bf16(logits)
    top = np.argmax(x, axis=1)
    x[np.arange(x.shape[0]), top] += 6.5
    logits[:] = S.bf16_from_f32(x)


def deep_targets(w, g, seed=4242):
    """Targets whose walk follows each tree's deepest root path to its end:
    per-depth td [batch, L + 1] (entry k = token of the path's node at depth
    k + 1) and per-node (troot = the path's first token, node path[k] ->
    token of path[k + 1]); every other entry is a seeded draw.  Returns
    (td, troot, tnode, [(depth, path)] per sequence)."""
    rng = np.random.default_rng(seed)
    td = rng.integers(0, w.V, size=(w.batch, w.L + 1)).astype(np.int32)
    tnode = rng.integers(0, w.V, size=(w.batch, w.n_max)).astype(np.int32)
    troot = rng.integers(0, w.V, size=w.batch).astype(np.int32)
    want = []
    for b in range(w.batch):
        n = int(g["n_nodes"][b])
        par, tok = g["parents"][b], g["tokens"][b]
        depth = np.zeros(n, np.int64)
        for i in range(n):
            depth[i] = 1 if par[i] < 0 else depth[par[i]] + 1
        j = int(np.argmax(depth))               # deepest node, lowest index first
        path = []
        while j >= 0:
            path.append(j)
            j = int(par[j])
        path = path[::-1]
        for k, j in enumerate(path):
            td[b, k] = tok[j]
        troot[b] = tok[path[0]]
        for k in range(len(path) - 1):
            tnode[b, path[k]] = tok[path[k + 1]]
        tnode[b, n:] = -1
        want.append((len(path), path))
    return td, troot, tnode, want


def test_deep_acceptance_w3():
    """Acceptance walks that follow each tree's deepest root path to its end
    (full-size workload 3; even sequences have a dominant chain, so their trees
    reach depth L = 16 and the bonus token comes from target_depth[L]).  The
    path's nodes lie past the first 64 canonical indices, so the walk scans
    several 64-node chunks.  Per-depth and per-node targets."""
    w = S.workload(3)
    inp, sc, sp, results = WL.audited_round(w, 0, "literal", transform=_peaked_chain)
    ctx = WL.gpu_context(w, sc, sp, torch)
    g = WL.gpu_round(ctx, w, inp, torch)
    end_to_end_check(w, g, inp, results)
    td, troot, tnode, want = deep_targets(w, g)
    for b in range(0, w.batch, 2):
        assert want[b][0] == w.L, (b, want[b][0])
    assert max(p[-1] for _, p in want) >= 64
    out = g["_out"]
    for mode in ("depth", "node"):
        if mode == "depth":
            acc = ctx.accept(out.n_nodes, out.tokens, out.parents,
                             target_depth=torch.from_numpy(td).cuda())
        else:
            acc = ctx.accept(out.n_nodes, out.tokens, out.parents,
                             target_root=torch.from_numpy(troot).cuda(),
                             target_node=torch.from_numpy(tnode).cuda())
        a, nodes, bonus = (x.cpu().numpy() for x in acc)
        for b, (D, path) in enumerate(want):
            assert a[b] == D, (mode, b, a[b], D)
            assert np.array_equal(nodes[b][:D], path) and (nodes[b][D:] == -1).all()
            ra, rn, rb = (oracle.accept(g["n_nodes"][b], g["tokens"][b], g["parents"][b], w.L,
                                        target_depth=td[b]) if mode == "depth" else
                          oracle.accept(g["n_nodes"][b], g["tokens"][b], g["parents"][b], w.L,
                                        int(troot[b]), target_node=tnode[b]))
            assert (ra, rb) == (a[b], bonus[b]) and np.array_equal(rn, nodes[b])
            assert bonus[b] == (td[b, D] if mode == "depth" else tnode[b, path[-1]])
    _say("deep acceptance: depths", sorted(set(D for D, _ in want)))
    assert ctx.device_status() == 0
    ctx.close()


def test_largest_supported_sizes():
    """Every size at the library's limit at once: L = 64 depths, K = 64
    candidates, N_max = 1024 nodes, score dimension 64, a 64-entry history
    ring whose mean is SABA's hist_t, and a grid of 63 budgets up to 1024.  A
    sequence's edge rows (1 MiB) exceed selection's LDS stage, so only the
    first depth is staged; the masks are 16 words a row.  End-to-end parity
    with the oracle on every sequence (even sequences get a dominant chain, so
    their trees reach depth 64), then acceptance along each tree's deepest
    path: acc_len = 64 and the bonus token from target_depth[64]."""
    import paper_2608_20375_amd as G
    w = S.workload(4, batch=3, L=64, V=4099, K=64, n_max=1024, emb_dim=64, rank=64,
                   targets="depth")
    rng = np.random.default_rng(77)
    ring = rng.integers(0, w.L + 1, size=(w.batch, 64)).astype(np.int32)
    hist = ring.astype(np.float64).mean(axis=1)
    inp, sc, sp, results = WL.audited_round(w, 0, "paper", hist=hist, transform=_peaked_chain)
    assert len(results) == w.batch
    ctx = G.Context(w.batch, w.L, w.V, w.K, w.n_max, 64)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    ctx.set_scorer(T(sc["emb"]), T(sc["g_parent"]), T(sc["g_child"]), T(sc["depth_emb"]),
                   sc["scale"], sc["beta"], sc["center"])
    ctx.set_saba(list(sp["grid"]), list(sp["phi"]), sp["tau_min"], sp["c0"], sp["c1"], sp["c2"])
    ctx.set_history(T(ring))
    g = WL.gpu_round(ctx, w, inp, torch, use_ring=True)
    end_to_end_check(w, g, inp, results)
    staged_check(w, g, sc, sp, inp, range(w.batch))
    td, troot, tnode, want = deep_targets(w, g)
    for b in range(0, w.batch, 2):
        assert want[b][0] == w.L, (b, want[b][0])
    out = g["_out"]
    acc = ctx.accept(out.n_nodes, out.tokens, out.parents, target_depth=T(td))
    a, nodes, bonus = (x.cpu().numpy() for x in acc)
    for b, (D, path) in enumerate(want):
        ra, rn, rb = oracle.accept(g["n_nodes"][b], g["tokens"][b], g["parents"][b], w.L,
                                   target_depth=td[b])
        assert (ra, rb) == (a[b], bonus[b]) and np.array_equal(rn, nodes[b])
        assert a[b] == D and bonus[b] == td[b, D]
    _say("largest sizes: budgets", g["budget"].tolist(), "depths", [D for D, _ in want])
    assert ctx.device_status() == 0
    ctx.close()


def _frontier_check(w, g, b, logq):
    """The selected set of sequence b is the first N prefixes of the whole trie
    under the heap order (higher path score, then smaller depth, then the
    smaller token path), with path scores the fp64 sums of the GPU's fp32 log q:
    it is prefix-closed and no unselected child of a selected prefix (or of the
    root) precedes its last selected prefix.  Valid because every score is <= 0,
    so a child never precedes its parent."""
    n = int(g["n_nodes"][b])
    tok, par = g["tokens"][b][:n], g["parents"][b][:n]
    ids = g["topk_ids"][b]
    path, score = [], []
    for i in range(n):
        p = int(par[i])
        d = 1 if p < 0 else len(path[p]) + 1
        slot = int(np.flatnonzero(ids[d - 1] == tok[i])[0])
        path.append((() if p < 0 else path[p]) + (int(tok[i]),))
        score.append((0.0 if p < 0 else score[p]) + float(logq[d - 1][slot]))
        assert score[i] == g["node_scores"][b][i]
    key = lambda s, pth: (-s, len(pth), pth)
    worst_selected = max(key(s, p) for s, p in zip(score, path))
    chosen = set(path)
    best_left = None
    for parent_path, parent_score in [((), 0.0)] + list(zip(path, score)):
        d = len(parent_path)
        if d == w.L:
            continue
        for slot in range(w.K):
            cp = parent_path + (int(ids[d][slot]),)
            if cp in chosen:
                continue
            k = key(parent_score + float(logq[d][slot]), cp)
            best_left = k if best_left is None or k < best_left else best_left
    assert best_left is None or worst_selected < best_left


def test_ddtree_mode_beta0_w3():
    """DDTree mode on the HIP path (eq. ddtree-path-score): the paper-mode scorer
    with beta = 0 leaves every edge score equal to log q of the child, so the
    tree is the top-budget product-of-probability tree.  Exact ties between
    sums of bf16 log-probabilities are common here; end-to-end parity holds on
    sequences re-drawn until the boundary has a margin, staged parity on every
    sequence, and each tree is checked to be the first N prefixes of the trie."""
    w = S.workload(3)
    sc = WL.scorer_inputs(w, "paper")
    sc["beta"] = 0.0
    inp, sc, sp, results = WL.audited_round(w, 0, "paper", scorer=sc)
    _say("beta = 0: attempts per sequence mean %.2f" % (inp["attempts"].mean() + 1))
    ctx = WL.gpu_context(w, sc, sp, torch)
    g = WL.gpu_round(ctx, w, inp, torch)
    end_to_end_check(w, g, inp, results)
    staged_check(w, g, sc, sp, inp, range(w.batch))
    for b in range(w.batch):
        lq = g["topk_logq"][b]
        e = g["edge_scores"][b]
        assert (e[0, 0] == lq[0]).all()
        assert (e[1:] == lq[1:, None, :]).all()
        _frontier_check(w, g, b, lq)
    assert ctx.device_status() == 0
    ctx.close()


EDGE_SHAPES = [
    # K, score dim m, embedding dim
    (1, 8, 16),       # K = 1: one lane per parent run, 64 parents a pass
    (5, 30, 32),      # m % 4 != 0: the element-wise gathers instead of 16-byte ones
    (13, 20, 32),     # m = 20 (VALU passes): K = 13 in runs of 16 lanes, 4 parents a pass
    (33, 64, 64),     # K = 33, m = 64: three column tiles of the matrix-core path, one partial
    (20, 48, 32),     # m = 48: twelve k-slots a lane, two column tiles
    (64, 64, 64),     # the largest K and m: four parent tiles by four column tiles
]


@pytest.mark.parametrize("K,m,E", EDGE_SHAPES)
@pytest.mark.parametrize("mode", ["literal", "paper"])
def test_edge_score_shapes(K, m, E, mode):
    """Edge scores (and the trees selected on them) at candidate counts and
    score dimensions that the workloads above do not reach."""
    _say("edge shapes", K, m, E, mode)
    w = S.workload(0, batch=3, L=5, V=3000, K=K, n_max=128, fixed_budget=100, emb_dim=E, rank=m)
    inp, sc, sp, results = WL.audited_round(w, 0, mode, seqs=None)
    ctx = WL.gpu_context(w, sc, sp, torch)
    g = WL.gpu_round(ctx, w, inp, torch)
    end_to_end_check(w, g, inp, results)
    staged_check(w, g, sc, sp, inp, range(w.batch))
    assert ctx.device_status() == 0
    ctx.close()


# Sizes at which the selection kernel computes the edge scores and the budget
# itself (graft_set_fusion): workload id, overrides, scorer mode, hidden dim
FUSION_CASES = [
    (0, {}, "literal", 0),                  # L = 8, K = 4: one depth a wave, fixed budgets
    (2, {}, "paper", 0),                    # K = 8, m = 16, SABA, centered scores
    (3, {"batch": 16}, "literal", 0),       # K = 16, m = 32: two depths a wave
    (3, {"batch": 8}, "paper", 64),         # SABA on the hidden-state degeneration signal
    (0, dict(batch=3, L=5, V=3000, K=13, n_max=128, fixed_budget=100, emb_dim=32, rank=16),
     "paper", 0),                           # K = 13: a partial 16 x 16 tile, m = 16
    (0, dict(batch=2, L=4, V=3000, K=24, n_max=256, fixed_budget=200, emb_dim=32, rank=16),
     "paper", 0),                           # K = 24: two column tiles, the second partial
    (0, dict(batch=2, L=1, V=3000, K=64, n_max=64, fixed_budget=64, emb_dim=32, rank=32),
     "literal", 0),                         # K = 64: four column tiles, one depth
    (0, dict(batch=3, L=12, V=3000, K=1, n_max=16, fixed_budget=12, emb_dim=16, rank=16),
     "literal", 0),                         # K = 1, L = 12: waves 0-3 take two depths
    (0, dict(batch=2, L=64, V=3000, K=8, n_max=256, fixed_budget=200, emb_dim=32, rank=16),
     "paper", 0),                           # L K = 512: every thread ranks a candidate, the
                                            # budget wave included; eight depths a wave
    (0, dict(batch=2, L=40, V=3000, K=8, n_max=256, fixed_budget=200, emb_dim=32, rank=32),
     "literal", 0),                         # 5120 projection loads: two gather batches
]


@pytest.mark.parametrize("case", range(len(FUSION_CASES) + 1))
def test_fused_edges_match_edge_stage(case):
    """The fused path (edge scores and budget inside the selection kernel)
    and the separate edge stage give the same bits for every output; the
    last case has positive edge scores, so both run the serial selector."""
    if case < len(FUSION_CASES):
        wid, kw, mode, hd = FUSION_CASES[case]
        w = S.workload(wid, **kw)
        inp, sc, sp, _ = WL.audited_round(w, 0, mode, seqs=[], hidden_dim=hd or None)
    else:
        w = S.workload(0, batch=2, V=3000, L=5, K=3, n_max=64, fixed_budget=40)
        inp, sc, sp, _ = WL.audited_round(w, 0, "paper", seqs=[])
        sc["beta"] = 400.0
        sp = None
    _say("fusion case", case, w)
    ctx = WL.gpu_context(w, sc, sp, torch)
    assert ctx.set_fusion(True)
    fused = WL.gpu_round(ctx, w, inp, torch)
    assert not ctx.set_fusion(False)
    staged = WL.gpu_round(ctx, w, inp, torch)
    if case == len(FUSION_CASES):
        assert (fused["edge_scores"] > 0).any()
    for k, v in fused.items():
        if not k.startswith("_"):
            assert np.array_equal(v, staged[k]), k
    assert ctx.device_status() == 0
    ctx.close()


def test_budgets_spread_under_saba():
    """SABA picks several distinct budgets across the batch of workload 2."""
    w = S.workload(2)
    inp = S.gen_round(w, with_targets=False)
    sc, sp = WL.scorer_inputs(w, "literal"), WL.saba_inputs(w)
    ctx = WL.gpu_context(w, sc, sp, torch)
    g = WL.gpu_round(ctx, w, inp, torch)
    assert len(set(g["budget"].tolist())) >= 3
    ctx.close()


def test_determinism_bitwise():
    w = S.workload(3, batch=8)
    inp = S.gen_round(w, with_targets=False)
    sc, sp = WL.scorer_inputs(w, "literal"), WL.saba_inputs(w)
    ctx = WL.gpu_context(w, sc, sp, torch)
    first = WL.gpu_round(ctx, w, inp, torch)
    for _ in range(5):
        again = WL.gpu_round(ctx, w, inp, torch)
        for k in ("topk_ids", "topk_logq", "row_lse", "edge_scores", "budget", "tokens",
                  "parents", "mask", "node_scores"):
            assert np.array_equal(first[k], again[k]), k
    ctx.close()


def test_positive_edge_scores_staged():
    """Non-monotone path scores (a positive interaction term larger than
    -log q): the selection still matches the oracle bit for bit."""
    w = S.workload(0, batch=2, V=3000, L=5, K=3, n_max=64, fixed_budget=40)
    inp = S.gen_round(w, with_targets=False)
    sc = WL.scorer_inputs(w, "paper")
    sc["beta"] = 400.0                     # residual dominates log q
    ctx = WL.gpu_context(w, sc, None, torch)
    g = WL.gpu_round(ctx, w, inp, torch)
    assert (g["edge_scores"] > 0).any()
    staged_check(w, g, sc, None, inp, range(w.batch))
    ctx.close()


def test_history_ring_chain():
    """Chained rounds: acceptance pushes acc_len into the device ring and the
    next round's SABA reads the ring mean."""
    w = S.workload(2, batch=4, V=4000)
    sc, sp = WL.scorer_inputs(w, "literal"), WL.saba_inputs(w)
    ctx = WL.gpu_context(w, sc, sp, torch)
    ring = S.hist_ring_init(w)
    ctx.set_history(torch.from_numpy(ring).cuda())
    P = oracle.make_params(w.L, w.K, w.n_max, w.V, sc, sp)
    pos = np.zeros(w.batch, int)
    for rnd in range(4):
        inp = S.gen_round(w, rnd)
        g = WL.gpu_round(ctx, w, inp, torch, use_ring=True)
        hist = ring.astype(np.float64).mean(axis=1)
        for b in range(w.batch):
            assert g["saba_state"][b, 2] == np.float32(hist[b])
            conf = sum(float(v) for v in g["row_maxprob"][b]) / w.L
            ent = sum(float(v) for v in g["row_entropy"][b]) / w.L
            bud, _, rel, _ = oracle.saba(P, conf, ent, float(hist[b]), int(inp["prefix_len"][b]))
            if rel > 1e-12:
                assert bud == g["budget"][b]
        acc = ctx.accept(g["_out"].n_nodes, g["_out"].tokens, g["_out"].parents,
                         target_depth=torch.from_numpy(inp["target_depth"]).cuda(),
                         update_history=True)
        a = acc[0].cpu().numpy()
        for b in range(w.batch):
            ring[b, pos[b]] = a[b]
            pos[b] = (pos[b] + 1) % S.HIST_WINDOW
    ctx.close()


def test_abi_errors_on_device():
    import paper_2608_20375_amd as G
    w = S.workload(0, batch=2, V=1000)
    sc = WL.scorer_inputs(w, "literal")
    ctx = G.Context(2, w.L, w.V, w.K, w.n_max)
    logits = torch.zeros(2, w.L, w.V, dtype=torch.int16, device="cuda")
    root = torch.zeros(2, dtype=torch.int32, device="cuda")
    # no scorer yet
    with pytest.raises(G.GraftError) as e:
        ctx.build_tree(logits, root, root, fixed_budget=root)
    assert e.value.status == 1
    T = lambda a: torch.from_numpy(a).cuda()
    ctx.set_scorer(T(sc["emb"]), T(sc["g_parent"]), T(sc["g_child"]), None, sc["scale"], 1.0, 0)
    # SABA without parameters
    with pytest.raises(G.GraftError):
        ctx.build_tree(logits, root, root, hist=torch.zeros(2, device="cuda"))
    # bad SABA grids
    for grid in ([32, 16], [0, 8], [8, 10 ** 6], list(range(1, 70))):
        with pytest.raises(G.GraftError):
            ctx.set_saba(grid, [1, 0, 0, 0])
    # batch too large
    big = torch.zeros(3, w.L, w.V, dtype=torch.int16, device="cuda")
    r3 = torch.zeros(3, dtype=torch.int32, device="cuda")
    with pytest.raises(G.GraftError):
        ctx.build_tree(big, r3, r3, fixed_budget=r3)
    # misaligned logits
    flat = torch.zeros(2 * w.L * w.V + 8, dtype=torch.int16, device="cuda")
    mis = flat[1:1 + 2 * w.L * w.V].view(2, w.L, w.V)
    with pytest.raises(G.GraftError):
        ctx.build_tree(mis, root, root, fixed_budget=root)
    # out-of-range root token is reported by the device status
    bad_root = torch.full((2,), w.V + 5, dtype=torch.int32, device="cuda")
    ctx.build_tree(logits, bad_root, root, fixed_budget=torch.full((2,), 4, dtype=torch.int32,
                                                                   device="cuda"))
    assert ctx.device_status() == 5
    assert ctx.device_status() == 0
    # accept needs exactly one target mode
    n = torch.zeros(2, dtype=torch.int32, device="cuda")
    tk = torch.zeros(2, w.n_max, dtype=torch.int32, device="cuda")
    with pytest.raises(G.GraftError):
        ctx.accept(n, tk, tk)
    # buffers of the wrong shape are refused by the binding before any launch
    with pytest.raises(ValueError):
        ctx.build_tree(logits[:, :, :-8], root, root, fixed_budget=root)
    with pytest.raises(ValueError):
        ctx.build_tree(logits, root[:1], root, fixed_budget=root)
    with pytest.raises(ValueError):
        ctx.accept(n, tk[:, :-1], tk, target_depth=torch.zeros(2, w.L + 1, dtype=torch.int32,
                                                                device="cuda"))
    with pytest.raises(ValueError):
        ctx.accept(n, tk, tk, target_depth=torch.zeros(2, w.L, dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError):
        ctx.set_scorer(T(sc["emb"][:-1]), T(sc["g_parent"]), T(sc["g_child"]), None, 1.0, 1.0, 0)
    ctx.close()


def test_zero_budget_and_tiny_trees():
    w = S.workload(0, batch=3, V=2000, n_max=32)
    inp = S.gen_round(w)
    inp["fixed_budget"] = np.array([0, 1, 32], np.int32)
    sc = WL.scorer_inputs(w, "literal")
    ctx = WL.gpu_context(w, sc, None, torch)
    g = WL.gpu_round(ctx, w, inp, torch)
    assert g["n_nodes"].tolist() == [0, 1, 32]
    assert (g["tokens"][0] == -1).all() and (g["mask"][0] == 0).all()
    staged_check(w, g, sc, None, inp, range(3))
    acc = ctx.accept(g["_out"].n_nodes, g["_out"].tokens, g["_out"].parents,
                     target_depth=torch.from_numpy(inp["target_depth"]).cuda())
    a, nodes, bonus = [x.cpu().numpy() for x in acc]
    assert a[0] == 0 and bonus[0] == inp["target_depth"][0, 0]
    ctx.close()


@pytest.mark.parametrize("L,K,V,n_max", [(6, 8, 3000, 128), (20, 16, 5000, 512)])
def test_first_expansion_bound_budget_edges(L, K, V, n_max):
    """Budgets on both sides of K and of K + K^2, where the selector switches
    between bounding the first expansion by one histogram of the depth-1 and
    depth-2 prefixes and counting the depth-1 children first; the first shape
    stages its edge rows in LDS, the second (L * K * K > 4096) reads them from
    device memory.  beta = 0 (edge scores = log q <= 0) keeps every sequence
    on the parallel selector."""
    budgets = [K - 1, K, K + 1, K + K * K - 1, K + K * K, K + K * K + 1]
    w = S.workload(0, batch=len(budgets), L=L, K=K, V=V, n_max=n_max, fixed_budget=n_max)
    inp = S.gen_round(w)
    inp["fixed_budget"] = np.array(budgets, np.int32)
    sc = WL.scorer_inputs(w, "paper")
    sc["beta"] = 0.0
    ctx = WL.gpu_context(w, sc, None, torch)
    g = WL.gpu_round(ctx, w, inp, torch)
    assert (g["edge_scores"] <= 0).all()
    assert g["n_nodes"].tolist() == budgets
    staged_check(w, g, sc, None, inp, range(w.batch))
    assert ctx.device_status() == 0
    ctx.close()


@pytest.mark.parametrize("K", [16, 64])
def test_flat_scores_force_pool_compaction(K):
    """Uniform logits and a zero scorer make every edge score equal (and a few
    tie levels in the second sequence).  K = 64: the first expansion overflows
    the pool, partial expansions and tie ranking follow, and a later expansion
    only fits after the dead entries are compacted (the runs of children are
    remapped).  K = 16: the first expansion runs over (parent, child) pairs and
    fills the depth-1 entries' runs; the prune bound admits all 4,096 depth-3
    children, which do not fit, so 239 of the 256 depth-2 entries are
    expanded; the exact selection ranks 3,824 tied entries; the children of
    the last 17 depth-2 entries fit only after the pool is compacted; the
    preorder numbering reads the remapped runs.  The trees must still match
    the oracle bit for bit."""
    w = S.workload(0, batch=2, V=3000, L=4, K=K, n_max=1024, fixed_budget=1024)
    inp = S.gen_round(w, with_targets=False)
    flat = np.zeros((w.L, w.V), np.float32)
    g = np.random.default_rng(9)
    levels = -g.integers(0, 3, size=(w.L, w.V)).astype(np.float32)
    inp["logits"] = np.stack([S.bf16_from_f32(flat), S.bf16_from_f32(levels)])
    sc = WL.scorer_inputs(w, "literal")
    sc["g_parent"] = np.zeros_like(sc["g_parent"])
    sc["g_child"] = np.zeros_like(sc["g_child"])
    ctx = WL.gpu_context(w, sc, None, torch)
    gr = WL.gpu_round(ctx, w, inp, torch)
    assert gr["n_nodes"].tolist() == [1024, 1024]
    assert (gr["edge_scores"][0, 1:] == gr["edge_scores"][0, 1, 0, 0]).all()
    staged_check(w, gr, sc, None, inp, range(w.batch))
    assert ctx.device_status() == 0
    ctx.close()
