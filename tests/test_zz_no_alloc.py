"""graft_build_tree_static (no device allocation; the round's intermediates in
the library's static array) against graft_build_tree on the same inputs,
through the C ABI.  Both run the same kernels, so every output must be
identical bit for bit: candidates, log q, row statistics, edge scores, SABA
state, budgets, trees, masks, node scores, hidden-state cosines."""
import dataclasses
import os
import sys

import numpy as np
import pytest

import synthetic as S

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import workload as WL  # noqa: E402

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

FIELDS = ("budget", "n_nodes", "tokens", "parents", "pos_ids", "mask", "topk_ids", "topk_logq",
          "row_lse", "row_maxprob", "row_entropy", "edge_scores", "node_scores", "saba_state",
          "adj_cos")


def _say(*a):
    print(*a, flush=True)


def _inputs(w, rnd, batch, hidden_dim=None):
    wb = dataclasses.replace(w, batch=batch)
    inp = S.gen_round(wb, rnd)
    if hidden_dim:
        inp["hidden"] = S.gen_hidden(wb, rnd, hidden_dim)
    return inp


def _build(ctx, inp, static, hidden=False):
    import paper_2608_20375_amd as G
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    batch = inp["logits"].shape[0]
    out = G.TreeBuffers(ctx, batch, edges=True, adj_cos=hidden)
    ctx.build_tree(T(inp["logits"].view(np.int16)), T(inp["root_token"]), T(inp["base_pos"]),
                   prefix_len=T(inp["prefix_len"]), hist=T(inp["hist"]),
                   fixed_budget=T(inp["fixed_budget"]) if "fixed_budget" in inp else None,
                   hidden=T(inp["hidden"].view(np.int16)) if hidden else None,
                   out=out, static_scratch=static)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.as_dict().items()}


def _same(a, b):
    assert set(a) == set(b)
    for k in FIELDS:
        if k in a:
            assert np.array_equal(a[k], b[k]), k


def test_static_equals_workspace_two_calls_then_smaller():
    """Workload 3 (batch 64, L 16, V 128256, K 16, SABA), then a smaller call
    (8 sequences of the next round, with drafter hidden states) on the same
    context: the second static call reuses the array the first one filled."""
    w = S.workload(3)
    sc, sp = WL.scorer_inputs(w, "literal"), WL.saba_inputs(w)
    ctx = WL.gpu_context(w, sc, sp, torch)
    first = _inputs(w, 0, w.batch)
    _say("static build, batch", w.batch)
    st = _build(ctx, first, True)
    ws = _build(ctx, first, False)
    _same(st, ws)
    assert len(set(st["budget"].tolist())) >= 3
    second = _inputs(w, 1, 8, hidden_dim=512)
    _say("static build, batch 8 with hidden states")
    st2 = _build(ctx, second, True, hidden=True)
    ws2 = _build(ctx, second, False, hidden=True)
    _same(st2, ws2)
    assert (st2["adj_cos"] != 0).any()
    assert ctx.device_status() == 0
    ctx.close()


def test_static_at_the_largest_workload():
    """Workload 4 (batch 128, L 32, V 151936, K 32): about 18 MB of the 24 MiB
    array; then workload 0 (one sequence, split rows: the split-row partials
    are carved from the array too) on a second context of the same GPU."""
    w = S.workload(4)
    sc, sp = WL.scorer_inputs(w, "paper"), WL.saba_inputs(w)
    ctx = WL.gpu_context(w, sc, sp, torch)
    inp = _inputs(w, 0, w.batch)
    _say("static build, workload 4")
    _same(_build(ctx, inp, True), _build(ctx, inp, False))
    assert ctx.device_status() == 0
    ctx.close()
    w0 = S.workload(0)
    ctx0 = WL.gpu_context(w0, WL.scorer_inputs(w0, "literal"), None, torch)
    inp0 = _inputs(w0, 0, 1)
    _same(_build(ctx0, inp0, True), _build(ctx0, inp0, False))
    ctx0.close()


def test_static_rejects_a_batch_beyond_the_array():
    """L 64 and K 64: edge rows alone take 64 * 64 * 64 * 4 bytes per sequence,
    so 128 sequences need more than the array holds (GRAFT_ERR_UNSUPPORTED,
    nothing enqueued); 4 sequences fit and match the workspace path."""
    import paper_2608_20375_amd as G
    w = S.workload(0, batch=128, L=64, V=1000, K=64, n_max=64, fixed_budget=64, emb_dim=16,
                   rank=8)
    sc = WL.scorer_inputs(w, "literal")
    ctx = WL.gpu_context(w, sc, None, torch)
    big = _inputs(w, 0, 128)
    with pytest.raises(G.GraftError) as e:
        _build(ctx, big, True)
    assert e.value.status == 2
    assert "static" in str(e.value)
    small = _inputs(w, 0, 4)
    _same(_build(ctx, small, True), _build(ctx, small, False))
    assert ctx.device_status() == 0
    ctx.close()
