"""Parity of the representation-degeneration signal (the SABA decoding state's
degen_t, from the drafter's hidden states) between the HIP path and the CPU
oracle, through the C ABI.

Bars: the adjacent cosines r_d and degen agree with the fp64 oracle within
1e-5 relative (absolute floor 1e-6); with hidden states, budgets, trees and
masks are bit-exact on audited sequences (every floating-point decision,
including the SABA utility gap, has a margin an fp32 path cannot cross).
"""
import os
import sys

import numpy as np
import pytest

import oracle
import synthetic as S

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import workload as WL  # noqa: E402
import test_parity_gpu as TP  # noqa: E402

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(*a):
    print(*a, flush=True)


def _degen_from(r):
    """degen from given cosines r_1..r_{L-1}, summed left to right in fp64."""
    r = [float(x) for x in r]
    if not r:
        return 0.0
    return sum(r) / len(r) + (r[-1] - r[0])


SHAPES = [
    # batch, L, H
    (3, 16, 4096),     # the drafter width the synthetic workloads use
    (2, 9, 8),         # one 16-byte vector per row
    (1, 2, 2056),      # a single pair; 257 vectors per row (ragged over the lanes)
    (2, 5, 24),
    (4, 7, 1000),      # runs of 4 pairs plus a run of 2
    (1, 33, 520),      # L > 32
]


@pytest.mark.parametrize("shape", SHAPES)
def test_adjacent_cosines_and_degen(shape):
    B, L, H = shape
    _say("hidden-state cosines", shape)
    w = S.workload(0, batch=B, L=L, V=3000, K=4, n_max=32, fixed_budget=8)
    inp = S.gen_round(w, with_targets=False)
    hid = S.gen_hidden(w, 0, H)
    if B > 1:
        hid[1, L // 2] = 0          # a zero state: both of its cosines are 0
    inp["hidden"] = hid
    sc = WL.scorer_inputs(w, "literal")
    ctx = WL.gpu_context(w, sc, None, torch)
    g = WL.gpu_round(ctx, w, inp, torch)
    for b in range(B):
        d, r = oracle.degen(hid[b])
        assert TP.close(g["adj_cos"][b, :L - 1], r).all(), b
        assert TP.close(g["saba_state"][b, 1], d), (b, g["saba_state"][b, 1], d)
        if B > 1 and b == 1:
            assert g["adj_cos"][b, L // 2] == 0.0
            if L // 2 >= 1:
                assert g["adj_cos"][b, L // 2 - 1] == 0.0
    ctx.close()


def test_one_position_has_no_pair():
    """L = 1: no adjacent pair, degen = 0, and the cosine buffer is untouched."""
    w = S.workload(0, batch=2, L=1, V=3000, K=4, n_max=32, fixed_budget=4)
    inp = S.gen_round(w, with_targets=False)
    inp["hidden"] = S.gen_hidden(w, 0, 64)
    sc = WL.scorer_inputs(w, "literal")
    ctx = WL.gpu_context(w, sc, None, torch)
    g = WL.gpu_round(ctx, w, inp, torch)
    assert (g["adj_cos"] == 0).all()
    assert (g["saba_state"][:, 1] == 0).all()
    assert oracle.degen(inp["hidden"][0])[0] == 0.0
    ctx.close()


@pytest.mark.parametrize("wid,H", [(2, 4096), (3, 2048)])
def test_round_parity_with_hidden_states(wid, H):
    """SABA on [1, conf, degen, hist]: budgets, trees and masks bit-exact.
    The weight of the state's second feature is raised to 40 so that degen
    (about 0.3 to 1.5 here) moves tau by tens of nodes."""
    w = S.workload(wid)
    _say("round parity with hidden states, workload", wid, "H", H)
    phi = list(w.phi)
    phi[2] = 40.0
    inp, sc, sp, results = WL.audited_round(w, 0, "literal", hidden_dim=H, phi=phi)
    assert len(results) == w.batch
    _say("  inputs ready; attempts", inp["attempts"][list(results)].tolist())
    ctx = WL.gpu_context(w, sc, sp, torch)
    g = WL.gpu_round(ctx, w, inp, torch)
    TP.end_to_end_check(w, g, inp, results)
    P = oracle.make_params(w.L, w.K, w.n_max, w.V, sc, sp)
    for b in range(w.batch):
        conf = sum(float(v) for v in g["row_maxprob"][b]) / w.L
        dg = _degen_from(g["adj_cos"][b, :w.L - 1])
        assert TP.close(g["saba_state"][b, 1], dg)
        bud, _, rel, _ = oracle.saba(P, conf, dg, float(inp["hist"][b]), int(inp["prefix_len"][b]))
        if rel > 1e-12:
            assert bud == g["budget"][b], (b, bud, g["budget"][b], rel)
    for b, r in results.items():
        assert TP.close(g["adj_cos"][b, :w.L - 1], r["adj_cos"]).all(), b
        assert TP.close(g["saba_state"][b, 1], r["degen"]), b
    TP.staged_check(w, g, sc, sp, inp, range(w.batch))
    assert ctx.device_status() == 0
    ctx.close()


def test_hidden_state_argument_errors():
    import paper_2608_20375_amd as G
    w = S.workload(0, batch=2, V=1000)
    sc = WL.scorer_inputs(w, "literal")
    ctx = WL.gpu_context(w, sc, None, torch)
    logits = torch.zeros(2, w.L, w.V, dtype=torch.int16, device="cuda")
    z = torch.zeros(2, dtype=torch.int32, device="cuda")
    fb = torch.full((2,), 4, dtype=torch.int32, device="cuda")
    for H in (12, 4):   # not a multiple of 8 / below 8
        hid = torch.zeros(2, w.L, H, dtype=torch.int16, device="cuda")
        with pytest.raises(G.GraftError) as e:
            ctx.build_tree(logits, z, z, fixed_budget=fb, hidden=hid)
        assert e.value.status == 1
    flat = torch.zeros(2 * w.L * 64 + 8, dtype=torch.int16, device="cuda")
    mis = flat[1:1 + 2 * w.L * 64].view(2, w.L, 64)
    with pytest.raises(G.GraftError):
        ctx.build_tree(logits, z, z, fixed_budget=fb, hidden=mis)
    ctx.close()
