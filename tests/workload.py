"""Test-side helpers: audited synthetic rounds and oracle/GPU runners.

Audit: a sequence's inputs are re-drawn (attempt + 1) until every
floating-point decision the oracle takes for it has a margin that an fp32
implementation cannot cross (oracle.sequence_ok).  Only the oracle is consulted,
never the HIP path.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle
import synthetic as S

MAX_ATTEMPTS = 24


def scorer_inputs(w, mode):
    sc = S.gen_scorer(w, mode)
    # the ABI carries scale and beta as fp32; hand the oracle the same values
    sc["scale"] = float(np.float32(sc["scale"]))
    sc["beta"] = float(np.float32(sc["beta"]))
    return sc


def saba_inputs(w):
    if w.budget_mode != "saba":
        return None
    sp = S.saba_params(w)
    for k in ("tau_min", "c0", "c1", "c2"):
        sp[k] = float(np.float32(sp[k]))
    sp["phi"] = np.asarray(sp["phi"], np.float32)
    return sp


def oracle_threads() -> int:
    """Worker threads for the oracle: the cores this process may use, at most 16
    (the host share of one GPU).  The oracle's C calls release the GIL."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def audited_round(w, rnd=0, mode="literal", seqs=None, with_targets=True, hidden_dim=None,
                  phi=None, hist=None, transform=None, scorer=None):
    """Inputs for the whole batch; sequences in `seqs` (default: all) are
    audited with the oracle and re-drawn until their decisions are robust.
    With hidden_dim, drafter hidden states [batch, L, hidden_dim] are drawn too
    and the SABA state uses their degeneration signal.  phi overrides the SABA
    state weights; hist (fp64 [batch]) overrides the history feature the
    oracle sees (a chained round reads it from the device ring); transform(b,
    logits) may rewrite a draw's logits [L, V] in place before the audit;
    scorer replaces the workload's scorer of `mode`.
    Sequences are drawn and audited in parallel (one sequence per task).
    Returns (inputs, scorer, saba, {b: oracle result})."""
    sc = scorer_inputs(w, mode) if scorer is None else scorer
    sp = saba_inputs(w)
    if phi is not None and sp is not None:
        sp["phi"] = np.asarray(phi, np.float32)
    audit = set(range(w.batch)) if seqs is None else set(seqs)
    attempts = np.zeros(w.batch, np.int64)
    inp = S.gen_round(w, rnd, attempts, with_targets=with_targets, seqs=[])
    if hidden_dim:
        inp["hidden"] = np.zeros((w.batch, w.L, hidden_dim), np.uint16)
    P = oracle.make_params(w.L, w.K, w.n_max, w.V, sc, sp)
    fixed = w.fixed_budget if w.budget_mode == "fixed" else 0

    def one(b):
        for a in range(MAX_ATTEMPTS if b in audit else 1):
            d = S.gen_sequence(w, rnd, b, a, with_targets)
            if transform is not None:
                transform(b, d["logits"])
            h = S.gen_sequence_hidden(w, rnd, b, hidden_dim, a) if hidden_dim else None
            if b not in audit:
                return a, d, h, None
            hv = float(np.float32(d["hist_ring"])) if hist is None else float(hist[b])
            r = oracle.build_sequence(P, d["logits"], d["root_token"], d["prefix_len"] - 1,
                                      d["prefix_len"], fixed, hv, h)
            if oracle.sequence_ok(r, w.L):
                return a, d, h, r
        raise RuntimeError("no robust draw for sequence %d" % b)

    with ThreadPoolExecutor(oracle_threads()) as ex:
        done = list(ex.map(one, range(w.batch)))
    results = {}
    for b, (a, d, h, r) in enumerate(done):
        attempts[b] = a
        S.put_sequence(inp, b, d)
        if hidden_dim:
            inp["hidden"][b] = h
        if r is not None:
            results[b] = r
    if hist is not None:
        inp["hist"] = np.asarray(hist, np.float32)
    inp["attempts"] = attempts
    return inp, sc, sp, results


def gpu_context(w, sc, sp, torch, dev="cuda"):
    import paper_2608_20375_amd as G
    ctx = G.Context(w.batch, w.L, w.V, w.K, w.n_max, S.HIST_WINDOW)
    T = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    ctx.set_scorer(T(sc["emb"]), T(sc["g_parent"]), T(sc["g_child"]), T(sc["depth_emb"]),
                   sc["scale"], sc["beta"], sc["center"])
    if sp is not None:
        ctx.set_saba(list(sp["grid"]), list(sp["phi"]), sp["tau_min"], sp["c0"], sp["c1"],
                     sp["c2"])
    return ctx


def gpu_round(ctx, w, inp, torch, dev="cuda", use_ring=False, edges=True):
    """Upload a round, build trees on the GPU, return numpy copies."""
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    logits = T(inp["logits"].view(np.int16))
    out = ctx.build_tree(logits, T(inp["root_token"]), T(inp["base_pos"]),
                         prefix_len=T(inp["prefix_len"]),
                         hist=None if use_ring else T(inp["hist"]),
                         fixed_budget=T(inp["fixed_budget"]) if "fixed_budget" in inp else None,
                         hidden=T(inp["hidden"].view(np.int16)) if "hidden" in inp else None,
                         edges=edges, adj_cos="hidden" in inp)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.as_dict().items()}
    res["_out"] = out
    return res
