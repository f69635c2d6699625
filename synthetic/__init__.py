"""Seeded synthetic workloads for GRAFT's per-round draft-tree construction.

This module only draws inputs.  It holds none of the method's arithmetic (no
softmax, top-K, edge scoring, budget choice, selection or acceptance): both the
CPU oracle and the HIP library receive exactly the arrays produced here.

Workloads (shapes from the five benchmark configurations of the hot path):

  id  batch  L   V       K   N_max  budget                         scorer d/rank
  0   1      8   32000   4   32     fixed 32                       64/16
  1   1      16  151936  8   64     fixed 64                       64/16
  2   16     16  151936  8   256    SABA {16,32,64,128,256}        64/16
  3   64     16  128256  16  512    SABA 32..512 step 16           128/32
  4   128    32  151936  32  1024   SABA 32..1024 step 16          128/32

Drafter logits (one row per future position): z ~ N(0,1) per entry, divided by
a per-row temperature T ~ U(0.5, 1.5) in workloads 3 and 4, then n_boost
distinct uniformly drawn token ids get +6 * r**-1.2 for rank r = 1..n_boost
(n_boost = L), rounded to bf16 with round-to-nearest-even.  The vocabulary
sizes are those of the Qwen3 family (151936) and a 128256-entry vocabulary.

Every random stream is keyed by (workload seed, round, sequence, attempt,
stream id) through numpy's SeedSequence, so one sequence can be re-drawn
(attempt + 1) without touching the others.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "workload", "bf16_from_f32", "f32_from_bf16",
    "gen_sequence_logits", "gen_sequence", "put_sequence", "gen_round", "gen_scorer", "saba_params",
    "hist_ring_init", "node_targets", "splitmix64", "NODE_TARGET_P_NUM", "gen_hidden",
    "gen_sequence_hidden", "gen_traces", "gen_replay",
]

HIST_WINDOW = 4


@dataclass(frozen=True)
class Workload:
    wid: int
    batch: int
    L: int
    V: int
    K: int
    n_max: int
    budget_mode: str              # "fixed" or "saba"
    fixed_budget: int = 0
    grid: tuple = ()
    c1: float = 0.0
    c2: float = 0.0
    emb_dim: int = 64
    rank: int = 16
    temperature: bool = False
    targets: str = "depth"        # "depth" (second logit tensor) or "node" (counter hash)
    rounds: int = 1
    phi: tuple = (0.0, 0.0, 0.0, 0.0)
    seed: int = 0
    extra: dict = field(default_factory=dict)

    @property
    def n_boost(self) -> int:
        return self.L


WORKLOADS = {
    0: Workload(0, 1, 8, 32000, 4, 32, "fixed", fixed_budget=32, emb_dim=64, rank=16,
                seed=1000),
    1: Workload(1, 1, 16, 151936, 8, 64, "fixed", fixed_budget=64, emb_dim=64, rank=16,
                seed=1001),
    2: Workload(2, 16, 16, 151936, 8, 256, "saba", grid=(16, 32, 64, 128, 256),
                c1=1.0 / 128, c2=0.0, emb_dim=64, rank=16,
                phi=(6.0, 2000.0, 0.5, 14.0), seed=1002),
    3: Workload(3, 64, 16, 128256, 16, 512, "saba", grid=tuple(range(32, 513, 16)),
                c1=1.0 / 256, c2=2e-7, emb_dim=128, rank=32, temperature=True,
                phi=(6.0, 2000.0, 0.5, 18.0), seed=1003),
    4: Workload(4, 128, 32, 151936, 32, 1024, "saba", grid=tuple(range(32, 1025, 16)),
                c1=1.0 / 512, c2=2e-7, emb_dim=128, rank=32, temperature=True,
                targets="node", rounds=50, phi=(6.0, 2000.0, 0.5, 40.0), seed=1004),
}


def workload(wid: int, **overrides) -> Workload:
    """The named workload, optionally with fields replaced (smaller test shapes)."""
    w = WORKLOADS[wid]
    if overrides:
        d = dict(w.__dict__)
        d.update(overrides)
        w = Workload(**d)
    return w


def _rng(w: Workload, rnd: int, b: int, attempt: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([w.seed, w.wid, rnd, b, attempt, stream])


def bf16_from_f32(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round-to-nearest-even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def f32_from_bf16(h: np.ndarray) -> np.ndarray:
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _boost_weights(n: int) -> np.ndarray:
    r = np.arange(1, n + 1, dtype=np.float64)
    return (6.0 * r ** -1.2).astype(np.float32)


def gen_sequence_logits(w: Workload, rnd: int, b: int, attempt: int = 0):
    """Drafter logits of one sequence: (bf16 bits [L, V], boosted ids [L, n_boost])."""
    g = _rng(w, rnd, b, attempt, 0)
    z = g.standard_normal((w.L, w.V), dtype=np.float32)
    if w.temperature:
        t = g.uniform(0.5, 1.5, size=w.L).astype(np.float32)
        z /= t[:, None]
    boost_ids = np.stack([g.choice(w.V, size=w.n_boost, replace=False) for _ in range(w.L)])
    wts = _boost_weights(w.n_boost)
    rows = np.arange(w.L)[:, None]
    z[rows, boost_ids] += wts[None, :]
    return bf16_from_f32(z), boost_ids.astype(np.int64)


def _depth_targets(w: Workload, rnd: int, b: int, attempt: int, boost_ids: np.ndarray) -> np.ndarray:
    """Per-depth target tokens [L + 1] of one sequence.

    Entry j is the token the (synthetic) target model wants at draft depth j+1:
    the argmax of a second seeded bf16 logit row that boosts the same ids as
    the drafter row, with their ranks perturbed by adjacent swaps (p = 0.3).
    Entry L (the bonus after a fully accepted chain) is uniform over V.
    """
    g = _rng(w, rnd, b, attempt, 1)
    wts = _boost_weights(w.n_boost)
    z = g.standard_normal((w.L, w.V), dtype=np.float32)
    swaps = g.random((w.L, w.n_boost - 1)) < 0.3
    tgt = np.empty(w.L + 1, dtype=np.int32)
    for l in range(w.L):
        perm = np.arange(w.n_boost)
        for i in range(w.n_boost - 1):
            if swaps[l, i]:
                perm[i], perm[i + 1] = perm[i + 1], perm[i]
        z[l, boost_ids[l][perm]] += wts
    zb = f32_from_bf16(bf16_from_f32(z))
    tgt[:w.L] = np.argmax(zb, axis=1)          # first maximum: ties go to the lower id
    tgt[w.L] = int(g.integers(0, w.V))
    return tgt


def hist_ring_init(w: Workload, rnd: int = 0, attempts=None) -> np.ndarray:
    """Initial acceptance-history window [batch, HIST_WINDOW]: the previous
    accepted length a ~ U{0..16} of each sequence, repeated over the window so
    that hist (the window mean) equals it."""
    out = np.empty((w.batch, HIST_WINDOW), dtype=np.int32)
    for b in range(w.batch):
        a = 0 if attempts is None else int(attempts[b])
        out[b] = _rng(w, rnd, b, a, 2).integers(0, 17)
    return out


def gen_sequence(w: Workload, rnd: int, b: int, attempt: int = 0,
                 with_targets: bool = True) -> dict:
    """The per-round inputs of sequence b alone (draw `attempt`): logits [L, V]
    bf16 bits, boosted ids, root token, prefix length, the initial history
    window and, with per-depth targets, target_depth [L + 1]."""
    logits, boost = gen_sequence_logits(w, rnd, b, attempt)
    g = _rng(w, rnd, b, attempt, 3)
    root = int(g.integers(0, w.V))
    prefix = int(g.integers(64, 4097))
    out = dict(logits=logits, boost_ids=boost, root_token=root, prefix_len=prefix,
               hist_ring=_rng(w, rnd, b, attempt, 2).integers(0, 17))
    if with_targets and w.targets == "depth":
        out["target_depth"] = _depth_targets(w, rnd, b, attempt, boost)
    return out


def gen_round(w: Workload, rnd: int = 0, attempts=None, with_targets: bool = True,
              seqs=None) -> dict:
    """All per-round inputs for the batch (numpy, host memory).

    attempts[b] selects the re-draw index of sequence b (default 0).  seqs, if
    given, restricts generation to those sequence indices (others left zero);
    useful when only a sample of a large batch is compared against the oracle.
    """
    B = w.batch
    attempts = np.zeros(B, dtype=np.int64) if attempts is None else np.asarray(attempts)
    seqs = range(B) if seqs is None else seqs
    logits = np.zeros((B, w.L, w.V), dtype=np.uint16)
    boost = np.zeros((B, w.L, w.n_boost), dtype=np.int64)
    root = np.zeros(B, dtype=np.int32)
    prefix = np.zeros(B, dtype=np.int32)
    tdepth = np.zeros((B, w.L + 1), dtype=np.int32)
    ring = hist_ring_init(w, rnd, attempts)

    def one(b):
        one = gen_sequence(w, rnd, b, int(attempts[b]), with_targets)
        put_sequence(dict(logits=logits, boost_ids=boost, root_token=root, prefix_len=prefix,
                          target_depth=tdepth), b, one)

    seqs = list(seqs)
    if len(seqs) > 1 and w.L * w.V * len(seqs) > (1 << 22):
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(min(8, len(seqs))) as ex:
            list(ex.map(one, seqs))
    else:
        for b in seqs:
            one(b)
    hist = ring.astype(np.float64).mean(axis=1).astype(np.float32)
    out = dict(logits=logits, boost_ids=boost, root_token=root, prefix_len=prefix,
               base_pos=(prefix - 1).astype(np.int32), hist=hist, hist_ring=ring,
               attempts=attempts)
    if w.budget_mode == "fixed":
        out["fixed_budget"] = np.full(B, w.fixed_budget, dtype=np.int32)
    if w.targets == "depth":
        out["target_depth"] = tdepth
    return out


def put_sequence(batch: dict, b: int, one: dict) -> None:
    """Writes sequence b's draw (from gen_sequence) into the batch arrays of a
    gen_round result; the derived base position, history window and hist are
    refreshed when the batch holds them."""
    for k in ("logits", "boost_ids", "target_depth"):
        if k in one and k in batch:
            batch[k][b] = one[k]
    batch["root_token"][b] = one["root_token"]
    batch["prefix_len"][b] = one["prefix_len"]
    if "base_pos" in batch:
        batch["base_pos"][b] = one["prefix_len"] - 1
    if "hist_ring" in batch:
        batch["hist_ring"][b] = one["hist_ring"]
        batch["hist"][b] = np.float32(np.float64(one["hist_ring"]))


def gen_sequence_hidden(w: Workload, rnd: int, b: int, hidden_dim: int = 4096,
                        attempt: int = 0) -> np.ndarray:
    """Drafter hidden states of sequence b alone: [L, H] bf16 bits (see gen_hidden)."""
    L, H = w.L, int(hidden_dim)
    ramp = 0.5 + 2.5 * np.arange(L, dtype=np.float32) / max(L - 1, 1)
    g = _rng(w, rnd, b, int(attempt), 4)
    c = g.standard_normal(H, dtype=np.float32)
    n = g.standard_normal((L, H), dtype=np.float32)
    s_b = np.float32(g.uniform(0.3, 1.5))
    return bf16_from_f32((s_b * ramp)[:, None] * c[None, :] + n)


def gen_hidden(w: Workload, rnd: int = 0, hidden_dim: int = 4096, attempts=None,
               seqs=None) -> np.ndarray:
    """Drafter hidden states [batch, L, H] as bf16 bits, one per drafted position.

    h_d = a_d c + n_d with a shared direction c ~ N(0, I_H) and independent
    n_d ~ N(0, I_H): the share a_d = s (0.5 + 2.5 d / (L - 1)) of the common
    direction grows with the depth d = 0..L-1, so adjacent states grow more
    alike at later positions (the trend the degeneration signal measures);
    s ~ U(0.3, 1.5) per sequence spreads the signal over the batch.
    """
    B, L, H = w.batch, w.L, int(hidden_dim)
    attempts = np.zeros(B, dtype=np.int64) if attempts is None else np.asarray(attempts)
    seqs = range(B) if seqs is None else seqs
    out = np.zeros((B, L, H), dtype=np.uint16)
    for b in seqs:
        out[b] = gen_sequence_hidden(w, rnd, b, H, int(attempts[b]))
    return out


def gen_scorer(w: Workload, mode: str = "literal") -> dict:
    """Edge-scorer parameters.

    literal: the benchmark stand-in score log q(c) + e_p^T W e_c with W = U V^T,
      U, V in R^{d x rank} ~ N(0, 0.05^2), embeddings E in R^{V x d} ~ N(0, 0.1^2).
      Expressed as the bi-tower with g_p = U, g_c = V, scale = sqrt(m), no depth
      embedding, beta = 1 and no centering.
    paper: the same projections with a depth embedding u ~ N(0, 0.05^2) [L, m],
      scale 1.5, beta = 0.2 and centering on.
    """
    g = np.random.default_rng([w.seed, w.wid, 77])
    emb = (g.standard_normal((w.V, w.emb_dim), dtype=np.float32) * np.float32(0.1))
    U = (g.standard_normal((w.emb_dim, w.rank), dtype=np.float32) * np.float32(0.05))
    Vm = (g.standard_normal((w.emb_dim, w.rank), dtype=np.float32) * np.float32(0.05))
    u = (g.standard_normal((w.L, w.rank), dtype=np.float32) * np.float32(0.05))
    if mode == "literal":
        return dict(emb=emb, g_parent=U, g_child=Vm, depth_emb=None,
                    scale=float(np.float32(math.sqrt(w.rank))), beta=1.0, center=0)
    if mode == "paper":
        return dict(emb=emb, g_parent=U, g_child=Vm, depth_emb=u,
                    scale=1.5, beta=0.2, center=1)
    raise ValueError(mode)


def saba_params(w: Workload) -> dict:
    """SABA constants: utility (1 - exp(-B/tau)) / (c0 + c1 B + c2 B prefix),
    tau = max(phi . [1, conf, ent, hist], tau_min)."""
    return dict(grid=np.asarray(w.grid, dtype=np.int32), phi=np.asarray(w.phi, dtype=np.float32),
                tau_min=1.0, c0=1.0, c1=float(w.c1), c2=float(w.c2))


# ---------------------------------------------------------------------------
# Synthetic verifier for per-node targets (workload 4).
#
# The target model's greedy token after a draft node is replaced by a
# counter-based draw keyed on the node's identity (sequence, depth, parent
# token, token).  splitmix64 is Steele, Lea and Flood's published mixer
# ("Fast splittable pseudorandom number generators", OOPSLA 2014).  With
# probability 0.8 (an integer threshold on 24 hash bits) the target is the
# drafter's candidate of geometric(1/2) rank at the next depth; otherwise, and
# always at depth L, it is a hash of the identity modulo V.
# ---------------------------------------------------------------------------

_M64 = (1 << 64) - 1
NODE_TARGET_P_NUM = 13421773      # round(0.8 * 2**24)


def splitmix64(x):
    x = np.asarray(x, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = x + np.uint64(0x9E3779B97F4A7C15)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


def node_targets(seed: int, b, depth, parent_tok, tok, topk_ids_seq, V: int, L: int, K: int):
    """Target token of each node (vectorised over nodes of one sequence).

    depth: 0 for the root, 1..L for draft nodes.  parent_tok is -1 for the root
    and for depth-1 nodes' parent use the root token.  topk_ids_seq [L, K] holds
    the drafter candidates (rank order) of this sequence.
    """
    depth = np.asarray(depth, dtype=np.int64)
    enc = lambda t: (np.asarray(t, dtype=np.int64) + 1).astype(np.uint64)
    h = splitmix64(np.uint64(seed))
    h = splitmix64(h ^ np.uint64(b))
    h = splitmix64(h ^ depth.astype(np.uint64))
    h = splitmix64(h ^ enc(parent_tok))
    h = splitmix64(h ^ enc(tok))
    pick = (splitmix64(h ^ np.uint64(1)) >> np.uint64(40)) < np.uint64(NODE_TARGET_P_NUM)
    h2 = splitmix64(h ^ np.uint64(2))
    # count trailing zeros of h2 (64 when zero), capped at K-1
    r = np.zeros(h2.shape, dtype=np.int64)
    x = h2.copy()
    alive = np.ones(h2.shape, dtype=bool)
    for i in range(min(K - 1, 64)):
        bit = (x & np.uint64(1)) == np.uint64(0)
        alive &= bit
        r += alive
        x = x >> np.uint64(1)
    r = np.minimum(r, K - 1)
    h3 = splitmix64(h ^ np.uint64(3))
    hashed = (h3 % np.uint64(V)).astype(np.int64)
    topk = np.asarray(topk_ids_seq)
    nd = np.minimum(depth, L - 1)
    from_cand = topk[nd, r]
    use = pick & (depth < L)
    return np.where(use, from_cand, hashed).astype(np.int32)


def gen_traces(w: Workload, n_groups: int, n_pairs: int, step: int = 0) -> dict:
    """A batch of synthetic target-model traces for TDES training, shaped like
    the workload's rounds (its vocabulary, L and K).

    groups: parent tokens Zipf(1.1)-distributed over a fixed random permutation
      of the vocabulary; depth d in 1..L with P(d) proportional to 0.8^(d-1);
      K distinct children (Zipf draws, topped up uniformly); logq strictly
      descending, logq_k = -0.2 - 0.7 * (E_1 + ... + E_k), E_i ~ Exp(1);
      target logits z = 2 logq + N(0, 1); target token = the child with the
      largest z with probability 0.8, else a token outside the children.
    pairs: v+ = (parent, target, d) of a group whose target is a child; v- keeps
      the child under a uniformly drawn wrong parent, or (with probability 0.5)
      a competing child under the right parent.
    Integer arrays are int32, real ones float32.
    """
    g = np.random.default_rng([w.seed, w.wid, 91, step, n_groups, n_pairs])
    V, L, K = w.V, w.L, w.K
    perm = np.random.default_rng([w.seed, w.wid, 92]).permutation(V)

    def zipf_tokens(n):
        r = g.zipf(1.1, size=n) - 1
        r = np.where(r < V, r, g.integers(0, V, size=n))
        return perm[r]

    G = n_groups
    parent = zipf_tokens(G).astype(np.int32)
    pd = 0.8 ** np.arange(L)
    depth = (g.choice(L, size=G, p=pd / pd.sum()) + 1).astype(np.int32)
    child = np.empty((G, K), np.int32)
    for i in range(G):
        c = np.unique(zipf_tokens(2 * K))
        g.shuffle(c)
        c = list(c[:K])
        seen = set(int(x) for x in c)
        while len(c) < K:
            t = int(g.integers(0, V))
            if t not in seen:
                seen.add(t)
                c.append(t)
        child[i] = c
    logq = (-0.2 - 0.7 * np.cumsum(g.exponential(1.0, size=(G, K)), axis=1)).astype(np.float32)
    z = (2.0 * logq + g.standard_normal((G, K))).astype(np.float32)
    hit = g.random(G) < 0.8
    target = np.empty(G, np.int32)
    for i in range(G):
        if hit[i]:
            target[i] = child[i, int(np.argmax(z[i]))]
        else:
            t = int(g.integers(0, V))
            while t in set(child[i].tolist()):
                t = int(g.integers(0, V))
            target[i] = t
    pairs = np.empty((n_pairs, 6), np.int32)
    pos = np.flatnonzero(hit) if hit.any() else np.arange(max(G, 1))
    for i in range(n_pairs):
        if G == 0:
            p, c, q = (int(x) for x in g.integers(0, V, size=3))
            pairs[i] = (p, c, 1, q, c, 1)
            continue
        k = int(pos[int(g.integers(0, len(pos)))])
        p, c, d = int(parent[k]), int(target[k]), int(depth[k])
        if g.random() < 0.5 and K > 1:
            alt = [int(x) for x in child[k] if int(x) != c]
            pairs[i] = (p, c, d, p, alt[int(g.integers(0, len(alt)))], d)
        else:
            q = int(g.integers(0, V))
            while q == p:
                q = int(g.integers(0, V))
            pairs[i] = (p, c, d, q, c, d)
    return dict(parent=parent, depth=depth, child=child, logq=logq, z=z, target=target,
                pairs=pairs)


def gen_replay(n_rounds: int, grid=tuple(range(32, 513, 16)), phi=(6.0, 40.0, 30.0, 12.0),
               c=(20.0, 0.05, 2e-5), tau_min=8.0, noise=0.0, seed=0) -> dict:
    """A synthetic same-prefix budget-replay log for fitting SABA: every round
    replayed with each budget of the grid.  States conf ~ U(0.2, 0.95),
    degen ~ U(0.6, 1.4), hist ~ U(1, 12); prefix ~ U{64..4096}; the round's
    scale A ~ U(2, 14); accepted length A (1 - exp(-B / tau)) (1 + noise N(0,1)),
    tau = max(phi . [1, s], tau_min); latency (c0 + c1 B + c2 B prefix)
    (1 + noise N(0,1)).  float32 / int32 arrays."""
    g = np.random.default_rng([9009, n_rounds, seed])
    T = n_rounds
    B = np.asarray(grid, np.float64)
    state = np.stack([g.uniform(0.2, 0.95, T), g.uniform(0.6, 1.4, T), g.uniform(1, 12, T)],
                     axis=1)
    prefix = g.integers(64, 4097, T)
    tau = np.maximum(phi[0] + state @ np.asarray(phi[1:], np.float64), tau_min)
    A = g.uniform(2, 14, T)
    acc = A[:, None] * (1.0 - np.exp(-B[None, :] / tau[:, None]))
    acc *= 1.0 + noise * g.standard_normal(acc.shape)
    lat = c[0] + c[1] * B[None, :] + c[2] * B[None, :] * prefix[:, None]
    lat = lat * (1.0 + noise * g.standard_normal(lat.shape))
    return dict(budgets=np.asarray(grid, np.int32), state=state.astype(np.float32),
                prefix=prefix.astype(np.int32), accepted=acc.astype(np.float32),
                latency=lat.astype(np.float32), tau_min=float(tau_min))
