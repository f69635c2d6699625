"""CPU oracle for GRAFT's per-round draft-tree construction -- TEST INFRASTRUCTURE.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this package.  The product path (paper_2608_20375_amd) never does: it runs the
HIP library or fails.

The arithmetic lives in oracle.c (plain C, fp64); this module compiles it with
gcc and marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes as C
import math
import os
import subprocess
import threading
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so (gcc, fp64, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
               "-fno-fast-math", "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


class Params(C.Structure):
    _fields_ = [
        ("L", C.c_int32), ("K", C.c_int32), ("n_max", C.c_int32), ("V", C.c_int64),
        ("emb", C.c_void_p), ("emb_dim", C.c_int32), ("g_parent", C.c_void_p),
        ("g_child", C.c_void_p), ("depth_emb", C.c_void_p), ("score_dim", C.c_int32),
        ("scale", C.c_double), ("beta", C.c_double), ("center", C.c_int32),
        ("use_saba", C.c_int32), ("grid", C.c_void_p), ("n_grid", C.c_int32),
        ("phi", C.c_double * 4), ("tau_min", C.c_double), ("c0", C.c_double),
        ("c1", C.c_double), ("c2", C.c_double),
    ]


class SeqIn(C.Structure):
    _fields_ = [("logits", C.c_void_p), ("root_token", C.c_int32), ("base_pos", C.c_int32),
                ("prefix_len", C.c_int32), ("fixed_budget", C.c_int32), ("hist", C.c_double),
                ("hidden", C.c_void_p), ("hidden_dim", C.c_int32)]


class SeqOut(C.Structure):
    _fields_ = [
        ("topk_ids", C.c_void_p), ("topk_logq", C.c_void_p), ("row_lse", C.c_void_p),
        ("row_maxprob", C.c_void_p), ("row_entropy", C.c_void_p), ("edge", C.c_void_p),
        ("conf", C.c_double), ("ent", C.c_double), ("tau", C.c_double),
        ("budget", C.c_int32), ("saba_relgap", C.c_double),
        ("n_nodes", C.c_int32), ("tokens", C.c_void_p), ("parents", C.c_void_p),
        ("pos_ids", C.c_void_p), ("depth", C.c_void_p), ("node_scores", C.c_void_p),
        ("mask", C.c_void_p), ("boundary_gap", C.c_double), ("min_pop_gap", C.c_double),
        ("degen", C.c_double), ("adj_cos", C.c_void_p),
    ]


def lib():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build(force=True)
            L = C.CDLL(_LIB)
            L.oracle_row_stats.argtypes = [C.c_void_p, C.c_int64, C.POINTER(C.c_double),
                                           C.POINTER(C.c_double), C.POINTER(C.c_double)]
            L.oracle_row_stats.restype = None
            L.oracle_topk.argtypes = [C.c_void_p, C.c_int64, C.c_int32, C.c_void_p, C.c_void_p]
            L.oracle_topk.restype = C.c_int
            L.oracle_edge_scores.argtypes = [C.POINTER(Params), C.c_void_p, C.c_void_p,
                                             C.c_int32, C.c_void_p, C.c_void_p]
            L.oracle_edge_scores.restype = C.c_int
            L.oracle_saba.argtypes = [C.POINTER(Params), C.c_double, C.c_double, C.c_double,
                                      C.c_int32, C.POINTER(C.c_double), C.POINTER(C.c_double),
                                      C.c_void_p]
            L.oracle_saba.restype = C.c_int32
            L.oracle_degen.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.c_void_p]
            L.oracle_degen.restype = C.c_double
            L.oracle_build_sequence.argtypes = [C.POINTER(Params), C.POINTER(SeqIn),
                                                C.POINTER(SeqOut)]
            L.oracle_build_sequence.restype = C.c_int
            L.oracle_select_staged.argtypes = [C.POINTER(Params), C.c_void_p, C.c_void_p,
                                               C.c_int32, C.c_int32, C.POINTER(SeqOut)]
            L.oracle_select_staged.restype = C.c_int
            L.oracle_accept.argtypes = [C.c_int32, C.c_void_p, C.c_void_p, C.c_int32, C.c_int32,
                                        C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
            L.oracle_accept.restype = C.c_int32
            L.oracle_mask_to_bias.argtypes = [C.c_int32, C.c_int32, C.c_void_p, C.c_int32,
                                              C.c_void_p]
            L.oracle_mask_to_bias.restype = None
            L.oracle_gather_rows.argtypes = [C.c_int32, C.c_void_p, C.c_void_p, C.c_int64,
                                             C.c_void_p, C.c_int64, C.c_int64]
            L.oracle_gather_rows.restype = C.c_int
            _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def _c(a, dt):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


# ---------------------------------------------------------------------------
# Single-step wrappers
# ---------------------------------------------------------------------------

def row_stats(row: np.ndarray):
    row = _c(row, np.uint16)
    a, b, c = C.c_double(), C.c_double(), C.c_double()
    lib().oracle_row_stats(_p(row), row.size, C.byref(a), C.byref(b), C.byref(c))
    return a.value, b.value, c.value


def topk(row: np.ndarray, K: int):
    row = _c(row, np.uint16)
    ids = np.empty(K, np.int32)
    x = np.empty(K, np.float64)
    rc = lib().oracle_topk(_p(row), row.size, K, _p(ids), _p(x))
    if rc:
        raise ValueError("oracle_topk failed (%d)" % rc)
    return ids, x


class _Keep:
    """Keeps the arrays referenced by a Params struct alive."""

    def __init__(self):
        self.refs = []

    def __call__(self, a):
        self.refs.append(a)
        return a


def make_params(L, K, n_max, V, scorer: dict, saba: dict | None = None):
    keep = _Keep()
    P = Params()
    P.L, P.K, P.n_max, P.V = L, K, n_max, V
    P.emb = _p(keep(_c(scorer["emb"], np.float32)))
    P.emb_dim = scorer["emb"].shape[1]
    P.g_parent = _p(keep(_c(scorer["g_parent"], np.float32)))
    P.g_child = _p(keep(_c(scorer["g_child"], np.float32)))
    de = scorer.get("depth_emb")
    P.depth_emb = _p(keep(_c(de, np.float32))) if de is not None else None
    P.score_dim = scorer["g_parent"].shape[1]
    P.scale, P.beta, P.center = float(scorer["scale"]), float(scorer["beta"]), int(scorer["center"])
    if saba is not None:
        P.use_saba = 1
        grid = keep(_c(saba["grid"], np.int32))
        P.grid, P.n_grid = _p(grid), grid.size
        for i in range(4):
            P.phi[i] = float(saba["phi"][i])
        P.tau_min, P.c0, P.c1, P.c2 = (float(saba["tau_min"]), float(saba["c0"]),
                                       float(saba["c1"]), float(saba["c2"]))
    else:
        P.use_saba = 0
    P._keep = keep
    return P


def edge_scores(P: Params, cand: np.ndarray, logq: np.ndarray, root: int):
    L, K = P.L, P.K
    cand = _c(cand, np.int32)
    logq = _c(logq, np.float64)
    edge = np.empty((L, K, K), np.float64)
    f = np.empty((L, K, K), np.float64)
    rc = lib().oracle_edge_scores(C.byref(P), _p(cand), _p(logq), int(root), _p(edge), _p(f))
    if rc:
        raise RuntimeError("oracle_edge_scores failed (%d)" % rc)
    return edge, f


def saba(P: Params, conf: float, feat: float, hist: float, prefix: int):
    """feat: the state's second feature (degen, or the mean entropy)."""
    tau, rel = C.c_double(), C.c_double()
    util = np.empty(P.n_grid, np.float64)
    b = lib().oracle_saba(C.byref(P), conf, feat, hist, int(prefix), C.byref(tau), C.byref(rel),
                          _p(util))
    return int(b), tau.value, rel.value, util


def degen(hidden: np.ndarray):
    """O5a on hidden states [L, H] bf16 bits: (degen, r[L-1])."""
    hidden = _c(hidden, np.uint16)
    L, H = hidden.shape
    r = np.empty(max(L - 1, 1), np.float64)
    d = lib().oracle_degen(_p(hidden), int(L), int(H), _p(r))
    return float(d), r[:max(L - 1, 0)].copy()


def _alloc_out(L, K, n_max):
    words = (n_max + 63) // 64
    a = dict(adj_cos=np.empty(max(L - 1, 1)),
             topk_ids=np.empty((L, K), np.int32), topk_logq=np.empty((L, K), np.float64),
             row_lse=np.empty(L), row_maxprob=np.empty(L), row_entropy=np.empty(L),
             edge=np.empty((L, K, K)), tokens=np.empty(n_max, np.int32),
             parents=np.empty(n_max, np.int32), pos_ids=np.empty(n_max, np.int32),
             depth=np.empty(n_max, np.int32), node_scores=np.empty(n_max),
             mask=np.empty((n_max, words), np.uint64))
    o = SeqOut()
    for k, v in a.items():
        setattr(o, k, v.ctypes.data)
    return o, a


def _collect(o: SeqOut, a: dict) -> dict:
    a = dict(a)
    for k in ("conf", "ent", "tau", "budget", "saba_relgap", "n_nodes", "boundary_gap",
              "min_pop_gap", "degen"):
        a[k] = getattr(o, k)
    a["adj_cos"] = a["adj_cos"][:max(len(a["row_lse"]) - 1, 0)]
    return a


def build_sequence(P: Params, logits: np.ndarray, root: int, base_pos: int, prefix: int = 0,
                   fixed_budget: int = 0, hist: float = 0.0, hidden=None) -> dict:
    """O2..O7 for one sequence; logits [L, V] bf16 bits, hidden [L, H] bf16 bits or None."""
    logits = _c(logits, np.uint16)
    assert logits.shape == (P.L, P.V)
    hid = _c(hidden, np.uint16)
    if hid is not None:
        assert hid.ndim == 2 and hid.shape[0] == P.L
    si = SeqIn(_p(logits), int(root), int(base_pos), int(prefix), int(fixed_budget), float(hist),
               _p(hid), 0 if hid is None else int(hid.shape[1]))
    o, a = _alloc_out(P.L, P.K, P.n_max)
    rc = lib().oracle_build_sequence(C.byref(P), C.byref(si), C.byref(o))
    if rc:
        raise RuntimeError("oracle_build_sequence failed (%d)" % rc)
    return _collect(o, a)


def select_staged(P: Params, cand: np.ndarray, edge32: np.ndarray, budget: int,
                  base_pos: int) -> dict:
    """O6..O7 on given fp32 edge scores [L, K, K] and candidates [L, K]."""
    cand = _c(cand, np.int32)
    edge32 = _c(edge32, np.float32)
    o, a = _alloc_out(P.L, P.K, P.n_max)
    rc = lib().oracle_select_staged(C.byref(P), _p(cand), _p(edge32), int(budget), int(base_pos),
                                    C.byref(o))
    if rc:
        raise RuntimeError("oracle_select_staged failed (%d)" % rc)
    out = _collect(o, a)
    out["topk_ids"] = cand
    return out


def accept(n_nodes: int, tokens, parents, L: int, target_root: int = -1, target_node=None,
           target_depth=None):
    tokens = _c(tokens, np.int32)
    parents = _c(parents, np.int32)
    tn = _c(target_node, np.int32)
    td = _c(target_depth, np.int32)
    acc = np.empty(max(L, 1), np.int32)
    bonus = np.empty(1, np.int32)
    a = lib().oracle_accept(int(n_nodes), _p(tokens), _p(parents), int(L), int(target_root),
                            _p(tn), _p(td), _p(acc), _p(bonus))
    return int(a), acc[:L].copy(), int(bonus[0])


def mask_to_bias(n_nodes: int, mask: np.ndarray) -> np.ndarray:
    """V1: [n_max, n_max] additive bias (0 / -inf, fp64) from mask [n_max, words]."""
    mask = _c(mask, np.uint64)
    n_max, words = mask.shape
    out = np.empty((n_max, n_max), np.float64)
    lib().oracle_mask_to_bias(int(n_nodes), int(n_max), _p(mask), int(words), _p(out))
    return out


def gather_rows(acc_len: int, acc_nodes, src: np.ndarray, dst: np.ndarray) -> np.ndarray:
    """V2: dst[i] = src[acc_nodes[i]] for i < acc_len (rows of bytes); dst is
    modified in place and returned.  src may be dst."""
    nodes = _c(acc_nodes, np.int32)
    assert src.flags.c_contiguous and dst.flags.c_contiguous and src.dtype == dst.dtype
    row_bytes = src.strides[0]
    assert dst.strides[0] == row_bytes
    if acc_len > 0:
        assert nodes.max(initial=-1) < src.shape[0] and acc_len <= dst.shape[0]
    rc = lib().oracle_gather_rows(int(acc_len), _p(nodes), src.ctypes.data, row_bytes,
                                  dst.ctypes.data, row_bytes, row_bytes)
    if rc:
        raise MemoryError("oracle_gather_rows")
    return dst


# ---------------------------------------------------------------------------
# Batch helpers
# ---------------------------------------------------------------------------

def build_round(w, inputs: dict, scorer: dict, saba_p: dict | None, seqs=None,
                threads: int = 1) -> list:
    """Run build_sequence over the batch (or the listed sequences)."""
    P = make_params(w.L, w.K, w.n_max, w.V, scorer, saba_p if w.budget_mode == "saba" else None)
    seqs = list(range(w.batch)) if seqs is None else list(seqs)
    fb = inputs.get("fixed_budget")

    hid = inputs.get("hidden")

    def one(b):
        return build_sequence(P, inputs["logits"][b], inputs["root_token"][b],
                              inputs["base_pos"][b], inputs["prefix_len"][b],
                              0 if fb is None else fb[b], float(inputs["hist"][b]),
                              None if hid is None else hid[b])

    if threads > 1:
        with ThreadPoolExecutor(threads) as ex:
            res = list(ex.map(one, seqs))
    else:
        res = [one(b) for b in seqs]
    return res


def gap_threshold(L: int) -> float:
    """Absolute path-score margin that covers fp32 edge-score rounding plus the
    log-sum-exp error of an fp32 logits pass: L * 2**-17."""
    return L * 2.0 ** -17


SABA_REL_GAP = 1e-4


def sequence_ok(res: dict, L: int) -> bool:
    """Whether every floating-point decision of this sequence has a margin wide
    enough that an fp32 implementation must reach the same tree."""
    tau = gap_threshold(L)
    gap = res["boundary_gap"]
    edge = res.get("edge")
    if edge is not None and (np.asarray(edge) > 0).any():
        # a positive edge score lets a child outrank its parent: every pop
        # decision matters, not only the boundary one
        gap = min(gap, res["min_pop_gap"])
    if not (gap >= tau or math.isinf(gap)):
        return False
    if res["saba_relgap"] < SABA_REL_GAP:
        return False
    return True
