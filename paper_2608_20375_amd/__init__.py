"""Python binding of libgraft (include/graft.h): argument marshalling only.

Every step of GRAFT's per-round draft-tree construction runs in the HIP
kernels of libgraft.so; this module passes torch tensors' device pointers and
the current HIP stream through ctypes.  If the library is not built, importing
works but creating a Context raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

import torch

__all__ = ["Context", "TreeBuffers", "TdesTrainer", "TdesHyper", "saba_fit", "read_stream", "lib",
           "library_path", "GraftError", "EXPORTED_SYMBOLS"]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libgraft.so")
_lib = None

EXPORTED_SYMBOLS = (
    "graft_create", "graft_destroy", "graft_set_scorer", "graft_set_saba", "graft_set_history",
    "graft_get_history", "graft_set_fusion",
    "graft_build_tree", "graft_build_tree_static", "graft_accept", "graft_get_device_status",
    "graft_synth_node_targets", "graft_profile_begin", "graft_profile_end", "graft_status_string", "graft_last_error",
    "graft_mask_to_bias", "graft_commit_accepted", "graft_tdes_create", "graft_tdes_destroy",
    "graft_tdes_param_count", "graft_tdes_step", "graft_tdes_device_status", "graft_saba_fit",
    "graft_read_stream",
)

READ_STREAM_SINK_WORDS = 4096


class GraftError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        L = lib()
        super().__init__("%s: %s (%s)" % (where, L.graft_status_string(status).decode(),
                                          L.graft_last_error().decode()))


class Dims(C.Structure):
    _fields_ = [("max_batch", C.c_int32), ("num_pos", C.c_int32), ("vocab", C.c_int32),
                ("top_k", C.c_int32), ("max_nodes", C.c_int32), ("hist_window", C.c_int32)]


class ScorerDesc(C.Structure):
    _fields_ = [("emb", C.c_void_p), ("g_parent", C.c_void_p), ("g_child", C.c_void_p),
                ("depth_emb", C.c_void_p), ("emb_dim", C.c_int32), ("score_dim", C.c_int32),
                ("scale", C.c_float), ("beta", C.c_float), ("center", C.c_int32)]


class SabaDesc(C.Structure):
    _fields_ = [("budgets", C.c_void_p), ("n_budgets", C.c_int32), ("phi", C.c_float * 4),
                ("tau_min", C.c_float), ("c0", C.c_float), ("c1", C.c_float), ("c2", C.c_float)]


class RoundIn(C.Structure):
    _fields_ = [("batch", C.c_int32), ("logits", C.c_void_p), ("root_token", C.c_void_p),
                ("base_pos", C.c_void_p), ("prefix_len", C.c_void_p), ("hist", C.c_void_p),
                ("fixed_budget", C.c_void_p), ("hidden", C.c_void_p), ("hidden_dim", C.c_int32)]


class TreeOut(C.Structure):
    _fields_ = [("budget", C.c_void_p), ("n_nodes", C.c_void_p), ("tokens", C.c_void_p),
                ("parents", C.c_void_p), ("pos_ids", C.c_void_p), ("mask", C.c_void_p),
                ("topk_ids", C.c_void_p), ("topk_logq", C.c_void_p), ("row_lse", C.c_void_p),
                ("row_maxprob", C.c_void_p), ("row_entropy", C.c_void_p),
                ("edge_scores", C.c_void_p), ("node_scores", C.c_void_p),
                ("saba_state", C.c_void_p), ("adj_cos", C.c_void_p)]


class TdesDims(C.Structure):
    _fields_ = [("vocab", C.c_int32), ("emb_dim", C.c_int32), ("score_dim", C.c_int32),
                ("num_pos", C.c_int32), ("top_k", C.c_int32), ("max_groups", C.c_int32),
                ("max_pairs", C.c_int32)]


class TdesBatch(C.Structure):
    _fields_ = [("n_groups", C.c_int32), ("parent", C.c_void_p), ("depth", C.c_void_p),
                ("child", C.c_void_p), ("logq", C.c_void_p), ("z_target", C.c_void_p),
                ("target", C.c_void_p), ("n_pairs", C.c_int32), ("pairs", C.c_void_p)]


class TdesHyper(C.Structure):
    """Loss weights, margin, positive weight and AdamW settings; the defaults
    are the paper's training setup (lambda 1 / 1 / 0.25, lr 2e-3, weight decay
    1e-4) with the usual AdamW betas and eps, margin 1 and w1 = 1."""
    _fields_ = [(n, C.c_float) for n in ("lambda_kl", "lambda_pair", "lambda_bce", "gamma", "w1",
                                         "lr", "weight_decay", "beta1", "beta2", "eps")]

    def __init__(self, lambda_kl=1.0, lambda_pair=1.0, lambda_bce=0.25, gamma=1.0, w1=1.0,
                 lr=2e-3, weight_decay=1e-4, beta1=0.9, beta2=0.999, eps=1e-8):
        super().__init__(lambda_kl, lambda_pair, lambda_bce, gamma, w1, lr, weight_decay, beta1,
                         beta2, eps)


class SabaReplay(C.Structure):
    _fields_ = [("n_rounds", C.c_int32), ("n_budgets", C.c_int32), ("budgets", C.c_void_p),
                ("state", C.c_void_p), ("prefix", C.c_void_p), ("accepted", C.c_void_p),
                ("latency", C.c_void_p), ("tau_min", C.c_float)]


class Targets(C.Structure):
    _fields_ = [("target_root", C.c_void_p), ("target_node", C.c_void_p),
                ("target_depth", C.c_void_p)]


def library_path() -> str:
    return _LIB_PATH


def lib():
    """The loaded libgraft.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError("libgraft.so is not built (python -m paper_2608_20375_amd.build); "
                               "this package has no non-HIP path")
        L = C.CDLL(_LIB_PATH)
        vp, i32 = C.c_void_p, C.c_int32
        L.graft_create.argtypes = [C.POINTER(Dims), C.POINTER(vp)]
        L.graft_destroy.argtypes = [vp]
        L.graft_destroy.restype = None
        L.graft_set_scorer.argtypes = [vp, C.POINTER(ScorerDesc), vp]
        L.graft_set_saba.argtypes = [vp, C.POINTER(SabaDesc)]
        L.graft_set_history.argtypes = [vp, i32, vp, vp]
        L.graft_get_history.argtypes = [vp, i32, vp, vp, vp]
        L.graft_set_fusion.argtypes = [vp, i32, C.POINTER(C.c_int32)]
        L.graft_build_tree.argtypes = [vp, C.POINTER(RoundIn), C.POINTER(TreeOut), vp]
        L.graft_build_tree_static.argtypes = [vp, C.POINTER(RoundIn), C.POINTER(TreeOut), vp]
        L.graft_accept.argtypes = [vp, i32, vp, vp, vp, C.POINTER(Targets), vp, vp, vp, i32, vp]
        L.graft_get_device_status.argtypes = [vp, vp]
        L.graft_synth_node_targets.argtypes = [vp, i32, C.c_uint64, vp, vp, vp, vp, vp, vp, vp, vp]
        i64 = C.c_int64
        L.graft_mask_to_bias.argtypes = [vp, i32, vp, vp, vp, i32, i64, i64, vp]
        L.graft_commit_accepted.argtypes = [vp, i32, vp, vp, vp, vp, i64, i32, i64, i64, i64,
                                            i64, i64, i64, vp]
        L.graft_profile_begin.argtypes = [vp, i32]
        L.graft_profile_end.argtypes = [vp, C.POINTER(C.c_double), C.POINTER(C.c_int32)]
        L.graft_tdes_create.argtypes = [C.POINTER(TdesDims), C.POINTER(vp)]
        L.graft_tdes_destroy.argtypes = [vp]
        L.graft_tdes_destroy.restype = None
        L.graft_tdes_param_count.argtypes = [C.POINTER(TdesDims)]
        L.graft_tdes_param_count.restype = C.c_int64
        L.graft_tdes_step.argtypes = [vp, vp, C.POINTER(TdesBatch), C.POINTER(TdesHyper), i32, vp,
                                      vp, vp, vp, vp, vp]
        L.graft_tdes_device_status.argtypes = [vp, vp]
        L.graft_saba_fit.argtypes = [C.POINTER(SabaReplay), C.POINTER(C.c_float), i32,
                                     C.POINTER(C.c_float), C.POINTER(C.c_float),
                                     C.POINTER(C.c_double), vp]
        L.graft_read_stream.argtypes = [vp, C.c_int64, vp, vp]
        L.graft_status_string.argtypes = [C.c_int]
        L.graft_status_string.restype = C.c_char_p
        L.graft_last_error.argtypes = []
        L.graft_last_error.restype = C.c_char_p
        for n in ("graft_create", "graft_set_scorer", "graft_set_saba", "graft_set_history",
                  "graft_get_history", "graft_set_fusion",
                  "graft_build_tree", "graft_build_tree_static", "graft_accept",
                  "graft_get_device_status",
                  "graft_synth_node_targets", "graft_profile_begin", "graft_profile_end",
                  "graft_mask_to_bias", "graft_commit_accepted", "graft_tdes_create",
                  "graft_tdes_step", "graft_tdes_device_status", "graft_saba_fit",
                  "graft_read_stream"):
            getattr(L, n).restype = C.c_int
        _lib = L
    return _lib


def _ptr(t, dtype=None, name="tensor"):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError("%s must be a CUDA (HIP) tensor" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t.data_ptr()


def _need(t, name, *dims):
    """Raises ValueError unless tensor t (when given) has one extent per entry of
    dims: an int is the exact extent, a 1-tuple (n,) the least one.  Every
    kernel indexes its buffers by the context's sizes and the call's batch, so
    a buffer that is too small would be read or written out of bounds."""
    if t is None:
        return
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch tensor" % name)
    ok = t.dim() == len(dims) and all(
        (s >= d[0]) if isinstance(d, tuple) else (s == d) for s, d in zip(t.shape, dims))
    if not ok:
        want = ", ".join((">=%d" % d[0]) if isinstance(d, tuple) else str(d) for d in dims)
        raise ValueError("%s must be [%s], got %s" % (name, want, list(t.shape)))


def _batch_of(t, name):
    if not isinstance(t, torch.Tensor) or t.dim() < 1:
        raise ValueError("%s must be a tensor whose first extent is the batch" % name)
    return int(t.shape[0])


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _check(status: int, where: str):
    if status != 0:
        raise GraftError(status, where)


class TreeBuffers:
    """Preallocated outputs of one build_tree call (torch tensors on the device)."""

    def __init__(self, ctx: "Context", batch: int, mask=True, topk=True, stats=True, edges=False,
                 node_scores=True, saba_state=True, adj_cos=False, device=None):
        d = ctx.dims
        dev = device or torch.device("cuda", torch.cuda.current_device())
        L, K, N = d.num_pos, d.top_k, d.max_nodes
        W = (N + 63) // 64
        i32 = dict(dtype=torch.int32, device=dev)
        f32 = dict(dtype=torch.float32, device=dev)
        self.batch = batch
        self.sizes = (L, K, N)
        self.budget = torch.empty(batch, **i32)
        self.n_nodes = torch.empty(batch, **i32)
        self.tokens = torch.empty(batch, N, **i32)
        self.parents = torch.empty(batch, N, **i32)
        self.pos_ids = torch.empty(batch, N, **i32)
        # uint64 words of the ancestor bitset, held as int64 (same bits)
        self.mask = torch.empty(batch, N, W, dtype=torch.int64, device=dev) if mask else None
        self.topk_ids = torch.empty(batch, L, K, **i32) if topk else None
        self.topk_logq = torch.empty(batch, L, K, **f32) if topk else None
        self.row_lse = torch.empty(batch, L, **f32) if stats else None
        self.row_maxprob = torch.empty(batch, L, **f32) if stats else None
        self.row_entropy = torch.empty(batch, L, **f32) if stats else None
        self.edge_scores = torch.empty(batch, L, K, K, **f32) if edges else None
        self.node_scores = (torch.empty(batch, N, dtype=torch.float64, device=dev)
                            if node_scores else None)
        self.saba_state = torch.empty(batch, 4, **f32) if saba_state else None
        # cosines of adjacent hidden states (written only when build_tree gets them)
        self.adj_cos = torch.zeros(batch, max(L - 1, 1), **f32) if adj_cos else None
        t = TreeOut()
        for name, _ in TreeOut._fields_:
            setattr(t, name, _ptr(getattr(self, name), name=name))
        self._struct = t

    def as_dict(self) -> dict:
        return {n: getattr(self, n) for n, _ in TreeOut._fields_ if getattr(self, n) is not None}


class Context:
    """A graft_ctx: sizes fixed at creation, workspace owned by the library."""

    def __init__(self, max_batch: int, num_pos: int, vocab: int, top_k: int, max_nodes: int,
                 hist_window: int = 4):
        L = lib()
        self.dims = Dims(max_batch, num_pos, vocab, top_k, max_nodes, hist_window)
        h = C.c_void_p()
        _check(L.graft_create(C.byref(self.dims), C.byref(h)), "graft_create")
        self._h = h
        self._keep = []

    def close(self):
        if getattr(self, "_h", None):
            lib().graft_destroy(self._h)
            self._h = None

    def __del__(self):  # pragma: no cover
        try:
            self.close()
        except Exception:
            pass

    def set_scorer(self, emb, g_parent, g_child, depth_emb=None, scale=1.0, beta=1.0, center=0):
        dm = self.dims
        _need(emb, "emb", dm.vocab, (1,))
        E = int(emb.shape[1])
        _need(g_parent, "g_parent", E, (1,))
        m = int(g_parent.shape[1])
        _need(g_child, "g_child", E, m)
        _need(depth_emb, "depth_emb", dm.num_pos, m)
        d = ScorerDesc(_ptr(emb, torch.float32, "emb"), _ptr(g_parent, torch.float32, "g_parent"),
                       _ptr(g_child, torch.float32, "g_child"),
                       _ptr(depth_emb, torch.float32, "depth_emb"), emb.shape[1],
                       g_parent.shape[1], float(scale), float(beta), int(center))
        self._keep = [emb, g_parent, g_child, depth_emb]
        _check(lib().graft_set_scorer(self._h, C.byref(d), _stream()), "graft_set_scorer")

    def set_saba(self, budgets, phi, tau_min=1.0, c0=1.0, c1=0.0, c2=0.0):
        arr = (C.c_int32 * len(budgets))(*[int(b) for b in budgets])
        d = SabaDesc(C.cast(arr, C.c_void_p), len(budgets), (C.c_float * 4)(*map(float, phi)),
                     float(tau_min), float(c0), float(c1), float(c2))
        _check(lib().graft_set_saba(self._h, C.byref(d)), "graft_set_saba")

    def set_fusion(self, enable=True):
        """Lets the selection kernel compute the edge scores and the budget
        itself when the rows fit its stage (graft_set_fusion); returns True
        when that path is taken for this context."""
        active = C.c_int32(0)
        _check(lib().graft_set_fusion(self._h, 1 if enable else 0, C.byref(active)),
               "graft_set_fusion")
        return bool(active.value)

    def set_history(self, init):
        _need(init, "init", (1,), self.dims.hist_window)
        _check(lib().graft_set_history(self._h, init.shape[0], _ptr(init, torch.int32, "init"),
                                       _stream()), "graft_set_history")

    def get_history(self, batch: int):
        """(ring [batch, hist_window], pos [batch]) int32 copies of the device
        acceptance-history ring."""
        dev = torch.device("cuda", torch.cuda.current_device())
        ring = torch.empty(batch, self.dims.hist_window, dtype=torch.int32, device=dev)
        pos = torch.empty(batch, dtype=torch.int32, device=dev)
        _check(lib().graft_get_history(self._h, int(batch), _ptr(ring, torch.int32, "ring"),
                                       _ptr(pos, torch.int32, "pos"), _stream()),
               "graft_get_history")
        return ring, pos

    def build_tree(self, logits, root_token, base_pos, prefix_len=None, hist=None,
                   fixed_budget=None, hidden=None, out: TreeBuffers | None = None,
                   static_scratch=False, **want) -> TreeBuffers:
        """hidden: optional [batch, L, H] bf16 bit patterns of the drafter's hidden
        states; with them the SABA state uses the degeneration signal.
        static_scratch: call graft_build_tree_static (no device allocation in the
        library; pass preallocated `out` to allocate nothing here either)."""
        dm = self.dims
        batch = _batch_of(logits, "logits")
        _need(logits, "logits", batch, dm.num_pos, dm.vocab)
        for name, t in (("root_token", root_token), ("base_pos", base_pos),
                        ("prefix_len", prefix_len), ("hist", hist), ("fixed_budget", fixed_budget)):
            _need(t, name, batch)
        if root_token is None or base_pos is None:
            raise ValueError("root_token and base_pos are required")
        _need(hidden, "hidden", batch, dm.num_pos, (1,))
        if out is None:
            out = TreeBuffers(self, batch, **want)
        elif out.batch < batch or out.sizes != (dm.num_pos, dm.top_k, dm.max_nodes):
            raise ValueError("out holds %d sequences of sizes (L, K, max_nodes) = %s; this call "
                             "needs %d of %s" % (out.batch, out.sizes, batch,
                                                 (dm.num_pos, dm.top_k, dm.max_nodes)))
        if logits.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
            raise TypeError("logits must hold bf16 bit patterns")
        if hidden is not None and hidden.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
            raise TypeError("hidden must hold bf16 bit patterns")
        r = RoundIn(batch, _ptr(logits, None, "logits"), _ptr(root_token, torch.int32, "root_token"),
                    _ptr(base_pos, torch.int32, "base_pos"),
                    _ptr(prefix_len, torch.int32, "prefix_len"), _ptr(hist, torch.float32, "hist"),
                    _ptr(fixed_budget, torch.int32, "fixed_budget"), _ptr(hidden, None, "hidden"),
                    0 if hidden is None else int(hidden.shape[-1]))
        fn = "graft_build_tree_static" if static_scratch else "graft_build_tree"
        _check(getattr(lib(), fn)(self._h, C.byref(r), C.byref(out._struct), _stream()), fn)
        return out

    def accept(self, n_nodes, tokens, parents, target_root=None, target_node=None,
               target_depth=None, update_history=False, acc_len=None, acc_nodes=None, bonus=None):
        dm = self.dims
        batch = _batch_of(n_nodes, "n_nodes")
        _need(n_nodes, "n_nodes", batch)
        _need(tokens, "tokens", (batch,), dm.max_nodes)
        _need(parents, "parents", (batch,), dm.max_nodes)
        _need(target_root, "target_root", (batch,))
        _need(target_node, "target_node", (batch,), dm.max_nodes)
        _need(target_depth, "target_depth", (batch,), dm.num_pos + 1)
        _need(acc_len, "acc_len", (batch,))
        _need(acc_nodes, "acc_nodes", (batch,), dm.num_pos)
        _need(bonus, "bonus", (batch,))
        dev = n_nodes.device
        acc_len = torch.empty(batch, dtype=torch.int32, device=dev) if acc_len is None else acc_len
        acc_nodes = (torch.empty(batch, self.dims.num_pos, dtype=torch.int32, device=dev)
                     if acc_nodes is None else acc_nodes)
        bonus = torch.empty(batch, dtype=torch.int32, device=dev) if bonus is None else bonus
        t = Targets(_ptr(target_root, torch.int32, "target_root"),
                    _ptr(target_node, torch.int32, "target_node"),
                    _ptr(target_depth, torch.int32, "target_depth"))
        _check(lib().graft_accept(self._h, batch, _ptr(n_nodes, torch.int32, "n_nodes"),
                                  _ptr(tokens, torch.int32, "tokens"),
                                  _ptr(parents, torch.int32, "parents"), C.byref(t),
                                  _ptr(acc_len, torch.int32, "acc_len"),
                                  _ptr(acc_nodes, torch.int32, "acc_nodes"),
                                  _ptr(bonus, torch.int32, "bonus"), int(bool(update_history)),
                                  _stream()), "graft_accept")
        return acc_len, acc_nodes, bonus

    def synth_node_targets(self, seed, root_token, n_nodes, tokens, parents, topk_ids,
                           target_root=None, target_node=None):
        dm = self.dims
        batch = _batch_of(n_nodes, "n_nodes")
        _need(n_nodes, "n_nodes", batch)
        _need(root_token, "root_token", (batch,))
        _need(tokens, "tokens", (batch,), dm.max_nodes)
        _need(parents, "parents", (batch,), dm.max_nodes)
        _need(topk_ids, "topk_ids", (batch,), dm.num_pos, dm.top_k)
        _need(target_root, "target_root", (batch,))
        _need(target_node, "target_node", (batch,), dm.max_nodes)
        dev = n_nodes.device
        if target_root is None:
            target_root = torch.empty(batch, dtype=torch.int32, device=dev)
        if target_node is None:
            target_node = torch.empty(batch, self.dims.max_nodes, dtype=torch.int32, device=dev)
        _check(lib().graft_synth_node_targets(
            self._h, batch, C.c_uint64(int(seed) & ((1 << 64) - 1)),
            _ptr(root_token, torch.int32, "root_token"), _ptr(n_nodes, torch.int32, "n_nodes"),
            _ptr(tokens, torch.int32, "tokens"), _ptr(parents, torch.int32, "parents"),
            _ptr(topk_ids, torch.int32, "topk_ids"), _ptr(target_root, torch.int32, "target_root"),
            _ptr(target_node, torch.int32, "target_node"), _stream()), "graft_synth_node_targets")
        return target_root, target_node

    def mask_to_bias(self, n_nodes, mask, bias=None, dtype=torch.bfloat16):
        """Additive attention bias of the draft block (0 / -inf) from the ancestor
        masks.  bias: [batch, max_nodes, >= max_nodes] tensor or strided view with
        unit stride along the last dimension (e.g. the tree columns of a wider
        bias); allocated as [batch, max_nodes, max_nodes] when None."""
        batch = _batch_of(n_nodes, "n_nodes")
        N = self.dims.max_nodes
        _need(n_nodes, "n_nodes", batch)
        _need(mask, "mask", (batch,), N, (N + 63) // 64)
        if bias is None:
            bias = torch.empty(batch, N, N, dtype=dtype, device=n_nodes.device)
        if bias.dtype not in (torch.float32, torch.bfloat16):
            raise TypeError("bias must be float32 or bfloat16")
        if bias.dim() != 3 or bias.shape[0] < batch or bias.shape[1] < N or bias.shape[2] < N:
            raise ValueError("bias must be at least [batch, max_nodes, max_nodes]")
        if bias.stride(2) != 1:
            raise ValueError("bias must have unit stride along its last dimension")
        _check(lib().graft_mask_to_bias(self._h, batch, _ptr(n_nodes, torch.int32, "n_nodes"),
                                        _ptr(mask, torch.int64, "mask"), bias.data_ptr(),
                                        1 if bias.dtype == torch.bfloat16 else 0,
                                        bias.stride(1), bias.stride(0), _stream()),
               "graft_mask_to_bias")
        return bias

    def commit_accepted(self, acc_len, acc_nodes, src, dst=None):
        """Moves the accepted nodes' rows to rows 0..acc_len-1: src and dst are
        [planes, batch, rows, width] tensors (any dtype, unit stride along width);
        dst defaults to src (compaction in place)."""
        dst = src if dst is None else dst
        batch = _batch_of(acc_len, "acc_len")
        _need(acc_len, "acc_len", batch)
        _need(acc_nodes, "acc_nodes", (batch,), self.dims.num_pos)
        # node indices reach max_nodes - 1 in src; at most L rows are written in dst
        _need(src, "src", (1,), (batch,), (self.dims.max_nodes,), (1,))
        _need(dst, "dst", (1,), (batch,), (self.dims.num_pos,), (1,))
        for name, t in (("src", src), ("dst", dst)):
            if t.device.type != "cuda":
                raise TypeError("%s must be a CUDA (HIP) tensor [planes, batch, rows, width]" % name)
            if t.stride(3) != 1:
                raise ValueError("%s must have unit stride along its last dimension" % name)
        if src.dtype != dst.dtype or src.shape[0] != dst.shape[0] or src.shape[3] != dst.shape[3]:
            raise ValueError("src and dst must agree in dtype, planes and width")
        es = src.element_size()
        _check(lib().graft_commit_accepted(
            self._h, batch, _ptr(acc_len, torch.int32, "acc_len"),
            _ptr(acc_nodes, torch.int32, "acc_nodes"), src.data_ptr(), dst.data_ptr(),
            src.shape[3] * es, src.shape[0], src.stride(0) * es, src.stride(1) * es,
            src.stride(2) * es, dst.stride(0) * es, dst.stride(1) * es, dst.stride(2) * es,
            _stream()), "graft_commit_accepted")
        return dst

    def profile_begin(self, max_calls: int):
        _check(lib().graft_profile_begin(self._h, int(max_calls)), "graft_profile_begin")

    def profile_end(self):
        """(summed ms, timed launches) per stage: logits, edges + budget, select, accept."""
        ms = (C.c_double * 4)()
        n = (C.c_int32 * 4)()
        _check(lib().graft_profile_end(self._h, ms, n), "graft_profile_end")
        return list(ms), list(n)

    def device_status(self) -> int:
        return lib().graft_get_device_status(self._h, _stream())


class TdesTrainer:
    """A graft_tdes: one TDES training step per call (objectives of eq.
    tdes-training and AdamW), on tensors the caller owns.  theta, adam_m and
    adam_v are fp32 [param_count] vectors laid out as g_parent [E, m] |
    g_child [E, m] | depth_emb [L, m] | scale."""

    def __init__(self, vocab: int, emb_dim: int, score_dim: int, num_pos: int, top_k: int,
                 max_groups: int, max_pairs: int):
        L = lib()
        self.dims = TdesDims(vocab, emb_dim, score_dim, num_pos, top_k, max_groups, max_pairs)
        h = C.c_void_p()
        _check(L.graft_tdes_create(C.byref(self.dims), C.byref(h)), "graft_tdes_create")
        self._h = h
        self.param_count = int(L.graft_tdes_param_count(C.byref(self.dims)))

    def close(self):
        if getattr(self, "_h", None):
            lib().graft_tdes_destroy(self._h)
            self._h = None

    def __del__(self):  # pragma: no cover
        try:
            self.close()
        except Exception:
            pass

    def split(self, theta):
        """Views (g_parent, g_child, depth_emb, scale) of a parameter vector."""
        d = self.dims
        n = d.emb_dim * d.score_dim
        return (theta[:n].view(d.emb_dim, d.score_dim), theta[n:2 * n].view(d.emb_dim, d.score_dim),
                theta[2 * n:2 * n + d.num_pos * d.score_dim].view(d.num_pos, d.score_dim),
                theta[-1:])

    def step(self, emb, batch: dict, theta, adam_m, adam_v, step: int, hyper: TdesHyper = None,
             loss=None, grad=None):
        """One step on `batch` (CUDA tensors: parent, depth, target int32 [G]; child
        int32 [G, K]; logq, z float32 [G, K]; pairs int32 [P, 6]).  Updates theta,
        adam_m, adam_v in place; writes loss (float64 [4]) and grad when given."""
        d = self.dims
        G = int(batch["child"].shape[0]) if "child" in batch else 0
        P = int(batch["pairs"].shape[0]) if "pairs" in batch else 0
        if G and tuple(batch["child"].shape) != (G, d.top_k):
            raise ValueError("child must be [G, %d]" % d.top_k)
        i32, f32 = torch.int32, torch.float32
        b = TdesBatch(G, _ptr(batch["parent"], i32, "parent") if G else None,
                      _ptr(batch["depth"], i32, "depth") if G else None,
                      _ptr(batch["child"], i32, "child") if G else None,
                      _ptr(batch["logq"], f32, "logq") if G else None,
                      _ptr(batch["z"], f32, "z") if G else None,
                      _ptr(batch["target"], i32, "target") if G else None,
                      P, _ptr(batch["pairs"], i32, "pairs") if P else None)
        if G:
            for k in ("parent", "depth", "target"):
                if batch[k].numel() != G:
                    raise ValueError("%s must have %d entries" % (k, G))
            for k in ("logq", "z"):
                if tuple(batch[k].shape) != (G, d.top_k):
                    raise ValueError("%s must be [G, K]" % k)
        if P and tuple(batch["pairs"].shape) != (P, 6):
            raise ValueError("pairs must be [P, 6]")
        for name, t in (("theta", theta), ("adam_m", adam_m), ("adam_v", adam_v), ("grad", grad)):
            if t is not None and t.numel() != self.param_count:
                raise ValueError("%s must have %d entries" % (name, self.param_count))
        if tuple(emb.shape) != (d.vocab, d.emb_dim):
            raise ValueError("emb must be [%d, %d]" % (d.vocab, d.emb_dim))
        if loss is not None and (loss.dtype != torch.float64 or loss.numel() < 4):
            raise ValueError("loss must be float64 with 4 entries")
        h = hyper if hyper is not None else TdesHyper()
        _check(lib().graft_tdes_step(self._h, _ptr(emb, f32, "emb"), C.byref(b), C.byref(h),
                                     int(step), _ptr(theta, f32, "theta"),
                                     _ptr(adam_m, f32, "adam_m"), _ptr(adam_v, f32, "adam_v"),
                                     _ptr(loss, torch.float64, "loss"), _ptr(grad, f32, "grad"),
                                     _stream()), "graft_tdes_step")

    def device_status(self) -> int:
        return lib().graft_tdes_device_status(self._h, _stream())


def saba_fit(budgets, state, prefix, accepted, latency, tau_min, phi_init, max_iter=200):
    """SABA's gain weights phi and cost c0..c2 fitted on a same-prefix replay
    log (graft_saba_fit): budgets a host sequence of ints; state [T, 3],
    prefix [T] int32, accepted and latency [T, n_budgets] float32 as CUDA
    tensors.  Returns a dict with phi (4), c (3), gain_sse, cost_sse,
    iterations and converged."""
    import numpy as np
    T = int(state.shape[0])
    nb = len(budgets)
    b = np.ascontiguousarray(np.asarray(budgets, np.int32))
    for name, t, shape in (("state", state, (T, 3)), ("accepted", accepted, (T, nb)),
                           ("latency", latency, (T, nb))):
        if tuple(t.shape) != shape:
            raise ValueError("%s must be %s" % (name, shape))
    if tuple(prefix.shape) != (T,):
        raise ValueError("prefix must be [T]")
    log = SabaReplay(T, nb, b.ctypes.data, _ptr(state, torch.float32, "state"),
                     _ptr(prefix, torch.int32, "prefix"), _ptr(accepted, torch.float32, "accepted"),
                     _ptr(latency, torch.float32, "latency"), float(tau_min))
    phi0 = (C.c_float * 4)(*[float(v) for v in phi_init])
    phi = (C.c_float * 4)()
    c = (C.c_float * 3)()
    st = (C.c_double * 4)()
    _check(lib().graft_saba_fit(C.byref(log), phi0, int(max_iter), phi, c, st, _stream()),
           "graft_saba_fit")
    return dict(phi=list(phi), c=list(c), gain_sse=st[0], cost_sse=st[1], iterations=int(st[2]),
                converged=bool(st[3]))


def read_stream(src, sink=None):
    """A plain read of every byte of the contiguous CUDA tensor src
    (graft_read_stream): the streaming read rate to compare the logits pass
    with.  Returns the sink, READ_STREAM_SINK_WORDS int32 words whose xor is the
    xor of src's 32-bit words."""
    if not isinstance(src, torch.Tensor) or src.device.type != "cuda" or not src.is_contiguous():
        raise TypeError("src must be a contiguous CUDA (HIP) tensor")
    if sink is None:
        sink = torch.empty(READ_STREAM_SINK_WORDS, dtype=torch.int32, device=src.device)
    if sink.numel() < READ_STREAM_SINK_WORDS:
        raise ValueError("sink must hold %d words" % READ_STREAM_SINK_WORDS)
    _check(lib().graft_read_stream(src.data_ptr(), src.numel() * src.element_size(),
                                   _ptr(sink, torch.int32, "sink"), _stream()), "graft_read_stream")
    return sink
