"""Host-only checks of the C ABI: the built library loads and exports every
entry point of include/graft.h, and the ctypes mirrors of the header's structs
have the C layout (checked by compiling a probe with gcc)."""
import ctypes as C
import os
import re
import subprocess

import pytest

import paper_2608_20375_amd as G

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "graft.h")


def declared_symbols():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"GRAFT_API\s+[\w\s\*]*?\b(graft_\w+)\s*\(", src)))


def test_header_declares_expected_entry_points():
    syms = declared_symbols()
    assert set(syms) == set(G.EXPORTED_SYMBOLS)
    assert "graft_build_tree" in syms and "graft_accept" in syms


def test_library_exports_every_declared_symbol():
    if not os.path.exists(G.library_path()):
        pytest.fail("libgraft.so missing: run __graft_entry__.build()")
    lib = C.CDLL(G.library_path())
    for s in declared_symbols():
        assert hasattr(lib, s), s
    out = subprocess.run(["nm", "-D", "--defined-only", G.library_path()], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\b(graft_\w+)\b", out))
    assert set(declared_symbols()) <= exported


def test_status_strings_without_gpu():
    L = G.lib()
    assert L.graft_status_string(0) == b"ok"
    assert L.graft_status_string(2) == b"unsupported size"


def test_create_rejects_bad_dims_before_touching_the_device():
    L = G.lib()
    h = C.c_void_p()
    bad = [G.Dims(0, 8, 100, 4, 32, 4), G.Dims(1, 65, 100, 4, 32, 4),
           G.Dims(1, 8, 100, 65, 32, 4), G.Dims(1, 8, 3, 4, 32, 4),
           G.Dims(1, 8, 100, 4, 1025, 4), G.Dims(1, 8, 100, 4, 32, 65)]
    codes = [L.graft_create(C.byref(d), C.byref(h)) for d in bad]
    assert codes == [1, 2, 2, 1, 2, 2]
    assert h.value is None
    assert L.graft_create(None, C.byref(h)) == 1


def test_set_fusion_rejects_a_null_context():
    L = G.lib()
    active = C.c_int32(7)
    assert L.graft_set_fusion(None, 1, C.byref(active)) == 1
    assert active.value == 7   # untouched on error


PROBE = r"""
#include <stddef.h>
#include <stdio.h>
#include "graft.h"
#define P(T, f) printf(#T "." #f " %zu\n", offsetof(T, f))
#define S(T) printf(#T " %zu\n", sizeof(T))
int main(void) {
  S(graft_dims); S(graft_scorer_desc); S(graft_saba_desc); S(graft_round_in);
  S(graft_tree_out); S(graft_targets);
  P(graft_scorer_desc, scale); P(graft_scorer_desc, center);
  P(graft_saba_desc, phi); P(graft_saba_desc, c2);
  P(graft_round_in, logits); P(graft_round_in, fixed_budget);
  P(graft_round_in, hidden); P(graft_round_in, hidden_dim);
  P(graft_tree_out, mask); P(graft_tree_out, saba_state); P(graft_tree_out, adj_cos);
  P(graft_targets, target_depth);
  return 0;
}
"""


def test_ctypes_layout_matches_header(tmp_path):
    src = tmp_path / "probe.c"
    src.write_text(PROBE)
    exe = tmp_path / "probe"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.dirname(HEADER), "-o", str(exe), str(src)],
                   check=True)
    got = dict(l.split() for l in subprocess.run([str(exe)], capture_output=True, text=True,
                                                 check=True).stdout.splitlines())
    m = {"graft_dims": G.Dims, "graft_scorer_desc": G.ScorerDesc, "graft_saba_desc": G.SabaDesc,
         "graft_round_in": G.RoundIn, "graft_tree_out": G.TreeOut, "graft_targets": G.Targets}
    for k, v in got.items():
        if "." in k:
            t, f = k.split(".")
            assert getattr(m[t], f).offset == int(v), k
        else:
            assert C.sizeof(m[k]) == int(v), k


def _unbound_context(batch=4, L=3, V=100, K=2, N=32, window=4):
    """A Context object with sizes but no library handle: the binding's shape
    checks run (and raise) before anything reaches the library or a device."""
    ctx = G.Context.__new__(G.Context)
    ctx.dims = G.Dims(batch, L, V, K, N, window)
    ctx._h = None
    ctx._keep = []
    return ctx


def test_binding_rejects_mismatched_shapes_before_any_call():
    torch = pytest.importorskip("torch")
    ctx = _unbound_context()
    i32 = dict(dtype=torch.int32)
    z = lambda *s, **kw: torch.zeros(*s, **(kw or i32))
    logits = z(2, 3, 100, dtype=torch.int16)
    r2 = z(2)
    bad_build = [
        dict(logits=z(2, 4, 100, dtype=torch.int16), root_token=r2, base_pos=r2),   # L
        dict(logits=z(2, 3, 99, dtype=torch.int16), root_token=r2, base_pos=r2),    # V
        dict(logits=z(2, 300, dtype=torch.int16), root_token=r2, base_pos=r2),      # rank
        dict(logits=logits, root_token=z(1), base_pos=r2),
        dict(logits=logits, root_token=r2, base_pos=z(3)),
        dict(logits=logits, root_token=r2, base_pos=r2, prefix_len=z(1)),
        dict(logits=logits, root_token=r2, base_pos=r2, hist=z(1, dtype=torch.float32)),
        dict(logits=logits, root_token=r2, base_pos=r2, fixed_budget=z(2, 1)),
        dict(logits=logits, root_token=r2, base_pos=r2, hidden=z(2, 2, 8, dtype=torch.int16)),
        dict(logits=logits, root_token=None, base_pos=r2),
    ]
    for kw in bad_build:
        with pytest.raises(ValueError):
            ctx.build_tree(**kw)
    # output buffers made for fewer sequences or other sizes
    small = G.TreeBuffers.__new__(G.TreeBuffers)
    small.batch, small.sizes = 1, (3, 2, 32)
    with pytest.raises(ValueError):
        ctx.build_tree(logits, r2, r2, fixed_budget=r2, out=small)
    other = G.TreeBuffers.__new__(G.TreeBuffers)
    other.batch, other.sizes = 4, (3, 2, 64)
    with pytest.raises(ValueError):
        ctx.build_tree(logits, r2, r2, fixed_budget=r2, out=other)

    n = z(2)
    tk = z(2, 32)
    bad_accept = [
        dict(tokens=z(2, 31), parents=tk, target_depth=z(2, 4)),
        dict(tokens=tk, parents=z(1, 32), target_depth=z(2, 4)),
        dict(tokens=tk, parents=tk, target_depth=z(2, 3)),
        dict(tokens=tk, parents=tk, target_depth=z(1, 4)),
        dict(tokens=tk, parents=tk, target_root=z(2), target_node=z(2, 16)),
        dict(tokens=tk, parents=tk, target_root=z(1), target_node=tk),
        dict(tokens=tk, parents=tk, target_depth=z(2, 4), acc_nodes=z(2, 2)),
        dict(tokens=tk, parents=tk, target_depth=z(2, 4), acc_len=z(1)),
        dict(tokens=tk, parents=tk, target_depth=z(2, 4), bonus=z(1)),
    ]
    for kw in bad_accept:
        with pytest.raises(ValueError):
            ctx.accept(n, **kw)

    emb = z(100, 8, dtype=torch.float32)
    g = z(8, 4, dtype=torch.float32)
    for args in ((z(99, 8, dtype=torch.float32), g, g, None),
                 (emb, z(7, 4, dtype=torch.float32), g, None),
                 (emb, g, z(8, 5, dtype=torch.float32), None),
                 (emb, g, g, z(2, 4, dtype=torch.float32))):
        with pytest.raises(ValueError):
            ctx.set_scorer(*args)
    with pytest.raises(ValueError):
        ctx.set_history(z(2, 3))
    with pytest.raises(ValueError):
        ctx.synth_node_targets(1, r2, n, tk, tk, z(2, 3, 1))
    with pytest.raises(ValueError):
        ctx.mask_to_bias(n, z(2, 32, 2, dtype=torch.int64), bias=z(2, 32, 32,
                                                                    dtype=torch.float32))
    with pytest.raises(ValueError):
        ctx.commit_accepted(n, z(2, 3), z(1, 2, 16, 16, dtype=torch.uint8),
                            z(1, 2, 32, 16, dtype=torch.uint8))
