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
