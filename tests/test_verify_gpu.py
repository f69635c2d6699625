"""Parity of the verifier-side consumers (HIP path through the C ABI) with the
CPU oracle: the additive attention bias of the draft block and the commit of
the accepted path's key/value rows.  Both are integer/byte work: bit-exact."""
import os
import sys

import numpy as np
import pytest

import oracle
import synthetic as S

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import workload as WL  # noqa: E402

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(*a):
    print(*a, flush=True)


def _round(w, mode="literal"):
    inp = S.gen_round(w)
    sc = WL.scorer_inputs(w, mode)
    sp = WL.saba_inputs(w)
    ctx = WL.gpu_context(w, sc, sp, torch)
    g = WL.gpu_round(ctx, w, inp, torch)
    return ctx, inp, g


def _bias_ref(g, b, n_max, words):
    return oracle.mask_to_bias(int(g["n_nodes"][b]), g["mask"][b].view(np.uint64)
                               .reshape(n_max, words))


def _as_f64(t):
    return t.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("wid", [0, 2, 3])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_bias_from_mask(wid, dtype):
    w = S.workload(wid)
    _say("bias workload", wid, dtype)
    ctx, inp, g = _round(w)
    words = (w.n_max + 63) // 64
    out = g["_out"]
    bias = ctx.mask_to_bias(out.n_nodes, out.mask, dtype=dtype)
    got = _as_f64(bias)
    for b in range(w.batch):
        assert np.array_equal(got[b], _bias_ref(g, b, w.n_max, words)), b
    ctx.close()


def test_bias_into_a_wider_buffer_and_ragged_rows():
    """Tree columns of a [batch, N, prefix + N] bias: the prefix columns stay
    untouched; N = 70 is not a multiple of the 16-byte chunk."""
    w = S.workload(0, batch=3, V=5000, L=4, K=3, n_max=70, fixed_budget=70)
    ctx, inp, g = _round(w)
    words = (w.n_max + 63) // 64
    prefix, N = 8, w.n_max
    for dtype, ld in ((torch.bfloat16, 80), (torch.float32, 80)):
        big = torch.full((w.batch, N, prefix + ld), 7.0, dtype=dtype, device="cuda")
        ctx.mask_to_bias(g["_out"].n_nodes, g["_out"].mask, bias=big[:, :, prefix:prefix + N])
        got = _as_f64(big)
        assert (got[:, :, :prefix] == 7.0).all() and (got[:, :, prefix + N:] == 7.0).all()
        for b in range(w.batch):
            assert np.array_equal(got[b, :, prefix:prefix + N], _bias_ref(g, b, N, words)), b
    ctx.close()


def _accepted(ctx, g, inp):
    out = g["_out"]
    return ctx.accept(out.n_nodes, out.tokens, out.parents,
                      target_depth=torch.from_numpy(inp["target_depth"]).cuda())


@pytest.mark.parametrize("width_bytes", [16, 96, 4096, 5008])
def test_commit_accepted_rows(width_bytes):
    w = S.workload(2)
    _say("commit rows", width_bytes)
    ctx, inp, g = _round(w)
    acc_len, acc_nodes, _ = _accepted(ctx, g, inp)
    a, nodes = acc_len.cpu().numpy(), acc_nodes.cpu().numpy()
    assert a.max() > 0
    planes = 3
    gen = torch.Generator(device="cuda").manual_seed(width_bytes)
    src = torch.randint(0, 256, (planes, w.batch, w.n_max, width_bytes), dtype=torch.uint8,
                        device="cuda", generator=gen)
    src_h = src.cpu().numpy()
    # out of place
    dst = torch.zeros_like(src)
    ctx.commit_accepted(acc_len, acc_nodes, src, dst)
    got = dst.cpu().numpy()
    for p in range(planes):
        for b in range(w.batch):
            ref = np.zeros_like(src_h[p, b])
            oracle.gather_rows(int(a[b]), nodes[b, :a[b]], src_h[p, b], ref)
            assert np.array_equal(got[p, b], ref), (p, b)
    # in place (the accepted rows move down; later rows keep their bytes)
    ctx.commit_accepted(acc_len, acc_nodes, src)
    got = src.cpu().numpy()
    for p in range(planes):
        for b in range(w.batch):
            ref = src_h[p, b].copy()
            oracle.gather_rows(int(a[b]), nodes[b, :a[b]], ref, ref)
            assert np.array_equal(got[p, b], ref), (p, b)
    assert ctx.device_status() == 0
    ctx.close()


def test_commit_strided_planes_and_empty_paths():
    """A cache laid out [layers, batch, heads * rows, dim] viewed per head:
    planes and rows with gaps between them; sequences with nothing accepted
    keep every row."""
    w = S.workload(0, batch=4, V=3000, n_max=32, fixed_budget=20)
    ctx, inp, g = _round(w)
    acc_len, acc_nodes, _ = _accepted(ctx, g, inp)
    acc_len[0] = 0
    a, nodes = acc_len.cpu().numpy(), acc_nodes.cpu().numpy()
    full = torch.arange(2 * w.batch * (w.n_max + 8) * 40, dtype=torch.int32,
                        device="cuda").view(2, w.batch, w.n_max + 8, 40)
    view = full[:, :, 4:4 + w.n_max, 8:40]          # rows 4.., columns 8..39 of each row
    before = full.cpu().numpy().copy()
    ctx.commit_accepted(acc_len, acc_nodes, view)
    got = full.cpu().numpy()
    for p in range(2):
        for b in range(w.batch):
            ref = before[p, b].copy()
            rows = ref[4:4 + w.n_max, 8:40].copy()
            oracle.gather_rows(int(a[b]), nodes[b, :a[b]], rows, rows)
            ref[4:4 + w.n_max, 8:40] = rows
            assert np.array_equal(got[p, b], ref), (p, b)
    ctx.close()


def test_verifier_argument_errors():
    import paper_2608_20375_amd as G
    w = S.workload(0, batch=2, V=1000, n_max=32, fixed_budget=8)
    ctx, inp, g = _round(w)
    out = g["_out"]
    flat = torch.zeros(2 * 32 * 32 + 8, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(G.GraftError):              # misaligned bias
        ctx.mask_to_bias(out.n_nodes, out.mask, bias=flat[1:1 + 2 * 32 * 32].view(2, 32, 32))
    with pytest.raises(G.GraftError):              # row stride not a multiple of 8 bf16
        ctx.mask_to_bias(out.n_nodes, out.mask,
                         bias=torch.zeros(2, 32, 36, dtype=torch.bfloat16, device="cuda")[:, :, :32])
    src = torch.zeros(1, 2, 32, 24, dtype=torch.uint8, device="cuda")   # 24-byte rows
    acc_len, acc_nodes, _ = _accepted(ctx, g, inp)
    with pytest.raises(G.GraftError):
        ctx.commit_accepted(acc_len, acc_nodes, src)
    # a node index outside the tree is skipped and reported
    bad = acc_nodes.clone()
    bad[:, 0] = 1000
    acc1 = torch.ones_like(acc_len)
    ctx.commit_accepted(acc1, bad, torch.zeros(1, 2, 32, 16, dtype=torch.uint8, device="cuda"))
    assert ctx.device_status() == 5
    assert ctx.device_status() == 0
    ctx.close()
