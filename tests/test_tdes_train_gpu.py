"""Parity of the TDES training step (HIP path through the C ABI) with the CPU
oracle on the same seeded traces: the objective (eq. tdes-training), its
gradient and the AdamW update.

Tolerances.  The library computes in fp32 (projections on MFMA with fp32
accumulation, per-row softmax terms, per-wave gradient sums) and adds block
partials in fp64.  Every gradient component is a sum of products whose
rounding error is bounded by about (E + rows per wave + 8) * u * S, with u =
2^-24 and S the sum of the magnitudes of its terms (the oracle returns S); for
the shapes here that is below 2e-5 * S, and the test allows 1e-4 * S.  The
objective's terms are positive or cancel mildly: relative 2e-5.  After AdamW,
components whose gradient is large against its error bound must agree to fp32
rounding of the new value; the others only move by at most the learning rate
(the first Adam step has |m_hat / sqrt(v_hat)| <= 1)."""
import os
import sys

import numpy as np
import pytest

import synthetic as S
from oracle import tdes_train as T

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(*a):
    print(*a, flush=True)


def _setup(V, E, m, L, K, G, P, seed=0, step=0):
    import paper_2608_20375_amd as GR
    w = S.workload(3, V=V, L=L, K=K, emb_dim=E, rank=m, seed=seed)
    sc = S.gen_scorer(w, "paper")
    tr = S.gen_traces(w, G, P, step=step)
    theta = np.concatenate([sc["g_parent"].ravel(), sc["g_child"].ravel(),
                            sc["depth_emb"].ravel(), [np.float32(sc["scale"])]]).astype(np.float32)
    tr_gpu = {k: torch.from_numpy(np.ascontiguousarray(v)).cuda() for k, v in tr.items()}
    tt = GR.TdesTrainer(V, E, m, L, K, max(G, 1), max(P, 1))
    assert tt.param_count == theta.size
    return GR, w, sc, tr, tr_gpu, theta, tt


def _gpu_step(tt, emb_gpu, tr_gpu, theta, m1, m2, step, h):
    th = torch.from_numpy(theta.astype(np.float32)).cuda()
    a = torch.from_numpy(m1.astype(np.float32)).cuda()
    b = torch.from_numpy(m2.astype(np.float32)).cuda()
    loss = torch.zeros(4, dtype=torch.float64, device="cuda")
    grad = torch.zeros_like(th)
    tt.step(emb_gpu, tr_gpu, th, a, b, step, h, loss=loss, grad=grad)
    torch.cuda.synchronize()
    return dict(theta=th.cpu().numpy(), m1=a.cpu().numpy(), m2=b.cpu().numpy(),
                loss=loss.cpu().numpy(), grad=grad.cpu().numpy())


def _hyper(GR, **kw):
    d = dict(lambda_kl=1.0, lambda_pair=1.0, lambda_bce=0.25, gamma=1.0, w1=5.0, lr=2e-3,
             weight_decay=1e-4)
    d.update(kw)
    return GR.TdesHyper(**d), T.Hyper(beta1=float(np.float32(0.9)), beta2=float(np.float32(0.999)),
                                      eps=float(np.float32(1e-8)),
                                      **{k: float(np.float32(v)) for k, v in d.items()})


def _compare(got, ref, theta_in, m1_in, m2_in, h):
    np.testing.assert_allclose(got["loss"], np.array(ref["loss"]), rtol=2e-5, atol=1e-9)
    bound = 1e-4 * ref["abs_grad"] + 1e-12
    err = np.abs(got["grad"] - ref["grad"])
    worst = int(np.argmax(err / bound))
    assert (err <= bound).all(), (worst, got["grad"][worst], ref["grad"][worst], bound[worst])
    big = np.abs(ref["grad"]) > 10 * bound
    assert big.mean() > 0.5
    rt = np.abs(ref["theta"])
    np.testing.assert_allclose(got["theta"][big], ref["theta"][big], rtol=2e-6, atol=1e-9)
    decayed = theta_in.astype(np.float64) * (1 - h.lr * h.weight_decay)
    assert (np.abs(got["theta"] - decayed) <= h.lr * (1 + 1e-5) + 2e-6 * rt + 1e-9).all()
    gerr = bound
    np.testing.assert_array_less(np.abs(got["m1"] - ref["m1"]),
                                 (1 - h.beta1) * gerr + 1e-6 * np.abs(ref["m1"]) + 1e-30)
    np.testing.assert_array_less(np.abs(got["m2"] - ref["m2"]),
                                 (1 - h.beta2) * (2 * np.abs(ref["grad"]) + gerr) * gerr
                                 + 1e-6 * np.abs(ref["m2"]) + 1e-30)


SHAPES = [
    # V, E, m, L, K, G, P: ragged children, several waves and blocks
    (500, 32, 8, 4, 5, 37, 11),
    (3000, 64, 16, 16, 8, 300, 70),
    (3000, 64, 40, 8, 33, 150, 50),       # m padded to 48, K over two row tiles
    (2000, 64, 64, 16, 64, 90, 24),       # four row tiles, m = 64
    (5000, 128, 32, 16, 16, 600, 400),
    (5000, 128, 16, 32, 32, 200, 100),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "V%d_E%d_m%d_L%d_K%d_G%d_P%d" % s)
def test_step_matches_oracle(shape):
    V, E, m, L, K, G, P = shape
    _say("tdes step", shape)
    GR, w, sc, tr, tr_gpu, theta, tt = _setup(*shape)
    hg, ho = _hyper(GR)
    emb_gpu = torch.from_numpy(sc["emb"]).cuda()
    z = np.zeros_like(theta)
    got = _gpu_step(tt, emb_gpu, tr_gpu, theta, z, z, 1, hg)
    ref = T.train_step(theta.astype(np.float64), z, z, 1, sc["emb"], tr, ho, E, m, L)
    _compare(got, ref, theta, z, z, ho)
    assert tt.device_status() == 0
    tt.close()


def test_three_steps_from_the_oracle_state():
    """Steps 2 and 3 start from the oracle's state (rounded to fp32): bias
    corrections and moment updates past the first step."""
    shape = (4000, 64, 16, 8, 8, 256, 128)
    V, E, m, L, K, G, P = shape
    GR, w, sc, tr, tr_gpu, theta, tt = _setup(*shape)
    hg, ho = _hyper(GR)
    emb_gpu = torch.from_numpy(sc["emb"]).cuda()
    th, m1, m2 = theta.astype(np.float64), np.zeros(theta.size), np.zeros(theta.size)
    for step in (1, 2, 3):
        th32, a32, b32 = (x.astype(np.float32) for x in (th, m1, m2))
        got = _gpu_step(tt, emb_gpu, tr_gpu, th32, a32, b32, step, hg)
        ref = T.train_step(th32.astype(np.float64), a32.astype(np.float64),
                           b32.astype(np.float64), step, sc["emb"], tr, ho, E, m, L)
        np.testing.assert_allclose(got["loss"], np.array(ref["loss"]), rtol=2e-5, atol=1e-9)
        bound = 1e-4 * ref["abs_grad"] + 1e-12
        assert (np.abs(got["grad"] - ref["grad"]) <= bound).all(), step
        big = np.abs(ref["grad"]) > 10 * bound
        np.testing.assert_allclose(got["theta"][big], ref["theta"][big], rtol=2e-6, atol=1e-9)
        th, m1, m2 = ref["theta"], ref["m1"], ref["m2"]
    tt.close()


def test_full_size_step():
    """The benchmark's batch: 4096 groups of 16 children and 4096 pairs over a
    128256-token vocabulary, E = 128, m = 32, L = 16."""
    shape = (128256, 128, 32, 16, 16, 4096, 4096)
    V, E, m, L, K, G, P = shape
    _say("tdes full-size step")
    GR, w, sc, tr, tr_gpu, theta, tt = _setup(*shape)
    hg, ho = _hyper(GR, w1=15.0)
    emb_gpu = torch.from_numpy(sc["emb"]).cuda()
    z = np.zeros_like(theta)
    got = _gpu_step(tt, emb_gpu, tr_gpu, theta, z, z, 1, hg)
    ref = T.train_step(theta.astype(np.float64), z, z, 1, sc["emb"], tr, ho, E, m, L)
    _compare(got, ref, theta, z, z, ho)
    # deterministic: a second run is bit-identical
    again = _gpu_step(tt, emb_gpu, tr_gpu, theta, z, z, 1, hg)
    for k in ("theta", "m1", "m2", "loss", "grad"):
        assert np.array_equal(got[k], again[k]), k
    tt.close()


@pytest.mark.parametrize("G,P", [(0, 9), (13, 0), (0, 0)])
def test_empty_groups_or_pairs(G, P):
    shape = (700, 32, 8, 4, 4, G, P)
    GR, w, sc, tr, tr_gpu, theta, tt = _setup(*shape)
    hg, ho = _hyper(GR)
    emb_gpu = torch.from_numpy(sc["emb"]).cuda()
    z = np.zeros_like(theta)
    batch = {k: v for k, v in tr_gpu.items() if (G and k != "pairs") or (P and k == "pairs")}
    got = _gpu_step(tt, emb_gpu, batch, theta, z, z, 1, hg)
    ref = T.train_step(theta.astype(np.float64), z, z, 1, sc["emb"], tr, ho, 32, 8, 4)
    np.testing.assert_allclose(got["loss"], np.array(ref["loss"]), rtol=2e-5, atol=1e-12)
    assert (np.abs(got["grad"] - ref["grad"]) <= 1e-4 * ref["abs_grad"] + 1e-12).all()
    if G == 0 and P == 0:
        assert not got["grad"].any()
        # weight decay alone
        np.testing.assert_allclose(got["theta"], theta * np.float32(1 - 2e-3 * 1e-4), rtol=1e-7)
    tt.close()


def test_invalid_ids_are_reported():
    shape = (700, 32, 8, 4, 4, 20, 16)
    GR, w, sc, tr, tr_gpu, theta, tt = _setup(*shape)
    hg, _ = _hyper(GR)
    emb_gpu = torch.from_numpy(sc["emb"]).cuda()
    bad = dict(tr_gpu)
    bad["child"] = tr_gpu["child"].clone()
    bad["child"][3, 1] = 700
    bad["pairs"] = tr_gpu["pairs"].clone()
    bad["pairs"][5, 2] = 0          # depth 0
    z = np.zeros_like(theta)
    got = _gpu_step(tt, emb_gpu, bad, theta, z, z, 1, hg)
    assert np.isfinite(got["theta"]).all() and np.isfinite(got["loss"]).all()
    assert tt.device_status() == 5
    assert tt.device_status() == 0
    tt.close()


def test_argument_errors():
    import paper_2608_20375_amd as GR
    with pytest.raises(GR.GraftError):
        GR.TdesTrainer(1000, 48, 16, 4, 4, 10, 10)        # E not in {32, 64, 128}
    with pytest.raises(GR.GraftError):
        GR.TdesTrainer(1000, 128, 64, 4, 4, 10, 10)       # E * M > 4096
    with pytest.raises(GR.GraftError):
        GR.TdesTrainer(1000, 64, 16, 4, 65, 10, 10)       # K > 64
    shape = (700, 32, 8, 4, 4, 20, 16)
    GR, w, sc, tr, tr_gpu, theta, tt = _setup(*shape)
    hg, _ = _hyper(GR)
    emb_gpu = torch.from_numpy(sc["emb"]).cuda()
    th = torch.from_numpy(theta).cuda()
    z = torch.zeros_like(th)
    with pytest.raises(GR.GraftError):                  # step 0
        tt.step(emb_gpu, tr_gpu, th, z, z.clone(), 0, hg)
    big = {k: torch.cat([v, v]) for k, v in tr_gpu.items()}
    with pytest.raises(GR.GraftError):                  # more groups than the trainer holds
        tt.step(emb_gpu, big, th, z, z.clone(), 1, hg)
    tt.close()
