"""CPU pins of the block-level surrogate oracle (oracle/block_oracle.py): every backward against
central finite differences of the unrounded forward, the reduction of the down projection's
gradient to the module-level surrogate, and the sweep's reductions to plain GPTQ."""
import numpy as np
import pytest

import synth
from oracle import block_oracle as B
from oracle.realq_oracle import QParams, quantize_layer


def _blk(seed, d=8, f=12, dense=True):
    r = np.random.default_rng(seed)
    A = r.standard_normal((d, 2 * d))
    return B.MLPBlock(gamma=1.0 + 0.1 * r.standard_normal(d), Wg=0.3 * r.standard_normal((f, d)),
                      Wu=0.3 * r.standard_normal((f, d)), Wd=0.3 * r.standard_normal((d, f)),
                      F=(A @ A.T / (2 * d)) if dense else None)


def _fd(fun, x, idx, h=1e-6):
    xp, xm = x.copy(), x.copy()
    xp[idx] += h
    xm[idx] -= h
    return (fun(xp) - fun(xm)) / (2 * h)


def test_rmsnorm_backward_matches_finite_differences():
    r = np.random.default_rng(1)
    h = r.standard_normal((5, 7))
    gamma = 1 + 0.2 * r.standard_normal(7)
    c = r.standard_normal((5, 7))
    du = c                                   # L = sum(c * rmsnorm(h))
    g = B.rmsnorm_backward(h, gamma, du)
    for idx in [(0, 0), (2, 3), (4, 6), (1, 5)]:
        num = _fd(lambda x: float(np.sum(c * B.rmsnorm(x, gamma))), h, idx)
        assert g[idx] == pytest.approx(num, rel=1e-7, abs=1e-10)


def test_block_input_gradient_matches_finite_differences():
    blk = _blk(2)
    r = np.random.default_rng(3)
    T = 6
    h = r.standard_normal((T, 8))
    ystar = r.standard_normal((T, 8))

    def L(x):
        fw = B.mlp_forward(x, blk.gamma, blk.Wg, blk.Wu, blk.Wd, rnd=False)
        return B.fisher_loss(fw.y - ystar, blk.F, T)

    fw = B.mlp_forward(h, blk.gamma, blk.Wg, blk.Wu, blk.Wd, rnd=False)
    gy = (fw.y - ystar) @ blk.F / T
    _, _, dh = B.mlp_backward(fw, gy, blk.gamma, blk.Wg, blk.Wu, blk.Wd)
    for idx in [(0, 0), (3, 4), (5, 7), (2, 1)]:
        assert dh[idx] == pytest.approx(_fd(L, h, idx), rel=1e-6, abs=1e-10)


@pytest.mark.parametrize("which", ["gate", "up", "down"])
@pytest.mark.parametrize("alpha", [1.0, 0.3])
def test_module_gradients_match_finite_differences(which, alpha):
    blk, nxt = _blk(4), _blk(5)
    r = np.random.default_rng(6)
    T = 7
    X = r.standard_normal((T, 8))
    Xh = X + 0.05 * r.standard_normal((T, 8))
    ystar = B.mlp_forward(X, blk.gamma, blk.Wg, blk.Wu, blk.Wd, rnd=False).y
    y2star = B.mlp_forward(ystar, nxt.gamma, nxt.Wg, nxt.Wu, nxt.Wd, rnd=False).y
    W = {"gate": blk.Wg + 0.02 * r.standard_normal(blk.Wg.shape),
         "up": blk.Wu + 0.02 * r.standard_normal(blk.Wu.shape),
         "down": blk.Wd + 0.02 * r.standard_normal(blk.Wd.shape)}
    J = slice(3, W[which].shape[1])

    def L(Wm):
        Wc = dict(W)
        Wc[which] = Wm
        fw = B.mlp_forward(Xh, blk.gamma, Wc["gate"], Wc["up"], Wc["down"], rnd=False)
        return B.surrogate(fw, ystar, blk.F, T, nxt, y2star, alpha, rnd=False)[0]

    fw = B.mlp_forward(Xh, blk.gamma, W["gate"], W["up"], W["down"], rnd=False)
    _, gy = B.surrogate(fw, ystar, blk.F, T, nxt, y2star, alpha, rnd=False)
    G = B.module_grad(which, fw, gy, W["gate"], W["up"], W["down"], J)
    assert G.shape == (W[which].shape[0], W[which].shape[1] - 3)
    for (i, j) in [(0, 3), (2, 5), (W[which].shape[0] - 1, W[which].shape[1] - 1), (1, 4)]:
        num = _fd(L, W[which], (i, j))
        assert G[i, j - 3] == pytest.approx(num, rel=1e-6, abs=1e-11)


def test_down_gradient_reduces_to_the_module_surrogate_with_metric_F():
    """Unperturbed block input and no roundings: y - y* = (z Wd^T - z Wd0^T), so the block
    surrogate's gradient of the down projection is the module-level one with M = F."""
    blk = _blk(7)
    r = np.random.default_rng(8)
    T = 9
    X = r.standard_normal((T, 8))
    Wd = blk.Wd + 0.03 * r.standard_normal(blk.Wd.shape)
    fw0 = B.mlp_forward(X, blk.gamma, blk.Wg, blk.Wu, blk.Wd, rnd=False)
    fw = B.mlp_forward(X, blk.gamma, blk.Wg, blk.Wu, Wd, rnd=False)
    _, gy = B.surrogate(fw, fw0.y, blk.F, T, rnd=False)
    J = slice(4, 12)
    G = B.module_grad("down", fw, gy, blk.Wg, blk.Wu, Wd, J)
    ref = B.module_surrogate_grad_of_down(fw.z, fw0.z, Wd, blk.Wd, blk.F, J)
    np.testing.assert_allclose(G, ref, rtol=1e-12, atol=1e-15)


def _inputs(T=256, d=256, f=384, seed=9):
    L = synth.make_module("single_512", m=f, n=d, T=T, seed=seed)
    r = np.random.default_rng(seed)
    blk = B.MLPBlock(gamma=1.0 + 0.1 * r.standard_normal(d), Wg=L.W0.astype(np.float64),
                     Wu=(0.02 * r.standard_normal((f, d))), Wd=(0.02 * r.standard_normal((d, f))), F=None)
    return L.X, L.Xhat, blk


def test_sweep_without_bgd_is_gptq_on_each_modules_input():
    X, Xh, blk = _inputs()
    res = B.mlp_block_sweep(X, Xh, blk, steps=0)
    fw = B.mlp_forward(Xh, blk.gamma, blk.Wg, blk.Wu, blk.Wd)
    g = quantize_layer(blk.Wg, fw.u, fw.u)
    u = quantize_layer(blk.Wu, fw.u, fw.u)
    assert (res.modules["gate"].codes == g.codes).all() and (res.modules["up"].codes == u.codes).all()
    fq = B.mlp_forward(Xh, blk.gamma, g.W_hat, u.W_hat, blk.Wd)
    d = quantize_layer(blk.Wd, fq.z, fq.z)
    assert (res.modules["down"].codes == d.codes).all()
    for r in res.modules.values():
        assert np.array_equal(r.W_hat, r.scales.repeat(128, axis=1)[:, :r.W_hat.shape[1]]
                              * (r.codes - r.zeros.repeat(128, axis=1)[:, :r.W_hat.shape[1]]))


def test_sweep_with_bgd_lowers_the_block_surrogate_and_window_off_ignores_the_partner():
    X, Xh, blk = _inputs(seed=10)
    nxt = B.MLPBlock(gamma=blk.gamma[::-1].copy(), Wg=blk.Wu.copy(), Wu=blk.Wg.copy() * 0.5,
                     Wd=blk.Wd[::-1].copy(), F=None)
    a = B.mlp_block_sweep(X, Xh, blk, steps=0)
    b = B.mlp_block_sweep(X, Xh, blk, steps=3, lr=1e-3)
    assert b.loss_final < a.loss_final
    c = B.mlp_block_sweep(X, Xh, blk, steps=3, lr=1e-3, nxt=nxt, window=False)
    assert c.loss_final == b.loss_final
    w = B.mlp_block_sweep(X, Xh, blk, steps=3, lr=1e-3, nxt=nxt, window=True)
    # first step of the sweep is b_global = 1: alpha = 1, so the first trace value is unchanged
    assert w.modules["gate"].loss_trace[0][2] == b.modules["gate"].loss_trace[0][2]
    assert w.loss_final != b.loss_final
