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


# ============================================================================ full decoder block

def _dec(seed, d=8, f=12, H=2, Hkv=1, hd=4, L=4, dense=True):
    r = np.random.default_rng(seed)
    A = r.standard_normal((d, 2 * d))
    return B.DecoderBlock(gamma1=1 + 0.1 * r.standard_normal(d), Wq=0.4 * r.standard_normal((H * hd, d)),
                          Wk=0.4 * r.standard_normal((Hkv * hd, d)), Wv=0.4 * r.standard_normal((Hkv * hd, d)),
                          Wo=0.4 * r.standard_normal((d, H * hd)), gamma2=1 + 0.1 * r.standard_normal(d),
                          Wg=0.3 * r.standard_normal((f, d)), Wu=0.3 * r.standard_normal((f, d)),
                          Wd=0.3 * r.standard_normal((d, f)), n_heads=H, n_kv=Hkv, head_dim=hd, seq_len=L,
                          F=(A @ A.T / (2 * d)) if dense else None)


def test_rope_is_a_rotation_and_its_inverse_undoes_it():
    r = np.random.default_rng(20)
    x = r.standard_normal((12, 3 * 8))
    y = B.rope(x, 3, 8, 5)
    np.testing.assert_allclose(B.rope(y, 3, 8, 5, inverse=True), x, rtol=0, atol=1e-13)
    # each (i, i + hd/2) pair keeps its length; position 0 is the identity
    xr, yr = x.reshape(12, 3, 8), y.reshape(12, 3, 8)
    np.testing.assert_allclose(xr[..., :4] ** 2 + xr[..., 4:] ** 2, yr[..., :4] ** 2 + yr[..., 4:] ** 2, rtol=1e-12)
    np.testing.assert_allclose(y[0], x[0], rtol=0, atol=0)
    np.testing.assert_allclose(y[5], x[5], rtol=0, atol=0)        # position 5 mod 5 = 0


def test_single_token_sequences_make_attention_the_identity_on_values():
    r = np.random.default_rng(21)
    qr, kr, v = r.standard_normal((6, 8)), r.standard_normal((6, 4)), r.standard_normal((6, 4))
    O, P = B.attention_forward(qr, kr, v, 2, 1, 4, 1)
    np.testing.assert_allclose(O, np.concatenate([v, v], axis=1), rtol=0, atol=1e-15)
    assert (P == 1.0).all()


def test_rope_pair0_turns_by_the_position_and_scores_depend_on_relative_position():
    """Pair 0 has frequency base^0 = 1, so at position t it turns by exactly t radians; and a
    rotary embedding makes q(t1) . k(t2) a function of t1 - t2 only."""
    hd, L = 8, 16
    e0 = np.zeros((L, hd))
    e0[:, 0] = 1.0
    y = B.rope(e0, 1, hd, L)
    t = np.arange(L)
    np.testing.assert_allclose(y[:, 0], np.cos(t), rtol=0, atol=1e-14)
    np.testing.assert_allclose(y[:, hd // 2], np.sin(t), rtol=0, atol=1e-14)
    r = np.random.default_rng(23)
    q, k = r.standard_normal(hd), r.standard_normal(hd)
    Q = B.rope(np.tile(q, (L, 1)), 1, hd, L)
    K = B.rope(np.tile(k, (L, 1)), 1, hd, L)
    S = Q @ K.T
    for dlt in range(-3, 4):
        vals = [S[i, i - dlt] for i in range(max(0, dlt), min(L, L + dlt))]
        np.testing.assert_allclose(vals, vals[0], rtol=1e-12, atol=1e-12)


def test_zero_queries_give_causal_prefix_means_per_sequence_and_kv_head():
    """With qr = 0 every allowed score is 0, so each query averages the values of its own sequence up
    to and including its position, read from key/value head h // (H / Hkv)."""
    r = np.random.default_rng(24)
    H, Hkv, hd, L = 4, 2, 3, 5
    T = 2 * L
    v = r.standard_normal((T, Hkv * hd))
    O, P = B.attention_forward(np.zeros((T, H * hd)), r.standard_normal((T, Hkv * hd)), v, H, Hkv, hd, L)
    for t in range(T):
        s0 = (t // L) * L
        for h in range(H):
            g = h // (H // Hkv)
            mean = v[s0:t + 1, g * hd:(g + 1) * hd].mean(axis=0)
            np.testing.assert_allclose(O[t, h * hd:(h + 1) * hd], mean, rtol=0, atol=1e-14)
    assert np.allclose(P.sum(axis=-1), 1.0) and (np.triu(P[0, 0], 1) == 0).all()


def test_two_token_scores_are_scaled_by_root_head_dim():
    """hd = 4, k0 = 0, k1 = e0, q1 = 2 ln(3) e0: the scores of query 1 are 0 and ln 3, so its
    weights are exactly 1/4 and 3/4."""
    hd = 4
    qr = np.zeros((2, hd))
    qr[1, 0] = 2.0 * np.log(3.0)
    kr = np.zeros((2, hd))
    kr[1, 0] = 1.0
    v = np.array([[1.0, 0, 0, 0], [0, 1.0, 0, 0]])
    O, P = B.attention_forward(qr, kr, v, 1, 1, hd, 2)
    np.testing.assert_allclose(P[0, 0, 1], [0.25, 0.75], rtol=1e-15)
    np.testing.assert_allclose(O[1], [0.25, 0.75, 0, 0], rtol=1e-15, atol=1e-16)
    np.testing.assert_allclose(O[0], v[0], rtol=0, atol=0)


def test_attention_backward_matches_finite_differences():
    r = np.random.default_rng(22)
    H, Hkv, hd, L = 4, 2, 3, 5
    T = 2 * L
    qr, kr, v = r.standard_normal((T, H * hd)), r.standard_normal((T, Hkv * hd)), r.standard_normal((T, Hkv * hd))
    c = r.standard_normal((T, H * hd))
    O, P = B.attention_forward(qr, kr, v, H, Hkv, hd, L)
    dq, dk, dv = B.attention_backward(c, P, qr, kr, v, H, Hkv, hd, L)
    L_of = lambda a, b, w: float(np.sum(c * B.attention_forward(a, b, w, H, Hkv, hd, L)[0]))
    for idx in [(0, 0), (3, 5), (9, 11), (7, 2)]:
        assert dq[idx] == pytest.approx(_fd(lambda x: L_of(x, kr, v), qr, idx), rel=1e-6, abs=1e-10)
    for idx in [(0, 0), (4, 5), (9, 3), (6, 1)]:
        assert dk[idx] == pytest.approx(_fd(lambda x: L_of(qr, x, v), kr, idx), rel=1e-6, abs=1e-10)
        assert dv[idx] == pytest.approx(_fd(lambda x: L_of(qr, kr, x), v, idx), rel=1e-6, abs=1e-10)


@pytest.mark.parametrize("which", list(B.DECODER_MODULES))
@pytest.mark.parametrize("alpha", [1.0, 0.4])
def test_decoder_module_gradients_match_finite_differences(which, alpha):
    blk, nxt = _dec(23), _dec(24)
    r = np.random.default_rng(25)
    T = 8
    X = r.standard_normal((T, 8))
    Xh = X + 0.05 * r.standard_normal((T, 8))
    ystar = B.decoder_forward(X, blk, rnd=False).y
    y2star = B.decoder_forward(ystar, nxt, rnd=False).y
    W = {k: v + 0.02 * r.standard_normal(v.shape) for k, v in blk.weights().items()}
    J = slice(2, W[which].shape[1])

    def Lf(Wm):
        Wc = dict(W)
        Wc[which] = Wm
        f = B.decoder_forward(Xh, blk, Wc, rnd=False)
        return B.decoder_surrogate(f, ystar, blk, T, Wc, nxt, y2star, alpha, rnd=False)[0]

    f = B.decoder_forward(Xh, blk, W, rnd=False)
    _, bw = B.decoder_surrogate(f, ystar, blk, T, W, nxt, y2star, alpha, rnd=False)
    G = B.decoder_module_grad(which, f, bw, J)
    rows, cols = W[which].shape
    for (i, j) in [(0, 2), (rows - 1, cols - 1), (rows // 2, 3), (1, cols - 2)]:
        num = _fd(Lf, W[which], (i, j))
        assert G[i, j - 2] == pytest.approx(num, rel=1e-6, abs=1e-11), (which, i, j)


def test_decoder_input_gradient_matches_finite_differences():
    blk = _dec(26)
    r = np.random.default_rng(27)
    T = 8
    X = r.standard_normal((T, 8))
    ystar = r.standard_normal((T, 8))
    Lf = lambda x: B.fisher_loss(B.decoder_forward(x, blk, rnd=False).y - ystar, blk.F, T)
    f = B.decoder_forward(X, blk, rnd=False)
    gy = (f.y - ystar) @ blk.F / T
    dx = B.decoder_backward(f, gy, blk)["x"]
    for idx in [(0, 0), (3, 5), (7, 7), (5, 2)]:
        assert dx[idx] == pytest.approx(_fd(Lf, X, idx), rel=1e-6, abs=1e-11)


def _dec_inputs(seed=30):
    inp = synth.make_mlp_block(256, 256, 384, seed=seed)
    r = np.random.default_rng(seed)
    d, H, Hkv, hd = 256, 4, 2, 64
    blk = B.DecoderBlock(gamma1=1 + 0.1 * r.standard_normal(d), Wq=0.02 * r.standard_normal((H * hd, d)),
                         Wk=0.02 * r.standard_normal((Hkv * hd, d)), Wv=0.02 * r.standard_normal((Hkv * hd, d)),
                         Wo=0.02 * r.standard_normal((d, H * hd)), gamma2=inp.gamma, Wg=inp.Wg, Wu=inp.Wu,
                         Wd=inp.Wd, n_heads=H, n_kv=Hkv, head_dim=hd, seq_len=64, F=None)
    return inp.X, inp.Xhat, blk


def test_decoder_sweep_of_leading_modules_matches_the_full_sweep():
    """Sweeping only q and k gives their codes and weights of the full sweep (the later modules
    come after them in Alg. 1), and the final loss is taken with the rest at their given weights."""
    X, Xh, blk = _dec_inputs(31)
    full = B.decoder_block_sweep(X, Xh, blk, steps=1, lr=1e-4)
    part = B.decoder_block_sweep(X, Xh, blk, steps=1, lr=1e-4, modules=("q", "k"))
    assert sorted(part.modules) == ["k", "q"]
    for name in ("q", "k"):
        assert (part.modules[name].codes == full.modules[name].codes).all(), name
        assert np.array_equal(part.modules[name].W_hat, full.modules[name].W_hat), name
    W = {k: np.asarray(v, np.float64) for k, v in blk.weights().items()}
    W["q"], W["k"] = part.modules["q"].W_hat, part.modules["k"].W_hat
    y = B.decoder_forward(Xh, blk, W).y
    assert part.loss_final == B.fisher_loss(y - part.ystar, blk.F, X.shape[0])
    with pytest.raises(ValueError):
        B.decoder_block_sweep(X, Xh, blk, modules=("k",))


def test_decoder_sweep_without_bgd_is_gptq_on_each_modules_input():
    X, Xh, blk = _dec_inputs()
    res = B.decoder_block_sweep(X, Xh, blk, steps=0)
    W = {k: np.asarray(v, np.float64) for k, v in blk.weights().items()}
    for name in B.DECODER_MODULES:
        f = B.decoder_forward(Xh, blk, W)
        inp = {"q": f.h1, "k": f.h1, "v": f.h1, "o": f.O, "gate": f.mlp.u, "up": f.mlp.u, "down": f.mlp.z}[name]
        ref = quantize_layer(W[name], inp, inp)
        assert (res.modules[name].codes == ref.codes).all(), name
        W[name] = ref.W_hat


# ============================================================================ mini-batch Block-GD

def _batch_sizes(T, batch):
    return [min(T, (i + 1) * batch) - i * batch for i in range(-(-T // batch))]


def _check_token_average(full, mb, sizes, T):
    """With lr = 0 the weights never move, so step k of a column block sees the weights of the
    full-batch run at the same step; each surrogate is a token average, hence the count-weighted
    mean of the batch losses over one cycle of batches is the full-batch loss."""
    nb = len(sizes)
    for name, r in full.modules.items():
        tr_f, tr_b = r.loss_trace, mb.modules[name].loss_trace
        assert len(tr_f) == len(tr_b) and len(tr_f) % nb == 0
        for i in range(0, len(tr_f), nb):
            # a module's steps count from t = 1, so every cycle starts at batch 0
            mean = sum(sizes[j] * tr_b[i + j][2] for j in range(nb)) / T
            assert mean == pytest.approx(tr_f[i][2], rel=1e-11), name
            assert len({tr_b[i + j][2] for j in range(nb)}) == nb   # distinct batches
        assert np.array_equal(r.W_hat, mb.modules[name].W_hat)
    assert mb.loss_final == full.loss_final


def test_mlp_minibatch_losses_average_to_the_full_batch_loss():
    X, Xh, blk = _inputs(seed=12)
    nxt = B.MLPBlock(gamma=blk.gamma[::-1].copy(), Wg=blk.Wu.copy(), Wu=blk.Wg.copy() * 0.5,
                     Wd=blk.Wd[::-1].copy(), F=None)
    T, batch = X.shape[0], 96                       # batches of 96, 96 and a ragged 64
    sizes = _batch_sizes(T, batch)
    kw = dict(steps=len(sizes), lr=0.0, nxt=nxt, window=True)
    full = B.mlp_block_sweep(X, Xh, blk, **kw)
    _check_token_average(full, B.mlp_block_sweep(X, Xh, blk, batch=batch, **kw), sizes, T)
    # a batch of at least T tokens is the full batch, bit for bit
    same = B.mlp_block_sweep(X, Xh, blk, steps=2, lr=1e-3, batch=T)
    ref = B.mlp_block_sweep(X, Xh, blk, steps=2, lr=1e-3)
    assert all(np.array_equal(same.modules[k].W_hat, ref.modules[k].W_hat) for k in B.MODULES)


def test_decoder_minibatch_losses_average_to_the_full_batch_loss():
    X, Xh, blk = _dec_inputs(seed=31)
    nxt = B.DecoderBlock(**{**blk.__dict__, "Wq": blk.Wk.repeat(2, axis=0), "Wo": blk.Wo[::-1].copy(),
                            "gamma1": blk.gamma1[::-1].copy()})
    T, batch = X.shape[0], 2 * blk.seq_len          # two batches of two sequences
    sizes = _batch_sizes(T, batch)
    kw = dict(steps=len(sizes), lr=0.0, nxt=nxt, window=True)
    full = B.decoder_block_sweep(X, Xh, blk, **kw)
    _check_token_average(full, B.decoder_block_sweep(X, Xh, blk, batch=batch, **kw), sizes, T)
    with pytest.raises(ValueError):
        B.decoder_block_sweep(X, Xh, blk, steps=1, batch=blk.seq_len + 8)
