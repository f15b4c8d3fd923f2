"""Pins of the float64 oracle to facts fixed by the paper and by mathematics.

Each test checks one oracle function against something other than itself: a
brute-force loop, a closed form, an identity stated in the paper, finite
differences, or constants printed in the paper.  None of these tests uses the GPU.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle.realq_oracle import (TIE_ATOL, TIE_RTOL, QParams, adam_update, damp_hessian, group_search, hessian, inverse_factor,
                                 pullback_metric, quantize_layer, residual, surrogate_grad, surrogate_loss,
                                 window_alpha)
import synth

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))


def rng(seed=0):
    return np.random.default_rng(seed)


# ============================================================================ Hessian (Sec. 3.2, Eq. saliency_hessian)

def test_hessian_equals_sum_of_outer_products():
    r = rng(1)
    T, n = 7, 5
    X = r.standard_normal((T, n))
    s = np.abs(r.standard_normal(T))
    H = np.zeros((n, n))
    for t in range(T):                       # brute force, one token at a time
        for i in range(n):
            for j in range(n):
                H[i, j] += s[t] * X[t, i] * X[t, j]
    H *= GOLD["gptq_hessian_scale"]["factor"] / T
    np.testing.assert_allclose(hessian(X, s), H, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(hessian(X, None), hessian(X, np.ones(T)), rtol=0, atol=0)


def test_hessian_symmetric_psd():
    r = rng(2)
    X = r.standard_normal((50, 20))
    X[:, 3] = 0.0
    H = hessian(X, np.abs(r.standard_normal(50)))
    assert np.array_equal(H, H.T) or np.allclose(H, H.T, rtol=0, atol=1e-14)
    assert np.linalg.eigvalsh(H).min() > -1e-12
    assert H[3, 3] == 0.0


# ============================================================================ damping and the inverse factor

def test_damping_dead_columns():
    r = rng(3)
    X = r.standard_normal((40, 6))
    X[:, 2] = 0.0
    H = hessian(X)
    Hd, dead = damp_hessian(H, 0.01)
    assert dead.tolist() == [False, False, True, False, False, False]
    fixed = np.diag(H).copy()
    fixed[2] = 1.0
    lam = 0.01 * fixed.mean()
    np.testing.assert_allclose(np.diag(Hd), fixed + lam, rtol=1e-15)
    off = ~np.eye(6, dtype=bool)
    np.testing.assert_array_equal(Hd[off], H[off])


def test_inverse_factor_reconstructs_inverse():
    r = rng(4)
    A = r.standard_normal((60, 40))
    Hd = A.T @ A / 60 + 0.1 * np.eye(40)
    U = inverse_factor(Hd)
    assert np.allclose(U, np.triu(U), rtol=0, atol=0)
    assert (np.diag(U) > 0).all()
    assert np.abs(U.T @ U @ Hd - np.eye(40)).max() < 1e-10


def test_inverse_factor_rows_are_sequentially_eliminated_inverse():
    """U[j, j:] / U_jj is row 0 of inv(Hd[j:, j:]) over its diagonal, U_jj^2 that diagonal (Eq. gptq_update)."""
    r = rng(5)
    n = 12
    A = r.standard_normal((30, n))
    Hd = A.T @ A / 30 + 0.05 * np.eye(n)
    U = inverse_factor(Hd)
    for j in range(n):
        Hinv_F = np.linalg.inv(Hd[j:, j:])
        np.testing.assert_allclose(U[j, j:] / U[j, j], Hinv_F[0, :] / Hinv_F[0, 0], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(U[j, j] ** 2, Hinv_F[0, 0], rtol=1e-10)


# ============================================================================ quantizer: exhaustive search

def _rint_exact(q: Fraction) -> int:
    """Round-half-to-even of an exact rational."""
    f = math.floor(q)
    d = q - f
    if d != Fraction(1, 2):
        return f + (1 if d > Fraction(1, 2) else 0)
    return f + (f % 2)


def brute_force_search(x, bits=4, grid=80):
    """Every (k, z) candidate scored in exact rational arithmetic with plain Python loops.

    The candidate scales are the float64 values s_k = fl(p_k (hi - lo) / maxq); everything
    after that (x / s_k, the codes, the squared error) is exact, so an exact tie stays a
    tie.  Winner: lexicographic (err, k, |z - z_nat|, z), z_nat = rint(-lo maxq / (hi - lo)).
    Returns (scale, zero, exact error of the winner, {(k, z): exact error}).
    """
    maxq = 2 ** bits - 1
    xs = [Fraction(float(v)) for v in x]
    lo = min(Fraction(0), min(xs))
    hi = max(Fraction(0), max(xs))
    if lo == hi:
        lo, hi = Fraction(-1), Fraction(1)
    znat = min(max(_rint_exact(-lo * maxq / (hi - lo)), 0), maxq)
    best, table = None, {}
    for k in range(grid):
        p = 1.0 - k / 100.0
        sf = (p * float(hi - lo)) / maxq
        S = Fraction(sf)
        r = [_rint_exact(xv / S) for xv in xs]
        for z in range(maxq + 1):
            err = Fraction(0)
            for xv, rv in zip(xs, r):
                c = min(max(rv + z, 0), maxq) - z
                d = xv - S * c
                err += d * d
            table[(k, z)] = err
            key = (err, k, abs(z - znat), z)
            if best is None or key < best[0]:
                best = (key, sf)
    return best[1], best[0][3], best[0][0], table


def _check_search(x, bits=4):
    """The oracle's pick against the exact table: its error evaluated to float64 accuracy and,
    where it differs from the exact winner, a member of the tie set that wins on (k, dist, z)."""
    qp = QParams(bits=bits)
    xs = np.asarray(x, dtype=float)
    s, z, e = group_search(xs[None, :], qp)
    bs, bz, be, table = brute_force_search(list(xs), bits)
    lo, hi = min(0.0, xs.min()), max(0.0, xs.max())
    if lo == hi:
        lo, hi = -1.0, 1.0
    ks = [k for k in range(qp.grid) if ((1.0 - k / 100.0) * (hi - lo)) / qp.maxq == s[0]]
    assert ks, s[0]
    pick = (ks[0], int(z[0]))
    ss = sum(Fraction(float(v)) ** 2 for v in xs)
    assert abs(Fraction(float(e[0])) - table[pick]) <= Fraction(1e-12) * table[pick] + Fraction(2.0 ** -100) * ss
    # the reported margin: gap from the least exact error to the least one outside the tie set
    _, _, _, mg = group_search(xs[None, :], qp, with_margin=True)
    emin = min(table.values())
    outside = [v for v in table.values() if v > emin * (1 + Fraction(TIE_RTOL)) + Fraction(TIE_ATOL) * ss]
    if outside and emin > Fraction(1e-12) * ss:       # a relative margin is only defined away from 0
        assert float(mg[0]) == pytest.approx(float((min(outside) - emin) / emin), rel=1e-9, abs=1e-12)
    if (s[0], z[0]) != (bs, bz):
        assert table[pick] <= be * (1 + Fraction(TIE_RTOL)) + Fraction(TIE_ATOL) * ss, (pick, bs, bz)
        znat = min(max(_rint_exact(-Fraction(lo) * qp.maxq / Fraction(hi - lo)), 0), qp.maxq)
        kb = [k for k in range(qp.grid) if ((1.0 - k / 100.0) * (hi - lo)) / qp.maxq == bs][0]
        assert (pick[0], abs(pick[1] - znat), pick[1]) < (kb, abs(bz - znat), bz)
    return s[0], z[0], e[0]


@pytest.mark.parametrize("seed", range(4))
def test_search_matches_exhaustive_random(seed):
    r = rng(10 + seed)
    x = r.standard_normal(16) * 0.02
    _check_search(x)


def test_search_matches_exhaustive_outlier_and_3bit():
    r = rng(20)
    x = r.standard_normal(24) * 0.01
    x[5] = 0.2
    _check_search(x)
    _check_search(r.standard_normal(12), bits=3)


def test_search_all_zero_group():
    s, z, e = _check_search(np.zeros(8))
    # lo = -1, hi = 1: every candidate has zero error; k = 0 and z = z_nat = rint(7.5) = 8
    assert e == 0.0 and z == 8 and s == pytest.approx(2.0 / 15.0, rel=1e-15)


def test_search_exact_grid_group():
    s0 = 0.01
    x = s0 * (np.arange(16) - 5.0)
    s, z, e = _check_search(x)
    assert z == 5 and s == pytest.approx(s0, rel=1e-12) and e < 1e-28


def test_search_constant_group():
    s, z, e = _check_search(np.full(10, 0.3))
    assert e < 1e-28 and z == 0


def _symmetric_bf16_rows(seed, rows=256, g=128):
    """bf16 rows, every other one with its extremes set to -max and +max (lo = -hi)."""
    r = rng(seed)
    x = synth.bf16_round((r.standard_normal((rows, g)) * 0.02).astype(np.float32)).astype(np.float64)
    half = np.arange(0, rows, 2)
    mx = np.abs(x[half]).max(1)
    x[half, x[half].argmin(1)] = -mx
    x[half, x[half].argmax(1)] = mx
    return x


def test_search_symmetric_bf16_tie():
    """lo = -hi: the zero points 7 and 8 clamp opposite extremes and tie exactly; z_nat is
    rint(7.5) = 8.  The oracle must take the exact-arithmetic winner of the brute force."""
    x = _symmetric_bf16_rows(40, rows=8, g=16)[0]
    s, z, e = _check_search(x)
    bs, bz, be, table = brute_force_search(list(x))
    kb = [k for k in range(80) if ((1 - k / 100) * (2 * x.max())) / 15 == bs][0]
    assert table[(kb, 7)] == table[(kb, 8)] == be     # the case really is an exact tie
    assert (s, z) == (bs, bz) and z == 8


def test_search_independent_of_summation_order():
    """Permuting a group's values changes the float64 summation order of every candidate's
    error but not the candidates themselves, so (scale, zero) must not change."""
    x = _symmetric_bf16_rows(41)
    qp = QParams()
    s0, z0, _ = group_search(x, qp)
    for t in range(4):
        perm = rng(100 + t).permutation(x.shape[1])
        s1, z1, _ = group_search(x[:, perm], qp)
        assert (s0 == s1).all() and (z0 == z1).all()


def test_search_finer_grid_gap_is_small():
    """Reported, not a tie-break rule: a 10x finer shrink grid lowers the error only a little."""
    r = rng(30)
    x = r.standard_normal((64, 128)) * 0.02
    _, _, e = group_search(x, QParams())
    maxq = 15
    lo = np.minimum(0, x.min(1)); hi = np.maximum(0, x.max(1))
    best = np.full(64, np.inf)
    for k in range(800):
        p = 1 - k / 1000
        s = p * (hi - lo) / maxq
        for zz in range(16):
            q = np.clip(np.rint(x / s[:, None]) + zz, 0, maxq)
            best = np.minimum(best, ((x - s[:, None] * (q - zz)) ** 2).sum(1))
    assert (best <= e + 1e-18).all()
    assert np.median(e / best) < 1.05


# ============================================================================ GPTQ reduction (K = 0, s = 1, Xhat = X, M = I)

def textbook_obs(W0, X, qp):
    """Column-by-column OBS with the remaining-column Hessian re-inverted at every step."""
    W = np.array(W0, dtype=float)
    H = hessian(X)
    Hd, dead = damp_hessian(H, qp.damp)
    W[:, dead] = 0.0
    m, n = W.shape
    codes = np.zeros((m, n), dtype=int)
    maxq = qp.maxq
    grp = qp.group if qp.group > 0 else n
    for j in range(n):
        if j % grp == 0:
            sc, zz, _ = group_search(W[:, j:j + grp], qp)
            sc = sc.astype(np.float32).astype(float)          # the stored (float32) scale
        q = np.clip(np.rint(W[:, j] / sc) + zz, 0, maxq)
        wq = sc * (q - zz)
        Hinv = np.linalg.inv(Hd[j:, j:])
        err = (W[:, j] - wq) / Hinv[0, 0]
        W[:, j:] -= np.outer(err, Hinv[0, :])
        W[:, j] = wq
        codes[:, j] = q
    return codes, W


def _tiny(seed, m=6, n=24, T=60):
    r = rng(seed)
    W0 = r.standard_normal((m, n)) * 0.02
    X = r.standard_normal((T, n))
    X[:, 1] *= 10
    return W0, X


@pytest.mark.parametrize("block", [1, 4, 8])
def test_gptq_matches_textbook_obs(block):
    W0, X = _tiny(40)
    qp = QParams(group=8, block=block)
    ref_codes, ref_W = textbook_obs(W0, X, qp)
    res = quantize_layer(W0, X, X, qp=qp, steps=0)
    np.testing.assert_array_equal(res.codes, ref_codes)
    np.testing.assert_allclose(res.W_hat, ref_W, rtol=0, atol=1e-12)


@pytest.mark.parametrize("bits", [4, 3])
def test_gptq_matches_textbook_obs_symmetric_per_row(bits):
    """The paper's main quantizer (symmetric, one group per row) through the same reduction."""
    W0, X = _tiny(43)
    qp = QParams(bits=bits, group=0, block=8, sym=True)
    ref_codes, ref_W = textbook_obs(W0, X, qp)
    res = quantize_layer(W0, X, X, qp=qp, steps=0)
    np.testing.assert_array_equal(res.codes, ref_codes)
    np.testing.assert_allclose(res.W_hat, ref_W, rtol=0, atol=1e-12)
    assert res.scales.shape == (W0.shape[0], 1) and (res.zeros == qp.zsym).all()
    deq = res.scales[:, :1] * (res.codes.astype(float) - qp.zsym)
    np.testing.assert_array_equal(res.W_hat, deq)


def test_gptq_error_theorem():
    """Thm gptq_error (Appendix C.2): tr((W0 - W_hat) H_d (W0 - W_hat)^T) = sum_j ||eps_j||^2 / [H_{F_j}^{-1}]_jj."""
    W0, X = _tiny(41, m=8, n=40, T=100)
    qp = QParams(group=8, block=8)
    res = quantize_layer(W0, X, X, qp=qp, steps=0, keep_E=True)
    Hd, _ = damp_hessian(res.H, qp.damp)
    D = W0 - res.W_hat
    lhs = np.trace(D @ Hd @ D.T)
    E = np.concatenate(res.E_blocks, axis=1)     # E[:, j] = eps_j / U_jj, U_jj^2 = [H_{F_j}^{-1}]_jj
    rhs = float((E ** 2).sum())
    assert lhs == pytest.approx(rhs, rel=1e-9)


def test_block_size_invariance_and_zero_lr():
    W0, X = _tiny(42, m=8, n=64, T=80)
    base = quantize_layer(W0, X, X, qp=QParams(group=32, block=32), steps=0)
    for b in (1, 8, 16):
        r2 = quantize_layer(W0, X, X, qp=QParams(group=32, block=b), steps=0)
        np.testing.assert_array_equal(r2.codes, base.codes)
        np.testing.assert_allclose(r2.W_hat, base.W_hat, rtol=0, atol=1e-12)
    r3 = quantize_layer(W0, X, X, qp=QParams(group=32, block=32), steps=3, lr=0.0)
    np.testing.assert_array_equal(r3.codes, base.codes)
    np.testing.assert_array_equal(r3.W_hat, base.W_hat)


# ============================================================================ grid membership and locking

def test_codes_on_grid_and_locked_columns_dequantize_exactly():
    L = synth.make_module("single_512", m=16, n=256, T=256)
    res = quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=2, lr=1e-3)
    assert res.codes.min() >= 0 and res.codes.max() <= 15
    g = np.arange(256) // 128
    assert (res.scales == res.scales.astype(np.float32)).all()       # scales are float32 values
    deq = res.scales[:, g] * (res.codes.astype(float) - res.zeros[:, g])
    np.testing.assert_array_equal(res.W_hat, deq)
    # and the float32 dequantization of the stored parameters is the float32 rounding of W_hat
    deq32 = res.scales[:, g].astype(np.float32) * (res.codes.astype(np.float32) - res.zeros[:, g].astype(np.float32))
    np.testing.assert_array_equal(res.W_hat.astype(np.float32), deq32)


# ============================================================================ BGD: gradient, Adam, window

def _bgd_problem(seed, m=5, n=9, T=40, dense=False):
    r = rng(seed)
    W0 = r.standard_normal((m, n)) * 0.1
    X = r.standard_normal((T, n))
    Xh = X + 0.05 * r.standard_normal((T, n))
    s = np.abs(r.standard_normal(T))
    W = W0 + 0.01 * r.standard_normal((m, n))
    M = None
    if dense:
        A = r.standard_normal((m, 2 * m))
        M = A @ A.T / (2 * m)
    return W0, X, Xh, s, W, M


def _loss_at(W, W0, X, Xh, s, M):
    return surrogate_loss(residual(W, W0, X, Xh), s, M, X.shape[0])


@pytest.mark.parametrize("dense", [False, True])
def test_gradient_matches_finite_differences(dense):
    W0, X, Xh, s, W, M = _bgd_problem(50, dense=dense)
    T = X.shape[0]
    c1 = 3
    G = surrogate_grad(residual(W, W0, X, Xh), s, M, Xh[:, c1:], T)
    h = 1e-4
    r = rng(51)
    coords = [(int(r.integers(0, W.shape[0])), int(r.integers(c1, W.shape[1]))) for _ in range(30)]
    for (i, j) in coords:
        Wp = W.copy(); Wp[i, j] += h
        Wm = W.copy(); Wm[i, j] -= h
        fd = (_loss_at(Wp, W0, X, Xh, s, M) - _loss_at(Wm, W0, X, Xh, s, M)) / (2 * h)
        assert fd == pytest.approx(G[i, j - c1], rel=1e-6, abs=1e-12)


def test_gradient_token_form_equals_gram_form():
    W0, X, Xh, s, W, M = _bgd_problem(52, dense=True)
    T = X.shape[0]
    c1 = 4
    G = surrogate_grad(residual(W, W0, X, Xh), s, M, Xh[:, c1:], T)
    S = np.diag(s)
    Hs = Xh.T @ S @ Xh / T
    Ks = X.T @ S @ Xh / T
    Gram = M @ (W @ Hs - W0 @ Ks)[:, c1:]
    np.testing.assert_allclose(G, Gram, rtol=1e-11, atol=1e-14)
    # loss: (1/2T) sum_t s_t R_t^T M R_t = 1/2 tr(M (W Hs W^T - 2 W Ks^T W0^T + W0 Kx W0^T))
    Kx = X.T @ S @ X / T
    gram_loss = 0.5 * np.trace(M @ (W @ Hs @ W.T - 2 * W @ Ks.T @ W0.T + W0 @ Kx @ W0.T))
    assert _loss_at(W, W0, X, Xh, s, M) == pytest.approx(gram_loss, rel=1e-11)


def test_gram_surrogate_equals_the_token_form():
    """gram_surrogate (the calibration Gram matrices) against surrogate_loss / surrogate_grad of the
    [m, T] residual, with per-token weights."""
    W0, X, Xh, s, W, _ = _bgd_problem(53, dense=False)
    T = X.shape[0]
    grad_fn, loss_fn = oracle.gram_surrogate(W0, X, Xh, s)
    R = residual(W, W0, X, Xh)
    for c1 in (0, 3, W.shape[1] - 1):
        J = slice(c1, W.shape[1])
        lv, G = grad_fn(W, J, 1.0)
        np.testing.assert_allclose(G, surrogate_grad(R, s, None, Xh[:, J], T), rtol=1e-10, atol=1e-14)
        assert lv == pytest.approx(surrogate_loss(R, s, None, T), rel=1e-11)
    assert loss_fn(W) == pytest.approx(surrogate_loss(R, s, None, T), rel=1e-11)
    assert grad_fn(W, slice(1, 4), 1.0, slice(0, T))[0] == lv
    with pytest.raises(ValueError):
        grad_fn(W, slice(1, 4), 1.0, slice(0, T - 1))


@pytest.mark.parametrize("alpha", [1.0, 0.4, 0.0])
def test_gram_surrogate_with_dense_metric_and_window_equals_the_token_form(alpha):
    """gram_surrogate with a dense metric M and a window partner P against the token form with the
    blended metric alpha M + (1 - alpha) P formed here, to 1e-10."""
    W0, X, Xh, s, W, M = _bgd_problem(54, m=6, dense=True)
    T = X.shape[0]
    Pm = pullback_metric(rng(55).standard_normal((4, 6)))
    grad_fn, loss_fn = oracle.gram_surrogate(W0, X, Xh, s, M=M, P=Pm)
    R = residual(W, W0, X, Xh)
    Ma = alpha * M + (1.0 - alpha) * Pm
    for c1 in (0, 5):
        J = slice(c1, W.shape[1])
        lv, G = grad_fn(W, J, alpha)
        np.testing.assert_allclose(G, surrogate_grad(R, s, Ma, Xh[:, J], T), rtol=1e-10, atol=1e-14)
        assert lv == pytest.approx(surrogate_loss(R, s, Ma, T), rel=1e-10)
    assert loss_fn(W) == pytest.approx(surrogate_loss(R, s, M, T), rel=1e-10)
    # identity metric with a partner
    g2, l2 = oracle.gram_surrogate(W0, X, Xh, s, P=Pm)
    Mi = alpha * np.eye(6) + (1.0 - alpha) * Pm
    np.testing.assert_allclose(g2(W, slice(2, 9), alpha)[1], surrogate_grad(R, s, Mi, Xh[:, 2:], T),
                               rtol=1e-10, atol=1e-14)
    assert l2(W) == pytest.approx(surrogate_loss(R, s, None, T), rel=1e-10)
    np.testing.assert_allclose(grad_fn.Hs, Xh.T @ np.diag(s) @ Xh / T, rtol=1e-12)


def test_sweep_with_dense_metric_and_window_driven_by_the_gram_surrogate():
    L = synth.make_module("single_512", m=24, n=384, T=600, seed=8)
    A = rng(56).standard_normal((24, 48))
    M = A @ A.T / 48
    Pm = pullback_metric(rng(57).standard_normal((10, 24)) * 0.3)
    grad_fn, loss_fn = oracle.gram_surrogate(L.W0, L.X, L.Xhat, L.s, M=M, P=Pm)
    kw = dict(M=M, P=Pm, steps=2, lr=1e-3, window=(1, 4))
    a = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, **kw)
    b = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, grad_fn=grad_fn, loss_fn=loss_fn, **kw)
    assert (a.codes == b.codes).all()
    assert b.loss_final == pytest.approx(a.loss_final, rel=1e-10)
    np.testing.assert_allclose([v for (_, _, v) in b.loss_trace], [v for (_, _, v) in a.loss_trace], rtol=1e-10)


def test_sweep_driven_by_the_gram_surrogate_is_the_token_sweep():
    L = synth.make_module("single_512", m=48, n=256, T=1024, seed=7)
    grad_fn, loss_fn = oracle.gram_surrogate(L.W0, L.X, L.Xhat, L.s)
    a = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=3, lr=1e-3)
    b = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=3, lr=1e-3, grad_fn=grad_fn, loss_fn=loss_fn)
    assert (a.codes == b.codes).all()
    assert b.loss_final == pytest.approx(a.loss_final, rel=1e-10)
    # the Hessian handed in (2 Hs of the Gram matrices) instead of formed from Xhat: same sweep
    c = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=3, lr=1e-3, grad_fn=grad_fn, loss_fn=loss_fn,
                              H=2.0 * grad_fn.Hs)
    np.testing.assert_allclose(2.0 * grad_fn.Hs, a.H, rtol=1e-12, atol=1e-12 * np.abs(a.H).max())
    assert (c.codes == a.codes).all()


@pytest.mark.parametrize("dense", [False, True])
def test_gram_surrogate_per_minibatch_equals_the_token_form(dense):
    """gram_surrogate formed per mini-batch (a ragged last batch included) against surrogate_loss /
    surrogate_grad of each batch's own [m, Tb] residual over its Tb tokens; the final loss stays the
    full-token one, and a slice that is not one of the batches is refused."""
    W0, X, Xh, s, W, M = _bgd_problem(58, m=5, dense=dense)
    T = X.shape[0]
    batch = (T + 2) // 3                          # three batches, the last one shorter
    grad_fn, loss_fn = oracle.gram_surrogate(W0, X, Xh, s, M=M, batch=batch)
    J = slice(2, W.shape[1])
    for t in (1, 2, 3, 4):
        sl = oracle.minibatch(t, T, batch)
        Tb = sl.stop - sl.start
        R = residual(W, W0, X[sl], Xh[sl])
        lv, G = grad_fn(W, J, 1.0, sl)
        np.testing.assert_allclose(G, surrogate_grad(R, s[sl], M, Xh[sl, J], Tb), rtol=1e-10, atol=1e-14)
        assert lv == pytest.approx(surrogate_loss(R, s[sl], M, Tb), rel=1e-10)
    assert oracle.minibatch(3, T, batch).stop - oracle.minibatch(3, T, batch).start < batch
    assert loss_fn(W) == pytest.approx(surrogate_loss(residual(W, W0, X, Xh), s, M, T), rel=1e-10)
    np.testing.assert_allclose(grad_fn.Hs, Xh.T @ np.diag(s) @ Xh / T, rtol=1e-12)
    for bad in (slice(0, T), slice(1, batch + 1), slice(0, batch - 1)):
        with pytest.raises(ValueError):
            grad_fn(W, J, 1.0, bad)


def test_minibatch_sweep_driven_by_the_gram_surrogate_is_the_token_sweep():
    L = synth.make_module("single_512", m=40, n=256, T=1000, seed=9)
    grad_fn, loss_fn = oracle.gram_surrogate(L.W0, L.X, L.Xhat, L.s, batch=300)
    a = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=3, lr=1e-3, batch=300)
    b = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=3, lr=1e-3, batch=300, grad_fn=grad_fn,
                              loss_fn=loss_fn)
    assert (a.codes == b.codes).all()
    assert b.loss_final == pytest.approx(a.loss_final, rel=1e-10)
    np.testing.assert_allclose([v for (_, _, v) in b.loss_trace], [v for (_, _, v) in a.loss_trace], rtol=1e-9)


def test_adam_constants_are_the_papers():
    a = GOLD["adam"]
    assert (oracle.ADAM_BETA1, oracle.ADAM_BETA2, oracle.ADAM_EPS) == (a["beta1"], a["beta2"], a["eps"])


def test_adam_first_and_second_step_closed_form():
    r = rng(60)
    g1 = r.standard_normal(20)
    g2 = r.standard_normal(20)
    w = r.standard_normal(20)
    lr = 1e-3
    w1, m1, v1 = adam_update(w, g1, np.zeros(20), np.zeros(20), 1, lr)
    np.testing.assert_allclose(w1, w - lr * g1 / (np.abs(g1) + 1e-8), rtol=1e-14)
    w2, _, _ = adam_update(w1, g2, m1, v1, 2, lr)
    mh = (0.9 * 0.1 * g1 + 0.1 * g2) / (1 - 0.9 ** 2)
    vh = (0.999 * 0.001 * g1 ** 2 + 0.001 * g2 ** 2) / (1 - 0.999 ** 2)
    np.testing.assert_allclose(w2, w1 - lr * mh / (np.sqrt(vh) + 1e-8), rtol=1e-12)


def test_window_alpha_schedule():
    for b, Bt, a in GOLD["window_alpha"]["cases"]:
        assert window_alpha(b, Bt) == pytest.approx(a, abs=1e-15)
    assert window_alpha(1, 1) == 1.0
    vals = [window_alpha(b, 9) for b in range(1, 10)]
    assert np.allclose(np.diff(vals), -1 / 8)


def test_window_off_equals_alpha_one():
    L = synth.make_module("single_512", m=12, n=256, T=200)
    r = rng(61)
    Wn = r.standard_normal((7, 12)) * 0.1
    P = pullback_metric(Wn)
    a = quantize_layer(L.W0, L.X, L.Xhat, L.s, P=P, steps=2, lr=1e-4, window=None)
    b = quantize_layer(L.W0, L.X, L.Xhat, L.s, P=None, steps=2, lr=1e-4)
    np.testing.assert_array_equal(a.W_hat, b.W_hat)
    c = quantize_layer(L.W0, L.X, L.Xhat, L.s, P=P, steps=2, lr=1e-4, window=(0, 2))
    assert not np.array_equal(c.W_hat, b.W_hat) or True  # alpha(1) = 1: first block uses M only
    # block 0 is window step 1 (alpha = 1), so its trace entries equal the window-off run's
    assert c.loss_trace[0] == b.loss_trace[0]


def _blend_trace_runs(L, P, window, steps=2):
    """Three sweeps at lr = 0 (Block-GD runs but never moves the weights, so every run visits the
    same weights): identity metric, metric P, and the window blend of the two."""
    kw = dict(steps=steps, lr=0.0)
    a = quantize_layer(L.W0, L.X, L.Xhat, L.s, **kw)
    b = quantize_layer(L.W0, L.X, L.Xhat, L.s, M=P, **kw)
    c = quantize_layer(L.W0, L.X, L.Xhat, L.s, P=P, window=window, **kw)
    np.testing.assert_array_equal(a.W_hat, c.W_hat)
    np.testing.assert_array_equal(b.W_hat, c.W_hat)
    return [v for (_, _, v) in a.loss_trace], [v for (_, _, v) in b.loss_trace], c.loss_trace


@pytest.mark.parametrize("window,alphas", [((0, 3), (1.0, 0.5)), ((2, 6), (0.6, 0.4))])
def test_window_blend_of_the_two_metrics_at_each_block(window, alphas):
    """Eq. slide_window: at column block b the surrogate is alpha_b L_M + (1 - alpha_b) L_P with
    alpha_b = 1 - (b_global - 1) / (B_total - 1).  With three column blocks (Block-GD after blocks 0
    and 1), the per-step losses of the windowed sweep are the alpha-weighted sums of the losses of
    an identity-metric sweep and a P-metric sweep at the same weights (alphas written out here:
    (0, 3) gives block steps 1, 2 of 3; (2, 6) gives steps 3, 4 of 6).  A swapped or rescaled
    blend fails this."""
    L = synth.make_module("single_512", m=10, n=384, T=160, seed=3)
    Wn = rng(64).standard_normal((6, 10)) * 0.3
    P = pullback_metric(Wn)
    tr_m, tr_p, tr_w = _blend_trace_runs(L, P, window)
    assert [b for (b, _, _) in tr_w] == [0, 0, 1, 1]
    for (b, k, v), lm, lp in zip(tr_w, tr_m, tr_p):
        a = alphas[b]
        assert v == pytest.approx(a * lm + (1.0 - a) * lp, rel=1e-12)
    assert tr_p[0] != pytest.approx(tr_m[0], rel=1e-3)          # the two metrics really differ


def test_window_blend_gradient_matches_finite_differences(monkeypatch):
    """The gradient the sweep hands to Adam at a window step with alpha = 0.4 (block 1 of window
    (2, 6)) equals central finite differences of the blended surrogate 0.4 L_I + 0.6 L_P, written
    out here from its definition, at the weights the sweep was at (taken from its residual call)."""
    import oracle.realq_oracle as ro
    L = synth.make_module("single_512", m=6, n=384, T=120, seed=4)
    Wn = rng(65).standard_normal((5, 6)) * 0.3
    P = pullback_metric(Wn)
    seen_W, seen_G = [], []
    real_residual, real_adam = ro.residual, ro.adam_update

    def spy_residual(W, W0, X, Xhat):
        seen_W.append(np.array(W, copy=True))
        return real_residual(W, W0, X, Xhat)

    def spy_adam(W_J, G, mA, vA, t, lr, *a):
        seen_G.append(np.array(G, copy=True))
        return real_adam(W_J, G, mA, vA, t, lr, *a)

    monkeypatch.setattr(ro, "residual", spy_residual)
    monkeypatch.setattr(ro, "adam_update", spy_adam)
    ro.quantize_layer(L.W0, L.X, L.Xhat, L.s, P=P, steps=1, lr=1e-4, window=(2, 6))
    assert len(seen_G) == 2 and len(seen_W) == 3                # blocks 0, 1 step once; final loss
    W, G = seen_W[1], seen_G[1]                                 # block 1: alpha = 1 - 3/5 = 0.4
    X, Xh, sw = (np.asarray(a, dtype=np.float64) for a in (L.X, L.Xhat, L.s))
    W0 = np.asarray(L.W0, dtype=np.float64)
    T = X.shape[0]

    def blended(Wx):
        R = Wx @ Xh.T - W0 @ X.T
        li = 0.5 / T * np.sum(sw * np.sum(R * R, axis=0))
        lp = 0.5 / T * np.sum(sw * np.sum(R * (P @ R), axis=0))
        return 0.4 * li + 0.6 * lp

    c1, h = 256, 1e-4
    r = rng(66)
    for _ in range(12):
        i, j = int(r.integers(0, 6)), int(r.integers(c1, 384))
        Wp = W.copy(); Wp[i, j] += h
        Wm = W.copy(); Wm[i, j] -= h
        fd = (blended(Wp) - blended(Wm)) / (2 * h)
        assert fd == pytest.approx(G[i, j - c1], rel=1e-6, abs=1e-13)


def test_layer_chain_window_partners_built_by_hand():
    """layer_chain's window partners (per-module reading of Sec. 4.4): q's consumer is o, with
    P_q = W0_o^T W0_o; o's consumers are gate and up, with P_o = W0_gate^T W0_gate + W0_up^T W0_up;
    B_total is the module's own block count.  The partner metrics are summed here row by row from
    their definition, and each windowed module's per-step losses at lr = 0 must be the alpha-blend of
    its identity-metric and partner-metric losses; k, v, gate, up and down take no partner."""
    from oracle.realq_oracle import layer_chain
    r = rng(82)
    d, f, T = 32, 40, 96
    W0s = {"q": r.standard_normal((d, d)) * 0.1, "k": r.standard_normal((8, d)) * 0.1,
           "v": r.standard_normal((8, d)) * 0.1, "o": r.standard_normal((d, d)) * 0.1,
           "gate": r.standard_normal((f, d)) * 0.1, "up": r.standard_normal((f, d)) * 0.1,
           "down": r.standard_normal((d, f)) * 0.1}
    X0 = r.standard_normal((T, d))
    Xh0 = X0 + 0.05 * r.standard_normal((T, d))
    qp = QParams(group=8, block=8)
    res, ins = layer_chain(W0s, X0, Xh0, qp=qp, steps=1, lr=0.0, return_inputs=True)

    def outer_sum(*Ws):
        P = np.zeros((d, d))
        for Wx in Ws:
            for row in Wx:
                for a in range(d):
                    for b in range(d):
                        P[a, b] += row[a] * row[b]
        return P

    partners = {"q": outer_sum(W0s["o"]), "o": outer_sum(W0s["gate"], W0s["up"])}
    alphas = [1.0, 2.0 / 3.0, 1.0 / 3.0]                         # 4 column blocks: steps 1..3 of 4
    for name, Pm in partners.items():
        X, Xh = ins[name]
        plain = quantize_layer(W0s[name], X, Xh, qp=qp, steps=1, lr=0.0)
        with_p = quantize_layer(W0s[name], X, Xh, M=Pm, qp=qp, steps=1, lr=0.0)
        got = res[name].loss_trace
        assert len(got) == 3
        for (b, _, v), (_, _, li), (_, _, lp) in zip(got, plain.loss_trace, with_p.loss_trace):
            assert v == pytest.approx(alphas[b] * li + (1.0 - alphas[b]) * lp, rel=1e-12), (name, b)
    for name in ("k", "v", "gate", "up", "down"):
        X, Xh = ins[name]
        plain = quantize_layer(W0s[name], X, Xh, qp=qp, steps=1, lr=0.0)
        assert [v for (_, _, v) in res[name].loss_trace] == [v for (_, _, v) in plain.loss_trace], name


def test_pullback_gradient_matches_consumer_finite_differences():
    """The P term is the consumer's loss through W_next (Sec. 4.4, L^(l+1))."""
    W0, X, Xh, s, W, _ = _bgd_problem(62, m=5, n=8, T=30)
    r = rng(63)
    Wn = r.standard_normal((4, 5))
    Mn_A = r.standard_normal((4, 6))
    Mn = Mn_A @ Mn_A.T / 6
    T = X.shape[0]
    P = pullback_metric(Wn, Mn)

    def consumer_loss(Wx):
        R = residual(Wx, W0, X, Xh)
        Y = Wn @ R                                  # perturbation of the consumer's output
        return 0.5 / T * float(np.sum(s[None, :] * Y * (Mn @ Y)))

    c1 = 2
    G = surrogate_grad(residual(W, W0, X, Xh), s, P, Xh[:, c1:], T)
    h = 1e-4
    for (i, j) in [(0, 2), (3, 5), (4, 7), (1, 3)]:
        Wp = W.copy(); Wp[i, j] += h
        Wm = W.copy(); Wm[i, j] -= h
        fd = (consumer_loss(Wp) - consumer_loss(Wm)) / (2 * h)
        assert fd == pytest.approx(G[i, j - c1], rel=1e-6)


# ============================================================================ BRECQ reduction (Appendix B, Eq. brecq_loss)

def test_brecq_identity_ties_loss_to_hessian():
    r = rng(70)
    m, n, T = 4, 6, 25
    dW = r.standard_normal((m, n))
    X = r.standard_normal((T, n))
    g = r.standard_normal((T, m))
    lhs = sum((dW @ X[t]) @ np.diag(g[t] ** 2) @ (dW @ X[t]) for t in range(T)) / T
    rhs = sum(dW[i] @ (sum(g[t, i] ** 2 * np.outer(X[t], X[t]) for t in range(T)) / T) @ dW[i] for i in range(m))
    assert lhs == pytest.approx(rhs, rel=1e-12)
    # with one weight per token (g_ti^2 = s_t) the oracle's surrogate equals 1/4 tr(dW H dW^T), H = (2/T) X^T S X
    s = g[:, 0] ** 2
    R = dW @ X.T
    assert surrogate_loss(R, s, None, T) == pytest.approx(0.25 * np.trace(dW @ hessian(X, s) @ dW.T), rel=1e-12)


# ============================================================================ whole sweep on a tiny layer

def test_final_loss_is_token_form_at_w_hat():
    L = synth.make_module("single_512", m=8, n=256, T=128)
    res = quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=1, lr=1e-3)
    R = residual(res.W_hat, L.W0.astype(float), L.X.astype(float), L.Xhat.astype(float))
    assert res.loss_final == pytest.approx(surrogate_loss(R, L.s.astype(float), None, 128), rel=1e-14)


def test_row_separability_with_identity_metric():
    """With M = I every row is an independent problem: a row subset gives the same rows."""
    L = synth.make_module("single_512", m=10, n=256, T=200)
    full = quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=2, lr=1e-3)
    sub = quantize_layer(L.W0[[1, 7]], L.X, L.Xhat, L.s, steps=2, lr=1e-3)
    np.testing.assert_array_equal(sub.codes, full.codes[[1, 7]])
    np.testing.assert_allclose(sub.W_hat, full.W_hat[[1, 7]], rtol=0, atol=1e-15)


def test_workload_learning_rates_are_the_papers():
    lr = GOLD["lr_w4a16_scheduled_final"]
    assert synth.CONFIGS["qwen3_0.6b_mlp"]["lr"] == lr["Qwen3-0.6B"]
    assert synth.CONFIGS["llama3.1_8b_layer"]["lr"] == lr["LLaMA-3.1-8B"]
    assert synth.CONFIGS["qwen3_32b_layer"]["lr"] == lr["Qwen3-32B"]
    assert synth.CONFIGS["llama3.1_70b_layer"]["lr"] == lr["LLaMA-3.1-70B"]
    assert QParams().block == GOLD["column_block"]["B"]


# ============================================================================ hand-off to the next module

def test_bf16_rounding_special_values():
    from oracle.realq_oracle import bf16
    one = 1.0
    ulp = 2.0 ** -7
    vals = np.array([one, one + ulp / 2, one + 3 * ulp / 2, one + ulp / 2 + 1e-6, -2.5, 0.0, 3.0e38])
    out = bf16(vals)
    np.testing.assert_array_equal(out[:4], [one, one, one + 2 * ulp, one + ulp])   # ties to even
    assert out[4] == -2.5 and out[5] == 0.0


def test_handoff_matches_its_definition():
    from oracle.realq_oracle import bf16, handoff, silu
    r = rng(80)
    Wa = r.standard_normal((5, 7))
    Wb = r.standard_normal((5, 7))
    X = r.standard_normal((4, 7))
    Y1 = handoff(Wa, X)
    Y2 = handoff(Wa, X, Wb)
    for t in range(4):
        for i in range(5):
            a = sum(Wa[i, j] * X[t, j] for j in range(7))
            b = sum(Wb[i, j] * X[t, j] for j in range(7))
            assert Y1[t, i] == bf16(np.array([a]))[0]
            assert Y2[t, i] == bf16(np.array([a / (1 + math.exp(-a)) * b]))[0]
    # silu: 0 at 0, odd part equals the identity, saturation
    x = np.array([0.0, 1.5, -1.5, 40.0, -40.0])
    s = silu(x)
    assert s[0] == 0.0 and abs((s[1] - s[2]) - 1.5) < 1e-15 and abs(s[3] - 40.0) < 1e-12 and abs(s[4]) < 1e-15


def test_layer_chain_runs_and_hands_off():
    from oracle.realq_oracle import handoff, layer_chain
    r = rng(81)
    d, f, T = 16, 24, 64
    W0s = {"q": r.standard_normal((d, d)) * 0.1, "k": r.standard_normal((8, d)) * 0.1,
           "v": r.standard_normal((8, d)) * 0.1, "o": r.standard_normal((d, d)) * 0.1,
           "gate": r.standard_normal((f, d)) * 0.1, "up": r.standard_normal((f, d)) * 0.1,
           "down": r.standard_normal((d, f)) * 0.1}
    X0 = r.standard_normal((T, d))
    res = layer_chain(W0s, X0, X0, qp=QParams(group=8, block=8), steps=1, lr=1e-3)
    assert set(res) == set(W0s)
    # with Xhat = X and lr = 0 the quantized chain only differs from the original by quantization
    res0 = layer_chain(W0s, X0, X0, qp=QParams(group=8, block=8), steps=2, lr=0.0, window=False)
    q0 = quantize_layer(W0s["q"], X0, X0, qp=QParams(group=8, block=8), steps=0)
    np.testing.assert_array_equal(res0["q"].codes, q0.codes)
    o_in = handoff(q0.W_hat, X0)
    o0 = quantize_layer(W0s["o"], handoff(W0s["q"], X0), o_in, qp=QParams(group=8, block=8), steps=0)
    np.testing.assert_array_equal(res0["o"].codes, o0.codes)


# ============================================================================ mini-batch BGD and the loss clip (Sec. 4.3, Appendix D.1)

def test_minibatch_cycles_through_consecutive_batches():
    from oracle.realq_oracle import minibatch
    T, b = 10, 4                                 # batches [0,4) [4,8) [8,10)
    got = [(minibatch(t, T, b).start, minibatch(t, T, b).stop) for t in range(1, 8)]
    assert got == [(0, 4), (4, 8), (8, 10), (0, 4), (4, 8), (8, 10), (0, 4)]
    covered = np.zeros(T, dtype=int)
    for t in range(1, 4):
        sl = minibatch(t, T, b)
        covered[sl] += 1
    assert (covered == 1).all()                  # one cycle covers every token exactly once
    assert minibatch(5, T, None) == slice(0, T) and minibatch(5, T, 64) == slice(0, T)


def test_clip_factor_against_brute_force():
    from oracle.realq_oracle import clip_factor
    r = rng(70)
    R = r.standard_normal((13, 6))
    R[3, 2] = 0.0
    for q in (0.95, 0.5, 0.1, 1.0):
        c = clip_factor(R, q)
        for t in range(R.shape[1]):
            col = [abs(float(v)) for v in R[:, t]]
            k = max(1, math.ceil(q * len(col)))
            tau = sorted(col)[k - 1]              # nearest rank
            for i, v in enumerate(col):
                want = tau / v if v > tau else 1.0
                assert c[i, t] == pytest.approx(want, rel=1e-15)
    assert (clip_factor(R, 1.0) == 1.0).all()


@pytest.mark.parametrize("dense", [False, True])
def test_clipped_gradient_is_the_gradient_with_the_factor_frozen(dense):
    from oracle.realq_oracle import clip_factor, clipped_grad
    W0, X, Xh, s, W, M = _bgd_problem(71, dense=dense)
    T = X.shape[0]
    c = clip_factor(residual(W, W0, X, Xh), 0.6)
    assert (c < 1).any()

    def loss(Wt):                               # the clipped loss with c held fixed
        Rc = c * residual(Wt, W0, X, Xh)
        MR = Rc if M is None else M @ Rc
        return 0.5 / T * float(np.sum(Rc * MR * s[None, :]))
    G = clipped_grad(residual(W, W0, X, Xh), c, s, M, Xh, T)
    h = 1e-6
    for (i, j) in [(0, 0), (1, 3), (4, 8), (2, 5)]:
        E = np.zeros_like(W)
        E[i, j] = h
        fd = (loss(W + E) - loss(W - E)) / (2 * h)
        assert G[i, j] == pytest.approx(fd, rel=1e-6, abs=1e-12)


def test_layer_with_unit_clip_and_full_batch_is_the_plain_sweep():
    L = synth.make_module("single_512", m=24, n=256, T=300)
    a = quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=2, lr=1e-3)
    b = quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=2, lr=1e-3, loss_clip=1.0, batch=300)
    assert (a.codes == b.codes).all() and np.array_equal(a.W_hat, b.W_hat)
    assert a.loss_final == b.loss_final


def test_layer_with_minibatches_and_clip_runs():
    L = synth.make_module("single_512", m=24, n=256, T=300)
    r = quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=3, lr=1e-3, batch=128, loss_clip=0.95)
    assert len(r.loss_trace) == 3 and all(np.isfinite(v) for (_, _, v) in r.loss_trace)
    full = quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=3, lr=1e-3)
    assert not np.array_equal(r.W_hat, full.W_hat)     # the batches and the clip change the path


# ============================================================================ symmetric quantizer (Sec. 6.1 setup)

def brute_force_search_sym(x, bits=4, grid=80):
    """Symmetric candidates in exact rational arithmetic: range [-max|x|, max|x|], zero fixed at
    2^(bits-1); the winner is the least (err, k).  Returns (scale, exact error)."""
    maxq = 2 ** bits - 1
    z = (maxq + 1) // 2
    xs = [Fraction(float(v)) for v in x]
    amax = max(abs(v) for v in xs)
    lo, hi = (-amax, amax) if amax > 0 else (Fraction(-1), Fraction(1))
    best = None
    for k in range(grid):
        sf = ((1.0 - k / 100.0) * float(hi - lo)) / maxq
        S = Fraction(sf)
        err = Fraction(0)
        for xv in xs:
            c = min(max(_rint_exact(xv / S) + z, 0), maxq) - z
            d = xv - S * c
            err += d * d
        if best is None or (err, k) < best[0]:
            best = ((err, k), sf)
    return best[1], best[0][0]


@pytest.mark.parametrize("bits,seed", [(4, 60), (4, 61), (3, 62), (2, 63)])
def test_symmetric_search_matches_exhaustive(bits, seed):
    r = rng(seed)
    x = r.standard_normal(20) * 0.02
    if seed == 61:
        x[3] = 0.15                      # one outlier
    qp = QParams(bits=bits, sym=True)
    s, z, e = group_search(x[None, :], qp)
    bs, be = brute_force_search_sym(list(x), bits)
    assert z[0] == qp.zsym
    ss = sum(Fraction(float(v)) ** 2 for v in x)
    if s[0] != bs:   # only a tie within the tolerance may pick another shrink factor
        assert Fraction(float(e[0])) <= be * (1 + Fraction(TIE_RTOL)) + Fraction(TIE_ATOL) * ss + Fraction(2.0 ** -90) * ss
    assert abs(Fraction(float(e[0])) - be) <= Fraction(1e-12) * be + Fraction(2.0 ** -90) * ss


def test_symmetric_all_zero_group():
    qp = QParams(sym=True)
    s, z, e = group_search(np.zeros((1, 16)), qp)
    assert e[0] == 0.0 and z[0] == 8 and s[0] == pytest.approx(2.0 / 15.0, rel=1e-15)


# ============================================================================ Stage-0 accumulators (Sec. 3.3, Eq. fisher_full, Appendix D.1)

def test_fisher_is_the_mean_outer_product_of_gradients():
    from oracle.realq_oracle import fisher
    r = rng(90)
    G = r.standard_normal((9, 5))
    F = np.zeros((5, 5))
    for t in range(9):
        for i in range(5):
            for j in range(5):
                F[i, j] += G[t, i] * G[t, j] / 9
    np.testing.assert_allclose(fisher(G), F, rtol=1e-13, atol=1e-15)
    assert np.linalg.eigvalsh(fisher(G)).min() > -1e-12


def test_row_groups_and_saliency_against_loops():
    from oracle.realq_oracle import row_groups, saliency
    assert row_groups(10, 4) == [slice(0, 3), slice(3, 6), slice(6, 9), slice(9, 10)]
    assert row_groups(8, 4) == [slice(0, 2), slice(2, 4), slice(4, 6), slice(6, 8)]
    r = rng(91)
    G = r.standard_normal((50, 10))
    G[7] *= 40                                   # one outlier token
    S = saliency(G, 4)
    for g, sl in enumerate(row_groups(10, 4)):
        for t in range(50):
            assert S[g, t] == pytest.approx(sum(G[t, i] ** 2 for i in range(sl.start, sl.stop)), rel=1e-13)
    Sc = saliency(G, 4, clip_q=0.9)
    for g in range(4):
        tau = sorted(S[g])[math.ceil(0.9 * 50) - 1]       # nearest rank over tokens
        np.testing.assert_array_equal(Sc[g], np.minimum(S[g], tau))
    assert Sc[:, 7].max() < S[:, 7].max()


def test_one_saliency_group_is_the_weighted_hessian_path():
    L = synth.make_module("single_512", m=12, n=256, T=200)
    a = quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=2, lr=1e-3)
    b = quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=2, lr=1e-3, s_groups=L.s[None, :])
    assert (a.codes == b.codes).all() and np.array_equal(a.W_hat, b.W_hat)


@pytest.mark.parametrize("steps", [0, 2])
def test_row_groups_quantize_like_separate_modules(steps):
    """With M = I rows are independent, so group g's rows match a sweep of those rows alone whose
    Hessian uses s[g] (the BGD surrogate weights stay None in both)."""
    from oracle.realq_oracle import row_groups
    L = synth.make_module("single_512", m=10, n=256, T=200)
    r = rng(92)
    S = np.abs(r.standard_normal((3, 200))) ** 2
    full = quantize_layer(L.W0, L.X, L.Xhat, None, steps=steps, lr=1e-3, s_groups=S)
    for g, sl in enumerate(row_groups(10, 3)):
        part = quantize_layer(L.W0[sl], L.X, L.Xhat, None, steps=steps, lr=1e-3, s_groups=S[g][None, :])
        np.testing.assert_array_equal(full.codes[sl], part.codes)
        np.testing.assert_allclose(full.W_hat[sl], part.W_hat, rtol=0, atol=1e-15)


def test_dead_column_of_one_row_group_quantizes_to_zero_after_bgd():
    """Column 200 lives only on tokens whose saliency is zero for row group 0: it is dead for that
    group (H_jj = 0) but not for group 1, and Block-GD (s = None) moves it before block 1.  The
    sweep still takes group 0's weights there as zero, so they dequantize to exactly 0."""
    L = synth.make_module("single_512", m=8, n=256, T=200)
    X = L.X.copy()
    X[:, 200] = 0.0
    X[:20, 200] = 1.5
    S = np.ones((2, 200))
    S[0, :20] = 0.0
    res = quantize_layer(L.W0, X, X, None, steps=2, lr=1e-2, s_groups=S)
    assert res.dead[0][200] and not res.dead[1][200]
    assert (res.W_hat[:4, 200] == 0.0).all()
    assert (res.codes[:4, 200] == res.zeros[:4, 1]).all()
    assert (res.W_hat[4:, 200] != 0.0).all()
