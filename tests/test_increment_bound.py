"""What the library's Block-GD increments rest on, checked on the oracle (not on the library):
one bias-corrected Adam step (Sec. 4.3; Adam constants of Appendix D.1) moves a weight by at most
lr (1 - b1) / sqrt((1 - b2)(1 - b1^2/b2)) whatever the gradient history (the history
g_i = (b2/b1)^(i - t) attains the finite-t form of the bound at step t), and a later step's loss
and gradient follow from the block's first step's and the weight change."""
import numpy as np
import pytest

from oracle.realq_oracle import adam_update


def _sup(b1, b2):
    return (1.0 - b1) / np.sqrt((1.0 - b2) * (1.0 - b1 * b1 / b2))


def _at(t, b1, b2):
    rho = b1 * b1 / b2
    return (1.0 - b1) / (1.0 - b1 ** t) * np.sqrt((1.0 - b2 ** t) / (1.0 - b2)) * np.sqrt((1.0 - rho ** t) / (1.0 - rho))


def _max_step(G, b1, b2, lr=1.0):
    """Largest |weight change| / lr over the steps of the gradient histories G [steps, k]."""
    w = np.zeros(G.shape[1])
    m = np.zeros_like(w)
    v = np.zeros_like(w)
    worst = 0.0
    for t in range(1, G.shape[0] + 1):
        w2, m, v = adam_update(w, G[t - 1], m, v, t, lr, b1=b1, b2=b2, eps=0.0)
        worst = max(worst, float(np.max(np.abs(w2 - w))) / lr)
        w = w2
    return worst


@pytest.mark.parametrize("b1,b2", [(0.9, 0.999), (0.5, 0.9), (0.95, 0.999), (0.0, 0.5)])
def test_adam_step_stays_within_the_bound(b1, b2):
    r = np.random.default_rng(3)
    steps, k = 1500, 64
    hist = [r.standard_normal((steps, k)),                                    # noise
            r.standard_t(1.5, (steps, k)),                                   # heavy tails
            np.where(np.arange(steps)[:, None] % 2, 1.0, -1.0) * np.ones((steps, k)),   # sign flips
            np.where(r.random((steps, k)) < 0.01, 1e4, 1e-6),                # rare bursts
            np.exp(np.minimum(np.arange(steps), 400)[:, None] * np.log(b2 / max(b1, 0.5)) * np.ones((1, k)))]  # growth
    for G in hist:
        assert _max_step(G, b1, b2) <= _sup(b1, b2) * (1 + 1e-9)


@pytest.mark.parametrize("t", [1, 2, 8, 200])
def test_the_bound_is_attained(t):
    b1, b2 = 0.9, 0.999
    G = ((b2 / b1) ** (np.arange(1, t + 1) - t))[:, None]
    w = np.zeros(1)
    m = np.zeros(1)
    v = np.zeros(1)
    for i in range(1, t + 1):
        w2, m, v = adam_update(w, G[i - 1], m, v, i, 1.0, b1=b1, b2=b2, eps=0.0)
        last = abs(float(w2[0] - w[0]))
        w = w2
    assert last == pytest.approx(_at(t, b1, b2), rel=1e-12)
    assert _at(t, b1, b2) <= _sup(b1, b2)
    # the finite-t form rises to the supremum: 7.2703 for the paper's constants
    assert _sup(b1, b2) == pytest.approx(7.2703, abs=1e-4)


def test_loss_and_gradient_of_a_later_step_from_the_first():
    """The identities a later Block-GD step of a column block uses (Sec. 4.3, surrogate of
    Eq. fisher_loss with per-token weights, identity metric): with Delta the change of the
    trailing weights since the block's first step and Q = Delta Xhat_J^T,
    L(W_k) = L(W_0) + <G(W_0), Delta> + sum_t s_t |Q_t|^2 / 2T and G(W_k) = G(W_0) + (Q o s) Xhat_J / T,
    checked on the oracle's loss and gradient in float64."""
    from oracle.realq_oracle import residual, surrogate_grad, surrogate_loss
    r = np.random.default_rng(5)
    m, n, T, c1 = 7, 40, 300, 16
    W0 = r.standard_normal((m, n))
    X = r.standard_normal((T, n))
    Xh = X + 0.01 * r.standard_normal((T, n))
    s = r.lognormal(0.0, 1.0, T)
    J = slice(c1, n)
    Wa = W0 + 0.05 * r.standard_normal((m, n))             # weights at the block's first step
    D = np.zeros((m, n))
    D[:, J] = 1e-3 * r.standard_normal((m, n - c1))        # the later step's change (trailing columns)
    Wb = Wa + D
    Ra, Rb = residual(Wa, W0, X, Xh), residual(Wb, W0, X, Xh)
    La, Lb = surrogate_loss(Ra, s, None, T), surrogate_loss(Rb, s, None, T)
    Ga, Gb = surrogate_grad(Ra, s, None, Xh[:, J], T), surrogate_grad(Rb, s, None, Xh[:, J], T)
    Q = D[:, J] @ Xh[:, J].T
    assert Lb == pytest.approx(La + np.sum(Ga * D[:, J]) + 0.5 / T * np.sum(s[None, :] * Q * Q), rel=1e-12)
    np.testing.assert_allclose(Gb, Ga + (Q * s[None, :]) @ Xh[:, J] / T, rtol=1e-10, atol=1e-14)
