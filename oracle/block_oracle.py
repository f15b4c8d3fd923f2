"""Float64 oracle of the block-level surrogate for the MLP half of a decoder block.

TEST INFRASTRUCTURE ONLY: imported by tests/, never by the product library.

The module-level sweep (realq_oracle.quantize_layer) evaluates the Block-GD surrogate at the
linear module's output.  The paper evaluates it at the transformer block's output
(Sec. 4.2, Eq. fisher_loss; Sec. 4.3: the gradient of the trailing columns comes from a
forward and backward pass through the current block) and blends in the next block's
objective over the column blocks of all modules of the block (Sec. 4.4, Eq. slide_window).
This module does that for a pre-norm SwiGLU MLP block

    u = bf16(rmsnorm(h) * gamma),  a = u Wg^T,  b = u Wu^T,  z = bf16(silu(a) * b),
    y = h + bf16(z Wd^T),

whose three linear modules (gate, up, down) are quantized in that order (Alg. 1) with
Block-GD on the surrogate

    L = (1/2T) sum_t (y_t - y*_t)^T F (y_t - y*_t),

y* the full-precision block on the full-precision input X, y the partially quantized block on
the input Xhat that the quantized model feeds it.  Readings (the paper gives the objective,
not the block's arithmetic): the block computes in bf16 activations, rounded where the formula
above writes bf16; the backward treats those roundings as the identity (a cast's gradient);
the residual stream y stays unrounded; the sliding window's partner is the same MLP block
structure with its own weights and Fisher applied to y (and y*), so that
L_slide = alpha L + (1 - alpha) L_next with alpha over b_global = the column blocks of gate,
then up, then down (Eq. slide_window, B_total = all three modules' column blocks).  Attention
is not part of this block.

Pins: every backward here is checked against central finite differences of the unrounded
forward (rnd=False), and the down projection's gradient reduces to the module-level surrogate
gradient with M = F (tests/test_oracle_pins.py).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, Optional

import numpy as np

from .realq_oracle import QParams, bf16, quantize_layer, surrogate_grad

RMS_EPS = 1e-6
MODULES = ("gate", "up", "down")


def _f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


def rmsnorm(h, gamma, eps=RMS_EPS):
    """h / sqrt(mean_i h_i^2 + eps) * gamma, per token (row)."""
    h = _f64(h)
    return h / np.sqrt(np.mean(h * h, axis=1, keepdims=True) + eps) * _f64(gamma)


def rmsnorm_backward(h, gamma, du, eps=RMS_EPS):
    """dL/dh from dL/du for u = rmsnorm(h) * gamma: with r = (mean h^2 + eps)^(-1/2),
    dL/dh = r (gamma du) - r^3 h mean(h gamma du)."""
    h, gdu = _f64(h), _f64(du) * _f64(gamma)
    r = 1.0 / np.sqrt(np.mean(h * h, axis=1, keepdims=True) + eps)
    return r * gdu - (r ** 3) * h * np.mean(h * gdu, axis=1, keepdims=True)


def _sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


@dataclass
class MLPForward:
    h: np.ndarray   # [T, d] block input
    u: np.ndarray   # [T, d] normalised input (the gate and up modules' input)
    a: np.ndarray   # [T, f] gate pre-activation
    b: np.ndarray   # [T, f] up output
    z: np.ndarray   # [T, f] SwiGLU output (the down module's input)
    y: np.ndarray   # [T, d] block output


def mlp_forward(h, gamma, Wg, Wu, Wd, eps=RMS_EPS, rnd=True) -> MLPForward:
    """The MLP block's forward; rnd=False drops the bf16 roundings (for derivative checks)."""
    r = bf16 if rnd else (lambda x: x)
    h = _f64(h)
    u = r(rmsnorm(h, gamma, eps))
    a = u @ _f64(Wg).T
    b = u @ _f64(Wu).T
    z = r(a * _sigmoid(a) * b)
    y = h + r(z @ _f64(Wd).T)
    return MLPForward(h=h, u=u, a=a, b=b, z=z, y=y)


def fisher_loss(dy, F, T):
    """(1/2T) sum_t dy_t^T F dy_t (F None: identity)."""
    dy = _f64(dy)
    Fd = dy if F is None else dy @ _f64(F)
    return 0.5 / T * float(np.sum(dy * Fd))


def mlp_backward(fw: MLPForward, gy, gamma, Wg, Wu, Wd, eps=RMS_EPS):
    """Backward of the block from gy = dL/dy: returns (dL/da, dL/db, dL/dh), bf16 casts taken
    as the identity."""
    gy = _f64(gy)
    dz = gy @ _f64(Wd)
    sa = _sigmoid(fw.a)
    da = dz * fw.b * sa * (1.0 + fw.a * (1.0 - sa))
    db = dz * fw.a * sa
    du = da @ _f64(Wg) + db @ _f64(Wu)
    dh = gy + rmsnorm_backward(fw.h, gamma, du, eps)
    return da, db, dh


@dataclass
class MLPBlock:
    gamma: np.ndarray   # [d]
    Wg: np.ndarray      # [f, d]
    Wu: np.ndarray      # [f, d]
    Wd: np.ndarray      # [d, f]
    F: Optional[np.ndarray] = None   # [d, d] Fisher at the block output (None: identity)


def surrogate(fw: MLPForward, ystar, F, T, nxt: Optional[MLPBlock] = None, y2star=None, alpha=1.0,
              eps=RMS_EPS, rnd=True):
    """(L_slide, dL_slide/dy) at the block output: alpha L + (1 - alpha) L_next, where L_next is
    the Fisher loss of the next block applied to y and y* (Eq. slide_window)."""
    dy = fw.y - _f64(ystar)
    L = fisher_loss(dy, F, T)
    gy = (dy if F is None else dy @ _f64(F)) / T
    if nxt is not None and alpha < 1.0:
        f2 = mlp_forward(fw.y, nxt.gamma, nxt.Wg, nxt.Wu, nxt.Wd, eps, rnd)
        dy2 = f2.y - _f64(y2star)
        L2 = fisher_loss(dy2, nxt.F, T)
        g2 = (dy2 if nxt.F is None else dy2 @ _f64(nxt.F)) / T
        _, _, dh2 = mlp_backward(f2, g2, nxt.gamma, nxt.Wg, nxt.Wu, nxt.Wd, eps)
        L = alpha * L + (1.0 - alpha) * L2
        gy = alpha * gy + (1.0 - alpha) * dh2
    return L, gy


def module_grad(which: str, fw: MLPForward, gy, Wg, Wu, Wd, J, eps=RMS_EPS):
    """Gradient of the surrogate with respect to columns J of one module's weights, from
    gy = dL/dy: down: gy^T z[:, J]; gate: (dL/da)^T u[:, J]; up: (dL/db)^T u[:, J]."""
    gy = _f64(gy)
    if which == "down":
        return gy.T @ fw.z[:, J]
    da, db, _ = mlp_backward(fw, gy, np.ones(fw.h.shape[1]), Wg, Wu, Wd, eps)
    return (da if which == "gate" else db).T @ fw.u[:, J]


@dataclass
class BlockResult:
    modules: Dict[str, object]   # name -> realq_oracle.LayerResult
    loss_final: float            # own-block surrogate (alpha = 1) at the quantized weights
    ystar: np.ndarray


def mlp_block_sweep(X, Xhat, blk: MLPBlock, *, qp: Optional[QParams] = None, steps=0, lr=1e-3,
                    nxt: Optional[MLPBlock] = None, window=False, eps=RMS_EPS,
                    modules=MODULES) -> BlockResult:
    """Quantize gate, up and down of one MLP block in order (Alg. 1), each with GPTQ on its own
    input in the quantized path (u for gate and up, z for down) and Block-GD on the block-output
    surrogate after every column block.  window=True blends in ``nxt`` over b_global."""
    qp = qp or QParams()
    X, Xhat = _f64(X), _f64(Xhat)
    T = X.shape[0]
    W = {"gate": _f64(blk.Wg).copy(), "up": _f64(blk.Wu).copy(), "down": _f64(blk.Wd).copy()}
    ystar = mlp_forward(X, blk.gamma, W["gate"], W["up"], W["down"], eps).y
    y2star = None
    if nxt is not None:
        y2star = mlp_forward(ystar, nxt.gamma, nxt.Wg, nxt.Wu, nxt.Wd, eps).y
    nb = {k: -(-W[k].shape[1] // qp.block) for k in MODULES}
    offset, B_total = {}, 0
    for k in MODULES:
        offset[k] = B_total
        B_total += nb[k]

    def forward(Wcur):
        return mlp_forward(Xhat, blk.gamma, Wcur["gate"], Wcur["up"], Wcur["down"], eps)

    res = {}
    for name in modules:
        fw = forward(W)
        inp = fw.u if name != "down" else fw.z

        def grad_fn(Wm, J, alpha, name=name):
            Wc = dict(W)
            Wc[name] = Wm
            f = forward(Wc)
            L, gy = surrogate(f, ystar, blk.F, T, nxt, y2star, alpha, eps)
            return L, module_grad(name, f, gy, Wc["gate"], Wc["up"], Wc["down"], J, eps)

        def loss_fn(Wm, name=name):
            Wc = dict(W)
            Wc[name] = Wm
            return surrogate(forward(Wc), ystar, blk.F, T)[0]

        r = quantize_layer(W[name], inp, inp, qp=qp, steps=steps, lr=lr,
                           window=(offset[name], B_total) if (window and nxt is not None) else None,
                           grad_fn=grad_fn, loss_fn=loss_fn)
        W[name] = r.W_hat
        res[name] = r
    loss = surrogate(forward(W), ystar, blk.F, T)[0]
    return BlockResult(modules=res, loss_final=loss, ystar=ystar)


def module_surrogate_grad_of_down(z, zstar, Wd, Wd0, F, J):
    """The module-level surrogate gradient of the down projection with metric F (the reduction
    the block surrogate meets when the block input is unperturbed and roundings are dropped)."""
    R = _f64(Wd) @ _f64(z).T - _f64(Wd0) @ _f64(zstar).T
    return surrogate_grad(R, None, F, _f64(z)[:, J], _f64(z).shape[0])
