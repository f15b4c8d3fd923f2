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
then up, then down (Eq. slide_window, B_total = all three modules' column blocks).

The full decoder block (decoder_* below) puts the attention half in front: RMSNorm, the q, k, v
projections, rotary position embedding, causal softmax attention with grouped key/value heads,
the o projection and the residual add, then the MLP half; its seven modules are quantized in
the order q, k, v, o, gate, up, down with b_global running over all of them.

Pins: every backward here is checked against central finite differences of the unrounded
forward (rnd=False), and the down projection's gradient reduces to the module-level surrogate
gradient with M = F (tests/test_block_oracle_pins.py).
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
                    modules=MODULES, batch: Optional[int] = None) -> BlockResult:
    """Quantize gate, up and down of one MLP block in order (Alg. 1), each with GPTQ on its own
    input in the quantized path (u for gate and up, z for down) and Block-GD on the block-output
    surrogate after every column block.  window=True blends in ``nxt`` over b_global.
    ``batch``: tokens per Adam step (Sec. 4.3 mini-batch, scheduled by realq_oracle.minibatch);
    a step's surrogate is the block's on those tokens alone, normalised by their count."""
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

    def forward(Wcur, tokens=slice(0, T)):
        return mlp_forward(Xhat[tokens], blk.gamma, Wcur["gate"], Wcur["up"], Wcur["down"], eps)

    res = {}
    for name in modules:
        fw = forward(W)
        inp = fw.u if name != "down" else fw.z

        def grad_fn(Wm, J, alpha, tokens, name=name):
            Wc = dict(W)
            Wc[name] = Wm
            f = forward(Wc, tokens)
            Tb = f.y.shape[0]
            L, gy = surrogate(f, ystar[tokens], blk.F, Tb, nxt, None if y2star is None else y2star[tokens],
                              alpha, eps)
            return L, module_grad(name, f, gy, Wc["gate"], Wc["up"], Wc["down"], J, eps)

        def loss_fn(Wm, name=name):
            Wc = dict(W)
            Wc[name] = Wm
            return surrogate(forward(Wc), ystar, blk.F, T)[0]

        r = quantize_layer(W[name], inp, inp, qp=qp, steps=steps, lr=lr,
                           window=(offset[name], B_total) if (window and nxt is not None) else None,
                           batch=batch, grad_fn=grad_fn, loss_fn=loss_fn)
        W[name] = r.W_hat
        res[name] = r
    loss = surrogate(forward(W), ystar, blk.F, T)[0]
    return BlockResult(modules=res, loss_final=loss, ystar=ystar)


def module_surrogate_grad_of_down(z, zstar, Wd, Wd0, F, J):
    """The module-level surrogate gradient of the down projection with metric F (the reduction
    the block surrogate meets when the block input is unperturbed and roundings are dropped)."""
    R = _f64(Wd) @ _f64(z).T - _f64(Wd0) @ _f64(zstar).T
    return surrogate_grad(R, None, F, _f64(z)[:, J], _f64(z).shape[0])


# ============================================================================ full decoder block
# The attention half: h1 = bf16(rmsnorm(x) gamma1), q/k/v = bf16(h1 W^T), rotary position
# embedding on q and k (rotate-half form, positions counted within each sequence of L tokens,
# rounded to bf16), causal softmax attention per sequence and head with grouped key/value heads
# (scores and softmax unrounded), O = bf16(P V), x2 = x + bf16(O Wo^T); then the MLP half on x2.
# Modules in Alg. 1 order: q, k, v, o, gate, up, down.

DECODER_MODULES = ("q", "k", "v", "o", "gate", "up", "down")


@dataclass
class DecoderBlock:
    gamma1: np.ndarray
    Wq: np.ndarray          # [H hd, d]
    Wk: np.ndarray          # [Hkv hd, d]
    Wv: np.ndarray          # [Hkv hd, d]
    Wo: np.ndarray          # [d, H hd]
    gamma2: np.ndarray
    Wg: np.ndarray
    Wu: np.ndarray
    Wd: np.ndarray
    n_heads: int
    n_kv: int
    head_dim: int
    seq_len: int
    F: Optional[np.ndarray] = None
    rope_base: float = 10000.0

    def weights(self):
        return {"q": self.Wq, "k": self.Wk, "v": self.Wv, "o": self.Wo, "gate": self.Wg, "up": self.Wu,
                "down": self.Wd}


def rope(x, n, hd, L, base=10000.0, inverse=False):
    """Rotary embedding of x [T, n hd] (n heads of hd), position t mod L; inverse=True applies
    the transposed rotation (the backward of the forward one)."""
    x = _f64(x)
    T = x.shape[0]
    pos = (np.arange(T) % L).astype(np.float64)
    inv = base ** (-2.0 * np.arange(hd // 2) / hd)
    ang = pos[:, None] * inv[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    xr = x.reshape(T, n, hd)
    x1, x2 = xr[..., :hd // 2], xr[..., hd // 2:]
    if inverse:
        s = -s
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1).reshape(T, n * hd)


def attention_forward(qr, kr, v, H, Hkv, hd, L):
    """Causal softmax attention per sequence of L tokens and head; head h reads key/value head
    h // (H / Hkv).  Returns (O [T, H hd] unrounded, P [T / L, H, L, L])."""
    T = qr.shape[0]
    S = T // L
    rep = H // Hkv
    O = np.zeros((T, H * hd))
    P = np.zeros((S, H, L, L))
    mask = np.triu(np.ones((L, L), dtype=bool), 1)
    for s in range(S):
        rows = slice(s * L, (s + 1) * L)
        for h in range(H):
            g = h // rep
            q = qr[rows, h * hd:(h + 1) * hd]
            k = kr[rows, g * hd:(g + 1) * hd]
            sc = q @ k.T / np.sqrt(hd)
            sc[mask] = -np.inf
            sc = sc - sc.max(axis=1, keepdims=True)
            e = np.exp(sc)
            p = e / e.sum(axis=1, keepdims=True)
            P[s, h] = p
            O[rows, h * hd:(h + 1) * hd] = p @ v[rows, g * hd:(g + 1) * hd]
    return O, P


def attention_backward(dO, P, qr, kr, v, H, Hkv, hd, L):
    """(dqr, dkr, dv) from dO [T, H hd]; key/value gradients summed over the heads that share them."""
    T = qr.shape[0]
    S = T // L
    rep = H // Hkv
    dq = np.zeros_like(qr)
    dk = np.zeros_like(kr)
    dv = np.zeros_like(v)
    for s in range(S):
        rows = slice(s * L, (s + 1) * L)
        for h in range(H):
            g = h // rep
            p = P[s, h]
            do = dO[rows, h * hd:(h + 1) * hd]
            vv = v[rows, g * hd:(g + 1) * hd]
            dp = do @ vv.T
            ds = p * (dp - np.sum(p * dp, axis=1, keepdims=True))
            dq[rows, h * hd:(h + 1) * hd] = ds @ kr[rows, g * hd:(g + 1) * hd] / np.sqrt(hd)
            dk[rows, g * hd:(g + 1) * hd] += ds.T @ qr[rows, h * hd:(h + 1) * hd] / np.sqrt(hd)
            dv[rows, g * hd:(g + 1) * hd] += p.T @ do
    return dq, dk, dv


@dataclass
class DecoderForward:
    x: np.ndarray
    h1: np.ndarray
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    qr: np.ndarray
    kr: np.ndarray
    P: np.ndarray
    O: np.ndarray       # bf16-rounded attention output [T, H hd] (the o module's input)
    x2: np.ndarray      # residual stream after attention
    mlp: MLPForward     # the MLP half on x2 (its y is the block output)

    @property
    def y(self):
        return self.mlp.y


def decoder_forward(x, blk: DecoderBlock, W=None, eps=RMS_EPS, rnd=True) -> DecoderForward:
    """Forward of the decoder block; W overrides the module weights (dict by module name)."""
    r = bf16 if rnd else (lambda a: a)
    Wm = blk.weights() if W is None else W
    H, Hkv, hd, L = blk.n_heads, blk.n_kv, blk.head_dim, blk.seq_len
    x = _f64(x)
    h1 = r(rmsnorm(x, blk.gamma1, eps))
    q = r(h1 @ _f64(Wm["q"]).T)
    k = r(h1 @ _f64(Wm["k"]).T)
    v = r(h1 @ _f64(Wm["v"]).T)
    qr = r(rope(q, H, hd, L, blk.rope_base))
    kr = r(rope(k, Hkv, hd, L, blk.rope_base))
    Oa, P = attention_forward(qr, kr, v, H, Hkv, hd, L)
    O = r(Oa)
    x2 = x + r(O @ _f64(Wm["o"]).T)
    mlp = mlp_forward(x2, blk.gamma2, Wm["gate"], Wm["up"], Wm["down"], eps, rnd)
    return DecoderForward(x=x, h1=h1, q=q, k=k, v=v, qr=qr, kr=kr, P=P, O=O, x2=x2, mlp=mlp)


def decoder_backward(fw: DecoderForward, gy, blk: DecoderBlock, W=None, eps=RMS_EPS):
    """Gradients of the surrogate from gy = dL/dy at every module output and at the block input:
    a dict with 'gate', 'up' (dL/da, dL/db), 'down' (gy), 'o' (dL/dx2), 'q', 'k', 'v' (before the
    rotary embedding for q and k) and 'x' (dL/dx).  bf16 casts are taken as the identity."""
    Wm = blk.weights() if W is None else W
    H, Hkv, hd, L = blk.n_heads, blk.n_kv, blk.head_dim, blk.seq_len
    gy = _f64(gy)
    da, db, dx2 = mlp_backward(fw.mlp, gy, blk.gamma2, Wm["gate"], Wm["up"], Wm["down"], eps)
    dO = dx2 @ _f64(Wm["o"])
    dqr, dkr, dv = attention_backward(dO, fw.P, fw.qr, fw.kr, fw.v, H, Hkv, hd, L)
    dq = rope(dqr, H, hd, L, blk.rope_base, inverse=True)
    dk = rope(dkr, Hkv, hd, L, blk.rope_base, inverse=True)
    dh1 = dq @ _f64(Wm["q"]) + dk @ _f64(Wm["k"]) + dv @ _f64(Wm["v"])
    dx = dx2 + rmsnorm_backward(fw.x, blk.gamma1, dh1, eps)
    return {"gate": da, "up": db, "down": gy, "o": dx2, "q": dq, "k": dk, "v": dv, "x": dx}


def decoder_module_grad(which, fw: DecoderForward, bw, J):
    """Gradient of the surrogate with respect to columns J of one module's weights."""
    inp = {"q": fw.h1, "k": fw.h1, "v": fw.h1, "o": fw.O, "gate": fw.mlp.u, "up": fw.mlp.u, "down": fw.mlp.z}[which]
    return bw[which].T @ inp[:, J]


def decoder_surrogate(fw: DecoderForward, ystar, blk: DecoderBlock, T, W=None, nxt: Optional[DecoderBlock] = None,
                      y2star=None, alpha=1.0, eps=RMS_EPS, rnd=True):
    """(L_slide, backward dict) at the block output; with alpha < 1 the next block's loss on y
    is blended in and its input gradient enters dL/dy."""
    dy = fw.y - _f64(ystar)
    L = fisher_loss(dy, blk.F, T)
    gy = (dy if blk.F is None else dy @ _f64(blk.F)) / T
    if nxt is not None and alpha < 1.0:
        f2 = decoder_forward(fw.y, nxt, None, eps, rnd)
        dy2 = f2.y - _f64(y2star)
        L2 = fisher_loss(dy2, nxt.F, T)
        g2 = (dy2 if nxt.F is None else dy2 @ _f64(nxt.F)) / T
        dx_next = decoder_backward(f2, g2, nxt, None, eps)["x"]
        L = alpha * L + (1.0 - alpha) * L2
        gy = alpha * gy + (1.0 - alpha) * dx_next
    return L, decoder_backward(fw, gy, blk, W, eps)


def decoder_block_sweep(X, Xhat, blk: DecoderBlock, *, qp: Optional[QParams] = None, steps=0, lr=1e-3,
                        nxt: Optional[DecoderBlock] = None, window=False, eps=RMS_EPS,
                        batch: Optional[int] = None, modules=DECODER_MODULES):
    """Quantize q, k, v, o, gate, up and down of one decoder block in order (Alg. 1): GPTQ on each
    module's input in the quantized path and Block-GD on the block-output surrogate after every
    column block; window=True blends in ``nxt`` over b_global across the seven modules.
    ``batch``: tokens per Adam step (Sec. 4.3 mini-batch), a multiple of seq_len so that every
    batch holds whole calibration sequences (attention mixes the tokens of a sequence).
    ``modules``: the leading modules to sweep (q, then k, ...); the rest keep their given weights."""
    qp = qp or QParams()
    X, Xhat = _f64(X), _f64(Xhat)
    T = X.shape[0]
    if batch is not None and batch % blk.seq_len:
        raise ValueError("decoder_block_sweep: batch must be a multiple of seq_len")
    W = {k: _f64(v).copy() for k, v in blk.weights().items()}
    ystar = decoder_forward(X, blk, W, eps).y
    y2star = decoder_forward(ystar, nxt, None, eps).y if nxt is not None else None
    nb = {k: -(-W[k].shape[1] // qp.block) for k in DECODER_MODULES}
    offset, B_total = {}, 0
    for k in DECODER_MODULES:
        offset[k] = B_total
        B_total += nb[k]
    inputs = {"q": "h1", "k": "h1", "v": "h1", "o": "O"}
    res = {}
    if tuple(modules) != DECODER_MODULES[:len(modules)]:
        raise ValueError("decoder_block_sweep: modules must be a leading run of q, k, v, o, gate, up, down")
    for name in modules:
        fw = decoder_forward(Xhat, blk, W, eps)
        inp = getattr(fw, inputs[name]) if name in inputs else (fw.mlp.u if name != "down" else fw.mlp.z)

        def grad_fn(Wm, J, alpha, tokens, name=name):
            Wc = dict(W)
            Wc[name] = Wm
            f = decoder_forward(Xhat[tokens], blk, Wc, eps)
            Tb = f.y.shape[0]
            Lv, bw = decoder_surrogate(f, ystar[tokens], blk, Tb, Wc, nxt,
                                       None if y2star is None else y2star[tokens], alpha, eps)
            return Lv, decoder_module_grad(name, f, bw, J)

        def loss_fn(Wm, name=name):
            Wc = dict(W)
            Wc[name] = Wm
            f = decoder_forward(Xhat, blk, Wc, eps)
            return fisher_loss(f.y - ystar, blk.F, T)

        r = quantize_layer(W[name], inp, inp, qp=qp, steps=steps, lr=lr,
                           window=(offset[name], B_total) if (window and nxt is not None) else None,
                           batch=batch, grad_fn=grad_fn, loss_fn=loss_fn)
        W[name] = r.W_hat
        res[name] = r
    loss = fisher_loss(decoder_forward(Xhat, blk, W, eps).y - ystar, blk.F, T)
    return BlockResult(modules=res, loss_final=loss, ystar=ystar)
