"""REAL-Q per-layer quantization sweep, written out plainly in float64 on the CPU.

TEST INFRASTRUCTURE ONLY.  This module is the oracle that the GPU library is
checked against.  Only the tests, the smoke entry point and the benchmark's CPU
baseline leg may import it; the product path never does.  It shares no code,
table or constant generator with the HIP library.

Notation (paper Sec. 3.1): a linear module has weights W in R^{m x n} (row = output
channel); the calibration set gives per-token inputs x_t (rows of X, T x n).
``Xhat`` holds the inputs the partially quantized model actually feeds this
module (perturbed by already-quantized upstream layers); ``X`` holds the
full-precision model's inputs, so the full-precision output is W0 x_t.

What the sweep computes (Alg. 1 of Appendix A, restricted to one linear module,
with the per-layer surrogate of the readings below):

  1. Hessian of the layer-wise MSE, H = (2/T) sum_t s_t xhat_t xhat_t^T
     (Sec. 3.2; per-token weights as in Eq. saliency_hessian with one row group).
  2. Dead columns fixed, relative damping, and the upper-triangular inverse factor
     U with (H + lambda I)^{-1} = U^T U, whose rows are GPTQ's sequentially
     eliminated inverse (Sec. 3.2, Eq. gptq_update).
  3. For each 128-column block: group scale/zero search, column-by-column
     quantization with in-block OBS compensation (Eq. gptq_update), then the
     trailing batch update with the block error E_b (Sec. 3.2).
  4. After every block: Block-wise gradient descent (Sec. 4.3, Eq. block_gd_update)
     on the trailing columns, with Adam (Appendix D.1), against the
     Fisher-weighted MSE of the layer output (Sec. 4.2, Eq. fisher_loss) between the
     partially quantized module fed Xhat and the full-precision module fed X.
  5. The sliding window (Sec. 4.4, Eq. slide_window) blends this module's metric with
     the pulled-back metric of its consumer.

Readings where the paper is silent (each is listed in the design notes):
  * quantizer: asymmetric by default (the symmetric variant of the paper's main tables
    takes the range [-max|x|, max|x|] and the fixed zero point (maxq + 1) / 2, searching the
    shrink factor only; ``group = 0`` is one group per row), per (row, group of ``group``
    columns), joint search
    over ``grid`` shrink factors p_k = 1 - k/100 and all 2^bits zero points,
    minimising squared error; errors within 2^-40 (relative) of the minimum, plus
    2^-60 of the group's sum of squares, count as equal (an exact tie can come out either
    way in floating point, depending on the order of the sum), and among those the least
    (k, |z - z_nat|, z) wins, with the
    natural zero z_nat = rint(-lo maxq / (hi - lo)) of the unshrunk range;
    round-half-to-even; parameters fixed from the weights as they stand when the
    group's first column is reached; the chosen scale is carried as float32 (the format
    of the output), and codes and dequantized values use that stored scale, so Ŵ is
    exactly what (codes, scales, zeros) describe;
  * damping: dead columns (H_jj == 0) get H_jj = 1, then lambda = damp * mean(diag H)
    is added to the diagonal; a dead column's weights count as zero from the moment the
    sweep reaches them (the search of the group holding it, and its block), so they are
    quantized to exactly zero whatever Block-GD did to them before;
  * BGD uses all T tokens per step unless a mini-batch size is given (then consecutive
    token batches in cyclic order, one per Adam step), ``steps`` Adam steps after every
    block except the last, one Adam step counter per module;
  * the optional output-perturbation clip (a_loss_clip) scales each token's channels above
    that token's nearest-rank q-quantile of |R| down to it, with the factor held fixed;
  * the surrogate is evaluated at the module output:
        R = W Xhat^T - W0 X^T,   L = (1/2T) sum_t s_t R_t^T M R_t,
        grad_W L = (1/T) M R diag(s) Xhat.
"""
from __future__ import annotations

import math

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

ADAM_BETA1 = 0.9      # Appendix D.1
ADAM_BETA2 = 0.999    # Appendix D.1
ADAM_EPS = 1e-8       # Appendix D.1


# ============================================================================ step 1: Hessian

def hessian(Xhat: np.ndarray, s: Optional[np.ndarray] = None) -> np.ndarray:
    """H = (2/T) sum_t s_t xhat_t xhat_t^T  (Sec. 3.2 GPTQ recap; Eq. saliency_hessian with N_g = 1).

    ``s = None`` means unit weights, the plain calibration Hessian of Sec. 3.2.
    """
    Xh = np.asarray(Xhat, dtype=np.float64)
    T = Xh.shape[0]
    if s is None:
        A = Xh
    else:
        A = Xh * np.asarray(s, dtype=np.float64)[:, None]
    return (2.0 / T) * (A.T @ Xh)


def row_groups(m: int, n_groups: int) -> List[slice]:
    """The N_g row groups of Eq. saliency_hessian: contiguous ranges of ceil(m / N_g) output
    channels (the last one shorter)."""
    size = -(-m // n_groups)
    return [slice(g * size, min(m, (g + 1) * size)) for g in range(n_groups) if g * size < m]


def fisher(G: np.ndarray) -> np.ndarray:
    """Aggregated Fisher F = (1/T) sum_t g_t g_t^T of the per-token output gradients (Eq. fisher_full)."""
    G = np.asarray(G, dtype=np.float64)
    return G.T @ G / G.shape[0]


def saliency(G: np.ndarray, n_groups: int, clip_q: Optional[float] = None) -> np.ndarray:
    """Per-token saliency of each row group, s[g, t] = ||g_t restricted to group g||^2 (Sec. 3.3),
    optionally clipped per group at the nearest-rank clip_q quantile over tokens (Appendix D.1,
    Hessian-side saliency clipping).  Returns [n_groups, T]."""
    G = np.asarray(G, dtype=np.float64)
    T, m = G.shape
    s = np.stack([np.sum(G[:, sl] ** 2, axis=1) for sl in row_groups(m, n_groups)])
    if clip_q is not None:
        k = max(1, int(math.ceil(clip_q * T)))
        tau = np.sort(s, axis=1)[:, k - 1][:, None]
        s = np.minimum(s, tau)
    return s


# ============================================================================ step 2: damping + inverse factor

def damp_hessian(H: np.ndarray, damp: float) -> Tuple[np.ndarray, np.ndarray]:
    """Dead-column fix and relative damping.  Returns (H_d, dead mask).

    A column with H_jj == 0 carries no calibration signal; its diagonal is set to 1
    (the caller zeroes its weights).  Then lambda = damp * mean_j H_jj is added to
    the diagonal so that H_d is safely positive definite.
    """
    Hd = np.array(H, dtype=np.float64, copy=True)
    d = np.diag(Hd).copy()
    dead = d == 0.0
    idx = np.nonzero(dead)[0]
    Hd[idx, idx] = 1.0
    lam = damp * float(np.mean(np.diag(Hd)))
    Hd[np.diag_indices_from(Hd)] += lam
    return Hd, dead


def inverse_factor(Hd: np.ndarray) -> np.ndarray:
    """Upper-triangular U with positive diagonal and Hd^{-1} = U^T U.

    Row j of U divided by U_jj is row j of the inverse of Hd restricted to the
    columns j..n-1 (the not-yet-quantized set), divided by its diagonal entry:
    this is the compensation direction of Eq. gptq_update evaluated with the
    sequentially eliminated inverse, and U_jj^2 is the [H^{-1}]_jj of that step.
    Computed as the transpose of the lower Cholesky factor of Hd^{-1}.
    """
    Hinv = np.linalg.inv(np.asarray(Hd, dtype=np.float64))
    Hinv = 0.5 * (Hinv + Hinv.T)
    L = np.linalg.cholesky(Hinv)
    return np.triu(L.T)


# ============================================================================ step 3: quantizer

@dataclass
class QParams:
    bits: int = 4
    group: int = 128        # 0 = one group per row (per-row quantization)
    block: int = 128
    grid: int = 80          # shrink factors p_k = 1 - k/100, k = 0 .. grid-1
    damp: float = 0.01
    sym: bool = False       # symmetric: range [-max|x|, max|x|], zero fixed at (maxq + 1) / 2

    @property
    def maxq(self) -> int:
        return (1 << self.bits) - 1

    @property
    def zsym(self) -> int:
        return (self.maxq + 1) // 2

    def group_of(self, n: int) -> int:
        return self.group if self.group > 0 else n


TIE_RTOL = 2.0 ** -40   # search errors within TIE_RTOL * least + TIE_ATOL * sum x^2 are one tie
TIE_ATOL = 2.0 ** -60


def group_search(x: np.ndarray, qp: QParams, row_chunk: int = 32, with_margin: bool = False):
    """Best asymmetric (scale, zero) per row of ``x`` ([rows, g]).

    For each row: lo = min(0, min x), hi = max(0, max x) (lo = -1, hi = 1 when both
    are 0).  Candidate k has scale s_k = p_k (hi - lo) / maxq; every zero point
    z in 0..maxq is tried, with codes q = clamp(rint(x / s_k) + z, 0, maxq) and
    squared error sum_j (x_j - s_k (q_j - z))^2.  Candidates whose error is at most
    least * (1 + TIE_RTOL) + TIE_ATOL * sum_j x_j^2 are equal (the absolute part makes
    errors at rounding level, as in a group lying exactly on a grid, one tie); among them
    the winner is
    the lexicographic minimum of (k, |z - z_nat|, z), with
    z_nat = clamp(rint(-lo maxq / (hi - lo)), 0, maxq) (the shrink factor cancels from
    -p_k lo / s_k, so one natural zero serves every k, and an exact half stays exact).

    Returns (scale [rows], zero [rows] int, err [rows]), and with ``with_margin`` also the relative
    margin (e2 - e1) / e1 between the least error e1 and the least error e2 of a candidate outside
    the tie set (inf when every candidate ties): a search whose margin is tiny is a near-tie, which
    a float reordering on another machine can decide the other way.
    """
    x = np.asarray(x, dtype=np.float64)
    rows = x.shape[0]
    best_s = np.empty(rows)
    best_z = np.empty(rows, dtype=np.int64)
    best_e = np.empty(rows)
    margin = np.empty(rows)
    for r0 in range(0, rows, row_chunk):
        r1 = min(rows, r0 + row_chunk)
        best_s[r0:r1], best_z[r0:r1], best_e[r0:r1], margin[r0:r1] = _group_search_rows(x[r0:r1], qp)
    if with_margin:
        return best_s, best_z, best_e, margin
    return best_s, best_z, best_e


def search_table(x: np.ndarray, qp: QParams):
    """All candidates of the search for rows ``x``: (s [rows,K], err [rows,K,Z], z_nat [rows])."""
    maxq = qp.maxq
    lo = np.minimum(0.0, x.min(axis=1))
    hi = np.maximum(0.0, x.max(axis=1))
    if qp.sym:
        amax = np.maximum(-lo, hi)
        lo, hi = -amax, amax
    flat = lo == hi
    lo = np.where(flat, -1.0, lo)
    hi = np.where(flat, 1.0, hi)
    p = 1.0 - np.arange(qp.grid) / 100.0                    # [K]
    s = (p[None, :] * (hi - lo)[:, None]) / maxq            # [rows, K]
    z = np.arange(maxq + 1, dtype=np.float64)               # [Z]
    r = np.rint(x[:, None, :] / s[:, :, None])              # [rows, K, g]
    q = np.clip(r[:, :, None, :] + z[None, None, :, None], 0, maxq)   # [rows, K, Z, g]
    d = x[:, None, None, :] - s[:, :, None, None] * (q - z[None, None, :, None])
    err = np.sum(d * d, axis=-1)                            # [rows, K, Z]
    znat = np.clip(np.rint(-lo * maxq / (hi - lo)), 0, maxq)  # [rows]
    return s, err, znat


def _group_search_rows(x, qp):
    maxq = qp.maxq
    s, err, znat = search_table(x, qp)
    rows, K, Z = err.shape
    kk = np.broadcast_to(np.arange(K)[None, :, None], err.shape)
    zz = np.broadcast_to(np.arange(Z)[None, None, :], err.shape)
    dist = np.abs(zz - znat[:, None, None])
    # near-least error first, then the lexicographic minimum of (k, dist, z), one key at a time
    ss = np.sum(x * x, axis=1)[:, None, None]
    if qp.sym:
        err = np.where(zz == qp.zsym, err, np.inf)    # the symmetric zero point only
    emin = err.min(axis=(1, 2), keepdims=True)
    cand = err <= emin * (1.0 + TIE_RTOL) + TIE_ATOL * ss
    e2 = np.where(cand, np.inf, err).min(axis=(1, 2))
    with np.errstate(divide="ignore", invalid="ignore"):
        margin = np.where(np.isinf(e2), np.inf, (e2 - emin[:, 0, 0]) / np.maximum(emin[:, 0, 0], 1e-300))
    for key in (kk, dist, zz):
        big = np.where(cand, key, np.inf)
        cand &= key == big.min(axis=(1, 2), keepdims=True)
    flat = cand.reshape(rows, -1).argmax(axis=1)
    kb, zb = np.divmod(flat, Z)
    ridx = np.arange(rows)
    return s[ridx, kb], zb.astype(np.int64), err[ridx, kb, zb], margin


def quantize_column(w: np.ndarray, scale: np.ndarray, zero: np.ndarray, maxq: int):
    """Codes and dequantized values of one column: q = clamp(rint(w/s) + z), w_hat = s (q - z)."""
    q = np.clip(np.rint(w / scale) + zero, 0, maxq)
    return q, scale * (q - zero)


# ============================================================================ step 4: surrogate + Adam

def residual(W, W0, X, Xhat):
    """R = W Xhat^T - W0 X^T  ([m, T]): output error of the partially quantized module."""
    return W @ Xhat.T - W0 @ X.T


def surrogate_loss(R, s, Ma, T):
    """L = (1/2T) sum_t s_t R_t^T Ma R_t  (Eq. fisher_loss with per-token weights)."""
    MR = R if Ma is None else Ma @ R
    w = 1.0 if s is None else s[None, :]
    return 0.5 / T * float(np.sum(R * MR * w))


def surrogate_grad(R, s, Ma, Xhat_J, T):
    """dL/dW_J = (1/T) Ma R diag(s) Xhat_J."""
    Rs = R if s is None else R * s[None, :]
    G = Rs @ Xhat_J
    if Ma is not None:
        G = Ma @ G
    return G / T


def gram_surrogate(W0, X, Xhat, s=None, trace_loss=True, M=None, P=None, batch=None):
    """The module-output surrogate of Eq. fisher_loss (per-token weights s, metric M, optionally
    blended with the window partner's P by Eq. slide_window) and its gradient, written through the
    calibration Gram matrices Hs = Xhat^T S Xhat / T and Ks = X^T S Xhat / T instead of the [m, T]
    residual R = W Xhat^T - W0 X^T:

        (1/T) Ma R S Xhat_J = Ma (W Hs - W0 Ks)[:, J]
        (1/2T) sum_t s_t R_t^T Ma R_t = 1/2 <Ma, W Hs W^T - 2 W Ks^T W0^T + C>,
        C = (1/T) (X W0^T)^T S (X W0^T),

    with Ma = alpha M + (1 - alpha) P (identity where M is None).  Equal to surrogate_grad /
    surrogate_loss of the token form in exact arithmetic.  It lets the oracle follow a sweep over
    hundreds of thousands of tokens: the Gram matrices are formed once, every Block-GD step then
    costs k n |J| for k rows (plus k^2 |J| for a dense metric, whose rows are coupled, so then all m
    rows must be followed).  With the identity metric the rows are independent and W0 may be a
    subset of rows.  Returns (grad_fn, loss_fn) for quantize_layer; loss_fn is the own-metric
    (alpha = 1) loss over all tokens.  With trace_loss False the per-step loss in the trace is NaN
    (only the final loss is evaluated), which saves one pass over Hs and Ks per step when only the
    final weights are checked.

    ``batch``: the Sec. 4.3 mini-batch of ``minibatch`` -- the same matrices are then formed for
    every batch of consecutive tokens, each over its own token count Tb (as the token form
    normalises a batch), and grad_fn answers the step's batch (``tokens`` must be one of them)."""
    W0 = np.asarray(W0, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    Xhat = np.asarray(Xhat, dtype=np.float64)
    M = None if M is None else np.asarray(M, dtype=np.float64)
    P = None if P is None else np.asarray(P, dtype=np.float64)
    T = X.shape[0]
    k = W0.shape[0]
    sw = np.ones(T) if s is None else np.asarray(s, dtype=np.float64)
    coupled = M is not None or P is not None
    nb = 1 if batch is None or batch >= T else -(-T // batch)
    slices = [minibatch(i + 1, T, batch if nb > 1 else None) for i in range(nb)]
    # unnormalised sums over each batch: Xhat_b^T S_b Xhat_b, X_b^T S_b Xhat_b and the constant term
    parts = []
    for sl in slices:
        SXh = Xhat[sl] if s is None else Xhat[sl] * sw[sl, None]
        X0 = X[sl] @ W0.T                          # [Tb, k]
        const = X0.T @ (X0 * sw[sl, None]) if coupled else np.sum(X0 * X0 * sw[sl, None], axis=0)
        parts.append((sl, Xhat[sl].T @ SXh, X[sl].T @ SXh, const))
    full = (sum(p[1] for p in parts) / T, sum(p[2] for p in parts) / T, sum(p[3] for p in parts) / T)
    per = {p[0].start: (p[1] / (p[0].stop - p[0].start), p[2] / (p[0].stop - p[0].start),
                        p[3] / (p[0].stop - p[0].start)) for p in parts}

    def loss_at(W, Ma, g):
        Hs, Ks, C = g
        if Ma is None and not coupled:
            quad = np.sum((W @ Hs) * W, axis=1) - 2.0 * np.sum((W @ Ks.T) * W0, axis=1)
            return float(np.sum(0.5 * quad + 0.5 * C))
        A = W @ Hs @ W.T - 2.0 * (W @ Ks.T @ W0.T) + C
        return 0.5 * float(np.trace(A) if Ma is None else np.sum(Ma * A))

    def loss_fn(W):
        return loss_at(W, M, full)

    def grad_fn(W, J, alpha, tokens=slice(0, T)):
        sl = range(T)[tokens]
        if nb == 1:
            g = full if sl == range(T) else None
        else:
            g = per.get(sl.start) if len(sl) > 0 and sl.start % batch == 0 else None
            if g is not None and sl != range(T)[minibatch(1 + sl.start // batch, T, batch)]:
                g = None
        if g is None:
            raise ValueError("gram_surrogate: tokens are not one of the batches it was formed for")
        Hs, Ks, _ = g
        Ma = _blend(M, P, alpha, k)
        G = W @ Hs[:, J] - W0 @ Ks[:, J]
        if Ma is not None:
            G = Ma @ G
        return (loss_at(W, Ma, g) if trace_loss else float("nan")), G

    grad_fn.Hs = full[0]       # the calibration Gram matrix Xhat^T S Xhat / T over all tokens, i.e. H / 2
    return grad_fn, loss_fn


@dataclass
class AdamState:
    m: np.ndarray
    v: np.ndarray
    t: int = 0


def adam_update(W_J, G, mA, vA, t, lr, b1=ADAM_BETA1, b2=ADAM_BETA2, eps=ADAM_EPS):
    """One bias-corrected Adam step (Kingma & Ba form; constants of Appendix D.1).

    Returns the new (W_J, m, v); ``t`` is the step count after incrementing.
    """
    mA = b1 * mA + (1.0 - b1) * G
    vA = b2 * vA + (1.0 - b2) * G * G
    mhat = mA / (1.0 - b1 ** t)
    vhat = vA / (1.0 - b2 ** t)
    return W_J - lr * mhat / (np.sqrt(vhat) + eps), mA, vA


def minibatch(t: int, T: int, batch: Optional[int]) -> slice:
    """Tokens of Adam step t (1-based, counted over the module) when each step uses a
    mini-batch (Sec. 4.3: the surrogate is evaluated on a calibration mini-batch): the
    calibration tokens are cut into consecutive batches of ``batch`` tokens (the last one
    shorter when batch does not divide T) and the steps cycle through them in order.
    ``batch = None`` (or >= T) means all tokens every step."""
    if batch is None or batch >= T:
        return slice(0, T)
    nb = -(-T // batch)
    i = (t - 1) % nb
    return slice(i * batch, min(T, (i + 1) * batch))


def clip_factor(R: np.ndarray, q: float) -> np.ndarray:
    """Detached per-entry scale of the output-perturbation clip (Appendix D.1, a_loss_clip):
    for every token (column of R) the channels whose |R| exceeds that token's q-quantile
    over channels are scaled down to it, c = min(1, tau_t / |R|).  The quantile is the
    nearest-rank order statistic: the ceil(q m)-th smallest |R[:, t]|."""
    A = np.abs(R)
    m = A.shape[0]
    k = max(1, int(math.ceil(q * m)))
    tau = np.sort(A, axis=0)[k - 1][None, :]
    with np.errstate(divide="ignore", invalid="ignore"):
        c = np.where(A > tau, tau / A, 1.0)
    return c


def clipped_grad(R, c, s, Ma, Xhat_J, T):
    """Gradient of (1/2T) sum_t s_t (c R)_t^T Ma (c R)_t with c held fixed:
    (1/T) (c o Ma (c o R)) diag(s) Xhat_J."""
    Rc = c * R
    MRc = Rc if Ma is None else Ma @ Rc
    Y = c * MRc
    if s is not None:
        Y = Y * s[None, :]
    return Y @ Xhat_J / T


def window_alpha(b_global: int, B_total: int) -> float:
    """alpha of Eq. slide_window with a 1-based column-block step b_global of B_total.

    alpha falls linearly from 1 at the first step to 0 at the last; with a single
    step (B_total = 1) the blend is not defined and alpha = 1.
    """
    if B_total <= 1:
        return 1.0
    return 1.0 - (b_global - 1) / (B_total - 1)


# ============================================================================ the sweep

@dataclass
class LayerResult:
    codes: np.ndarray          # uint8 [m, n]
    scales: np.ndarray         # float64 [m, ngroups]
    zeros: np.ndarray          # int [m, ngroups]
    W_hat: np.ndarray          # float64 [m, n]
    H: np.ndarray              # float64 [n, n], before damping
    U: np.ndarray              # float64 [n, n]
    dead: np.ndarray           # bool [n]
    loss_final: float
    loss_trace: List[Tuple[int, int, float]] = field(default_factory=list)  # (block, step, loss)
    prerounding: Optional[np.ndarray] = None   # float64 [m, n]: w/s + z just before rounding
    E_blocks: Optional[List[np.ndarray]] = None
    search_margin: Optional[np.ndarray] = None  # float64 [m, ngroups]: group_search's margin


def quantize_layer(W0, X, Xhat, s=None, M=None, P=None, *, qp: Optional[QParams] = None,
                   steps: int = 0, lr: float = 1e-3, window: Optional[Tuple[int, int]] = None,
                   keep_E: bool = False, batch: Optional[int] = None,
                   loss_clip: Optional[float] = None, s_groups: Optional[np.ndarray] = None,
                   grad_fn=None, loss_fn=None, H: Optional[np.ndarray] = None) -> LayerResult:
    """The per-module REAL-Q sweep (Alg. 1, one linear module), in float64.

    W0 [m, n]; X, Xhat [T, n]; s [T] or None; M [m, m] or None (identity);
    P [m, m] or None: the consumer's pulled-back metric used by the sliding window;
    ``window = (b_offset, B_total)`` turns the window on: column block b of this
    module is window step b_global = b_offset + b + 1 of B_total.
    ``batch``: tokens per Adam step (see ``minibatch``; None = all T).  ``loss_clip``: the
    output-perturbation clip quantile q of ``clip_factor`` applied to the residual of every
    BGD step (None = off).  The final loss is always over all tokens, unclipped.
    ``s_groups`` [N_g, T]: saliency per row group (Eq. saliency_hessian); row group g (see
    ``row_groups``) is then quantized with its own Hessian H_g = (2/T) sum_t s[g, t] x_t x_t^T
    (and its own damping, dead columns and inverse factor) instead of the one built from ``s``;
    ``s`` keeps weighting the tokens of the BGD surrogate.  H, U and dead of the result are
    then lists over the groups.
    ``grad_fn(W, J, alpha, tokens) -> (loss, grad of W[:, J])`` replaces the module-output
    surrogate of every BGD step (a surrogate evaluated further downstream, e.g. at a transformer
    block's output) on the calibration tokens ``tokens = minibatch(t, T, batch)`` of step t, and
    ``loss_fn(W)`` the final loss over all tokens; X and the surrogate arguments are then unused
    and the Hessian still comes from Xhat.
    ``H``: the Hessian of step 1 when the caller has already formed it from Xhat and s (for
    instance as 2 Hs of gram_surrogate); it is then used instead of forming it again.
    """
    qp = qp or QParams()
    W0 = np.asarray(W0, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    Xhat = np.asarray(Xhat, dtype=np.float64)
    s = None if s is None else np.asarray(s, dtype=np.float64)
    M = None if M is None else np.asarray(M, dtype=np.float64)
    P = None if P is None else np.asarray(P, dtype=np.float64)
    m, n = W0.shape
    T = X.shape[0]
    maxq = qp.maxq
    grp = qp.group_of(n)
    ng = -(-n // grp)

    if s_groups is None:
        groups = [slice(0, m)]
        Hs = [hessian(Xhat, s) if H is None else np.asarray(H, dtype=np.float64)]
    else:
        sg = np.asarray(s_groups, dtype=np.float64)
        groups = row_groups(m, sg.shape[0])
        Hs = [hessian(Xhat, sg[g]) for g in range(len(groups))]
    deads, Us = [], []
    for Hg in Hs:
        Hd, dead_g = damp_hessian(Hg, qp.damp)
        deads.append(dead_g)
        Us.append(inverse_factor(Hd))

    W = W0.copy()
    mA = np.zeros_like(W)
    vA = np.zeros_like(W)
    t = 0
    codes = np.zeros((m, n), dtype=np.uint8)
    scales = np.zeros((m, ng))
    zeros = np.zeros((m, ng), dtype=np.int64)
    pre = np.zeros((m, n))
    margin = np.full((m, ng), np.inf)
    trace: List[Tuple[int, int, float]] = []
    Es = [] if keep_E else None

    nb = -(-n // qp.block)
    cur_s = np.ones(m)
    cur_z = np.zeros(m)
    for b in range(nb):
        c0 = b * qp.block
        c1 = min(c0 + qp.block, n)
        E = np.zeros((m, c1 - c0))
        for rs, U, dead_g in zip(groups, Us, deads):   # each row group with its own inverse factor
            W[rs, c0:c1] = np.where(dead_g[c0:c1], 0.0, W[rs, c0:c1])
            for j in range(c0, c1):
                if j % grp == 0:
                    g = j // grp
                    g1 = min(j + grp, n)
                    s64, zi, _, mg = group_search(np.where(dead_g[j:g1], 0.0, W[rs, j:g1]), qp, with_margin=True)
                    margin[rs, g] = mg
                    cur_s[rs] = s64.astype(np.float32).astype(np.float64)   # scales are carried as float32
                    cur_z[rs] = zi.astype(np.float64)
                    scales[rs, g] = cur_s[rs]
                    zeros[rs, g] = zi
                w = W[rs, j].copy()
                pre[rs, j] = w / cur_s[rs] + cur_z[rs]
                q, wq = quantize_column(w, cur_s[rs], cur_z[rs], maxq)
                codes[rs, j] = q.astype(np.uint8)
                e = (w - wq) / U[j, j]
                W[rs, j] = wq
                W[rs, j + 1:c1] -= np.outer(e, U[j, j + 1:c1])
                E[rs, j - c0] = e
            W[rs, c1:] -= E[rs] @ U[c0:c1, c1:]
        if keep_E:
            Es.append(E)

        if c1 < n and steps > 0:
            alpha = 1.0 if window is None else window_alpha(window[0] + b + 1, window[1])
            Ma = _blend(M, P, alpha, m)
            J = slice(c1, n)
            for k in range(steps):
                t += 1
                sl = minibatch(t, T, batch)
                if grad_fn is not None:
                    lv, G = grad_fn(W, J, alpha, sl)
                    trace.append((b, k, lv))
                    W[:, J], mA[:, J], vA[:, J] = adam_update(W[:, J], G, mA[:, J], vA[:, J], t, lr)
                    continue
                Tb = sl.stop - sl.start
                sb = None if s is None else s[sl]
                R = residual(W, W0, X[sl], Xhat[sl])
                if loss_clip is None:
                    trace.append((b, k, surrogate_loss(R, sb, Ma, Tb)))
                    G = surrogate_grad(R, sb, Ma, Xhat[sl, J], Tb)
                else:
                    c = clip_factor(R, loss_clip)
                    trace.append((b, k, surrogate_loss(c * R, sb, Ma, Tb)))
                    G = clipped_grad(R, c, sb, Ma, Xhat[sl, J], Tb)
                W[:, J], mA[:, J], vA[:, J] = adam_update(W[:, J], G, mA[:, J], vA[:, J], t, lr)

    if loss_fn is not None:
        loss = loss_fn(W)
    else:
        loss = surrogate_loss(residual(W, W0, X, Xhat), s, M, T)
    one = s_groups is None
    return LayerResult(codes=codes, scales=scales, zeros=zeros, W_hat=W, H=Hs[0] if one else Hs,
                       U=Us[0] if one else Us, dead=deads[0] if one else deads,
                       loss_final=loss, loss_trace=trace, prerounding=pre, E_blocks=Es, search_margin=margin)


def _blend(M, P, alpha, m):
    """M_alpha = alpha M + (1 - alpha) P (identity where M is None); None means identity."""
    if P is None or alpha == 1.0:
        return M
    Mm = np.eye(m) if M is None else M
    return alpha * Mm + (1.0 - alpha) * P


# ============================================================================ window partners + hand-off

def pullback_metric(W_next: np.ndarray, M_next: Optional[np.ndarray] = None) -> np.ndarray:
    """P = W_next^T M_next W_next: the consumer's output metric pulled back to this module's output.

    For a linear consumer y' = W_next y, a perturbation dy of this module's output
    costs dy^T P dy under the consumer's metric (Sec. 4.4: L^(l+1) through the next stage).
    """
    Wn = np.asarray(W_next, dtype=np.float64)
    if M_next is None:
        return Wn.T @ Wn
    return Wn.T @ np.asarray(M_next, dtype=np.float64) @ Wn


def silu(x):
    return x / (1.0 + np.exp(-x))


def bf16(x):
    """Nearest bfloat16 value of each entry (ties to even), returned as float64.

    The value is first rounded to float32, then to bfloat16 by adding half a bfloat16
    ulp (minus one when the kept last bit is even) to the float32 bit pattern and
    truncating; the two roundings agree with a direct rounding except on the rare
    float32 values that land exactly on a bfloat16 midpoint.
    """
    u = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32)).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def handoff(Wa, X, Wb=None):
    """Inputs the next module of the layer sees (token-major, rounded to bf16).

    Wb is None: Y = X Wa^T (output of a linear module feeding the next one);
    otherwise Y = silu(X Wa^T) * (X Wb^T) (the SwiGLU input of a down projection).
    """
    Y = np.asarray(X, dtype=np.float64) @ np.asarray(Wa, dtype=np.float64).T
    if Wb is not None:
        Y = silu(Y) * (np.asarray(X, dtype=np.float64) @ np.asarray(Wb, dtype=np.float64).T)
    return bf16(Y)


def layer_chain(W0s, X0, Xhat0, *, qp: Optional[QParams] = None, steps=0, lr=1e-3, window=True,
                modules=("q", "k", "v", "o", "gate", "up", "down"), return_inputs=False):
    """Sweep every module of a synthetic decoder layer in order, handing inputs on.

    q, k, v read the layer input; o reads q's output (a linear stand-in for attention);
    gate and up read o's output; down reads silu(gate) * up.  The quantized chain feeds
    quantized outputs forward (Xhat), the full-precision chain the original ones (X).
    Window partners (Sec. 4.4, per-module reading): q's consumer is o, o's consumers are
    gate and up, each through P = sum W0_next^T W0_next; B_total is the module's own block
    count.  Returns {module: LayerResult}, and with return_inputs also {module: (X, Xhat)}.
    """
    qp = qp or QParams()
    res = {}
    X_in = {"q": (X0, Xhat0), "k": (X0, Xhat0), "v": (X0, Xhat0)}
    partners = {"q": ["o"], "o": ["gate", "up"]}
    for name in modules:
        X, Xh = X_in[name]
        W0 = W0s[name]
        P = None
        win = None
        if window and name in partners:
            P = sum(pullback_metric(W0s[p]) for p in partners[name])
            win = (0, -(-W0.shape[1] // qp.block))
        r = quantize_layer(W0, X, Xh, P=P, qp=qp, steps=steps, lr=lr, window=win)
        res[name] = r
        if name == "q":
            X_in["o"] = (handoff(W0, X), handoff(r.W_hat, Xh))
        elif name == "o":
            X_in["gate"] = X_in["up"] = (handoff(W0, X), handoff(r.W_hat, Xh))
        elif name == "up":
            Xg, Xhg = X_in["gate"]
            X_in["down"] = (handoff(W0s["gate"], Xg, W0),
                            handoff(res["gate"].W_hat, Xhg, r.W_hat))
    return (res, X_in) if return_inputs else res
