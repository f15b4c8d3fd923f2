"""Helpers shared by the GPU parity tests: moving seeded inputs to the device and
comparing GPU results with the oracle under the acceptance bars of the sweep."""
from __future__ import annotations

import math

import numpy as np

# acceptance bars
CODE_IDENTITY = 0.999      # fraction of identical int4 codes
SCALE_RTOL = 1e-4          # scales and zeros
LOSS_RTOL = 1e-3           # final surrogate loss
HESS_RTOL = 1e-3           # relative Frobenius error of H
# Groups searched after Block-GD steps: Adam's first step is close to lr * sign(g), so near-zero
# gradients step opposite ways under different rounding.  The oracle against itself, with its
# gradient perturbed by a bf16 hi/lo split's remainder (2^-17 of each token product), keeps
# 99.1-99.4% of the 512x512 layer's groups; the bar is twice that mean envelope.
GROUP_AGREEMENT_AFTER_BGD = 0.985


def to_device(L, torch):
    dev = "cuda"
    W0 = torch.from_numpy(np.ascontiguousarray(L.W0, dtype=np.float32)).to(dev)
    X = torch.from_numpy(np.ascontiguousarray(L.X, dtype=np.float32)).to(torch.bfloat16).to(dev)
    Xh = torch.from_numpy(np.ascontiguousarray(L.Xhat, dtype=np.float32)).to(torch.bfloat16).to(dev)
    s = None if L.s is None else torch.from_numpy(np.ascontiguousarray(L.s, dtype=np.float32)).to(dev)
    M = None if L.M is None else torch.from_numpy(np.ascontiguousarray(L.M, dtype=np.float32)).to(dev)
    return W0, X, Xh, s, M


def compare(gpu, ora, rows=None, group=128):
    """Metrics of a GPU LayerResult against an oracle LayerResult (optionally on a row subset)."""
    codes = gpu.codes.cpu().numpy()
    scales = gpu.scales.cpu().numpy()
    zeros = gpu.zeros.cpu().numpy()
    What = gpu.W_hat.cpu().numpy()
    if rows is not None:
        codes, scales, zeros, What = codes[rows], scales[rows], zeros[rows], What[rows]
    code_id = float((codes == ora.codes).mean())
    srel = np.abs(scales - ora.scales) / np.maximum(np.abs(ora.scales), 1e-30)
    grp_ok = (srel <= SCALE_RTOL) & (zeros == ora.zeros)
    return dict(
        code_identity=code_id,
        code_mismatches=int((codes != ora.codes).sum()),
        group_param_agreement=float(grp_ok.mean()),
        # groups searched before any Block-GD step (the first group of every row)
        first_group_agreement=float(grp_ok[:, 0].mean()),
        scale_rel_max_agreeing=float(srel[grp_ok].max()) if grp_ok.any() else math.nan,
        what_max_abs=float(np.abs(What - ora.W_hat).max()),
    )


def rel_fro(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def row_loss(W, W0, X, Xhat, s=None, M=None):
    """Surrogate loss of given weights, written out in numpy float64 in the test itself (used on
    GPU outputs, so it does not go through the oracle): (1/2T) sum_t s_t R_t^T M R_t."""
    W, W0, X, Xhat = (np.asarray(a, dtype=np.float64) for a in (W, W0, X, Xhat))
    R = W @ Xhat.T - W0 @ X.T
    MR = R if M is None else np.asarray(M, dtype=np.float64) @ R
    w = 1.0 if s is None else np.asarray(s, dtype=np.float64)[None, :]
    return 0.5 / X.shape[0] * float(np.sum(R * MR * w))
