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


# A code whose oracle pre-rounding value w/s + z lies within this many code units of a
# half-integer is a rounding tie: float rounding on either side may decide it either way.  The bound
# is the float drift of a weight between the two sides when every Adam step keeps its sign: the
# GPU's gradient carries about 2^-16 relative error (bf16 hi/lo operands), so each step differs by
# about lr 2^-16 and a weight that takes S steps drifts by at most S lr 2^-16 (about 4e-8 for 248
# steps at lr 1e-5, 2e-8 for 504 steps at lr 3e-6), i.e. below 1e-5 code units at the workloads'
# scales (0.004 - 0.006).  A Block-GD step whose sign flips moves a weight by up to 2 lr, 1e-3 code
# units and more, so it is not a tie.
TIE_TOL = 1e-5
# A group search whose two best candidates (outside the tie set) differ by this relative margin or
# less is a near-tie of the search; such groups are counted and reported.
SEARCH_NEAR_TIE = 1e-6


def tie_cascades(codes, ora, tol=TIE_TOL):
    """Rows whose first code mismatch is a rounding tie of the oracle (pre-rounding value within
    ``tol`` of a half-integer), with the column of that tie.  GPTQ compensates the rest of the row
    for the rounding it took, so after a tie the two sides quantize different weights and the rest
    of the row is a consequence of the tie, not a separate disagreement."""
    pre = np.asarray(ora.prerounding)
    out = {}
    for i in np.nonzero((codes != ora.codes).any(axis=1))[0]:
        j = int(np.nonzero(codes[i] != ora.codes[i])[0][0])
        v = float(pre[i, j])
        if abs(v - math.floor(v) - 0.5) <= tol:
            out[int(i)] = j
    return out


def compare(gpu, ora, rows=None, group=128, tie_cascade=False):
    """Metrics of a GPU LayerResult against an oracle LayerResult (optionally on a row subset).
    With ``tie_cascade`` the columns of a row from its first mismatch on are left out of the code
    and group metrics when that mismatch is a rounding tie (tie_cascades); the number of such rows
    and of the codes left out are reported.  Search near-ties of the oracle (groups whose best two
    candidates are within SEARCH_NEAR_TIE relative) are counted, with the group mismatches among
    them."""
    codes = gpu.codes.cpu().numpy()
    scales = gpu.scales.cpu().numpy()
    zeros = gpu.zeros.cpu().numpy()
    What = gpu.W_hat.cpu().numpy()
    if rows is not None:
        codes, scales, zeros, What = codes[rows], scales[rows], zeros[rows], What[rows]
    keep = np.ones(codes.shape, dtype=bool)
    gkeep = np.ones(scales.shape, dtype=bool)
    ties = tie_cascades(codes, ora) if tie_cascade else {}
    for i, j in ties.items():
        keep[i, j:] = False
        gkeep[i, (j // group) + 1:] = False      # groups searched after the tie
    code_id = float((codes == ora.codes)[keep].mean())
    srel = np.abs(scales - ora.scales) / np.maximum(np.abs(ora.scales), 1e-30)
    grp_ok = (srel <= SCALE_RTOL) & (zeros == ora.zeros)
    margin = getattr(ora, "search_margin", None)
    near = np.zeros(scales.shape, dtype=bool) if margin is None else np.asarray(margin) <= SEARCH_NEAR_TIE
    return dict(
        code_identity=code_id,
        code_mismatches=int((codes != ora.codes)[keep].sum()),
        tie_cascade_rows=len(ties),
        tie_cascade_codes=int((codes != ora.codes)[~keep].sum()),
        group_param_agreement=float(grp_ok[gkeep].mean()),
        # groups searched before any Block-GD step (the first group of every row)
        first_group_agreement=float(grp_ok[:, 0].mean()),
        search_near_ties=int((near & gkeep).sum()),
        group_mismatch_at_near_ties=int((near & gkeep & ~grp_ok).sum()),
        scale_rel_max_agreeing=float(srel[grp_ok].max()) if grp_ok.any() else math.nan,
        what_max_abs=float(np.abs(What - ora.W_hat).max()),
    )


def tile_rows(m, per_tile=1, extra=0, seed=0, tile=256):
    """Sampled output rows for a row-subset oracle: ``per_tile`` random rows of every ``tile``-row
    tile of the GPU GEMMs plus ``extra`` more drawn from the rest, sorted."""
    r = np.random.default_rng(seed)
    picks = set()
    for t0 in range(0, m, tile):
        t1 = min(m, t0 + tile)
        picks.update(int(v) for v in r.choice(np.arange(t0, t1), size=min(per_tile, t1 - t0), replace=False))
    rest = np.setdiff1d(np.arange(m), np.fromiter(picks, dtype=np.int64))
    if extra and len(rest):
        picks.update(int(v) for v in r.choice(rest, size=min(extra, len(rest)), replace=False))
    return np.array(sorted(picks), dtype=np.int64)


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
