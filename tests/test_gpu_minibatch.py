"""GPU parity of mini-batch BGD (Sec. 4.3: the surrogate on a calibration mini-batch per step) and
of the output-perturbation clip (Appendix D.1, a_loss_clip) against the float64 oracle."""
import numpy as np
import pytest

import oracle
import synth
from tests import parity as P

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


def _banner(msg):
    print(f"\n[gpu-case] {msg}", flush=True)


def _run(rq, ctx, L, steps, lr, batch=0, clip=0.0):
    torch = _torch()
    W0, X, Xh, s, _ = P.to_device(L, torch)
    res = rq.quantize_layer(ctx, W0, X, Xh, s, qp=rq.qparams(),
                            bgd=rq.bgd_params(steps=steps, lr=lr, batch=batch, loss_clip=clip))
    torch.cuda.synchronize()
    return res


# With the clip, the per-token threshold couples every channel of a token, so a different Adam
# step on one near-zero gradient moves other rows' clipped terms too: in the oracle itself,
# reversing the first Adam step of the three smallest-gradient weights of the 256x512 clip case
# leaves 99.86% of the codes and 88% of the group parameters unchanged (99.9% without the clip).
# Clipped runs keep the code and loss bars and hold scale/zero agreement to that envelope.
CLIP_GROUP_AGREEMENT = 0.85


def _check(g, o, steps, clip=False):
    met = P.compare(g, o)
    print(met, "loss", g.loss_final, o.loss_final, flush=True)
    assert met["code_identity"] >= P.CODE_IDENTITY
    assert met["first_group_agreement"] >= P.CODE_IDENTITY
    assert met["group_param_agreement"] >= (CLIP_GROUP_AGREEMENT if clip else P.GROUP_AGREEMENT_AFTER_BGD)
    assert abs(g.loss_final - o.loss_final) <= P.LOSS_RTOL * abs(o.loss_final)
    # the first block's step losses come before any divergence is possible
    tr = g.loss_trace.cpu().numpy().reshape(-1, steps)[0]
    ref = np.array([v for (b, _, v) in o.loss_trace if b == 0])
    np.testing.assert_allclose(tr, ref, rtol=1e-3)


def test_minibatch_with_a_ragged_last_batch(rq, ctx):
    L = synth.make_module("single_512", m=128, n=384, T=2000)
    _banner("mini-batch 512 of 2000 tokens")
    g = _run(rq, ctx, L, 3, 1e-3, batch=512)
    o = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=3, lr=1e-3, batch=512)
    _check(g, o, 3)


def test_loss_clip(rq, ctx):
    L = synth.make_module("qwen3_0.6b_mlp", "gate", m=256, n=384, T=2048)
    _banner("loss clip 0.95, m=256")
    g = _run(rq, ctx, L, 3, L.lr, clip=0.95)
    o = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=3, lr=L.lr, loss_clip=0.95)
    _check(g, o, 3, clip=True)


def test_minibatch_and_loss_clip(rq, ctx):
    L = synth.make_module("qwen3_0.6b_mlp", "gate", m=320, n=256, T=4096)
    _banner("mini-batch 1024 + loss clip 0.95")
    g = _run(rq, ctx, L, 4, L.lr, batch=1024, clip=0.95)
    o = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=4, lr=L.lr, batch=1024, loss_clip=0.95)
    _check(g, o, 4, clip=True)


def test_rejected_combinations(rq, ctx):
    torch = _torch()
    L = synth.make_module("single_512", m=16, n=128, T=256)
    W0, X, Xh, s, _ = P.to_device(L, torch)
    eye = torch.eye(16, dtype=torch.float32, device="cuda")
    bad = [dict(bgd=rq.bgd_params(steps=1, loss_clip=0.9), M=eye),               # clip with a dense metric
           dict(bgd=rq.bgd_params(steps=1, batch=64, form=rq.BGD_GRAM)),         # Gram form with a batch
           dict(bgd=rq.bgd_params(steps=1, loss_clip=1.5)),                      # quantile outside (0, 1]
           dict(bgd=rq.bgd_params(steps=1, batch=-3))]
    for kw in bad:
        with pytest.raises(rq.RealqError) as ei:
            rq.quantize_layer(ctx, W0, X, Xh, s, kw.get("M"), qp=rq.qparams(), bgd=kw["bgd"])
        assert ei.value.code == -1


def test_minibatch_llama_gate_full_width_sampled_rows(rq, ctx):
    """Mini-batch Block-GD at the full 14336 x 4096 width of the LLaMA-3.1-8B gate projection: 131072
    tokens cut into four batches of 32768 (16 calibration sequences of 2048 per Adam step), 8 steps
    per block at the workload's learning rate, so every block's steps cycle through the batches.
    The oracle follows 64 sampled rows (one in every 256-row tile, 8 more at random) with the
    surrogate written through each batch's own Gram matrices (oracle.gram_surrogate with a batch,
    pinned per batch against the token form); the Hessian over all tokens is checked whole."""
    import time
    torch = _torch()
    t0 = time.time()
    T, batch = 131072, 32768
    L = synth.make_module("llama3.1_8b_layer", "gate", T=T)
    m = L.W0.shape[0]
    _banner(f"mini-batch llama gate {m}x{L.W0.shape[1]} T={T} batch={batch}: inputs in {time.time() - t0:.0f} s")
    W0, X, Xh, s, _ = P.to_device(L, torch)
    g = rq.quantize_layer(ctx, W0, X, Xh, s, qp=rq.qparams(), bgd=rq.bgd_params(steps=L.steps, lr=L.lr, batch=batch),
                          want_H=True)
    torch.cuda.synchronize()
    del W0, X, Xh
    _banner(f"GPU sweep {g.ms_total:.0f} ms")
    Hg = g.H.cpu().numpy().astype(np.float64)
    g.H = None
    rows = P.tile_rows(m, per_tile=1, extra=8, seed=31)
    Xd, Xhd = L.X.astype(np.float64), L.Xhat.astype(np.float64)
    grad_fn, loss_fn = oracle.gram_surrogate(L.W0[rows], Xd, Xhd, L.s, trace_loss=False, batch=batch)
    _banner(f"per-batch Gram matrices formed at {time.time() - t0:.0f} s")
    herr = P.rel_fro(Hg, 2.0 * grad_fn.Hs)
    print("Hessian rel Frobenius", herr, flush=True)
    assert herr <= P.HESS_RTOL
    o = oracle.quantize_layer(L.W0[rows], Xd, Xhd, L.s, steps=L.steps, lr=L.lr, batch=batch, grad_fn=grad_fn,
                              loss_fn=loss_fn, H=2.0 * grad_fn.Hs)
    del Xd, Xhd
    _banner(f"oracle rows done at {time.time() - t0:.0f} s")
    met = P.compare(g, o, rows=rows, tie_cascade=True)
    print(met, flush=True)
    assert met["code_identity"] >= P.CODE_IDENTITY
    assert met["first_group_agreement"] >= P.CODE_IDENTITY
    assert met["group_param_agreement"] >= P.GROUP_AGREEMENT_AFTER_BGD
    assert met["tie_cascade_rows"] <= 1, met
    lg = loss_fn(g.W_hat.cpu().numpy()[rows].astype(np.float64))
    print("row loss", lg, o.loss_final, flush=True)
    assert abs(lg - o.loss_final) <= P.LOSS_RTOL * abs(o.loss_final)


@pytest.mark.parametrize("cfg,module", [("qwen3_0.6b_mlp", "gate"), ("llama3.1_8b_layer", "gate")])
def test_clipped_step_at_full_width(rq, ctx, cfg, module):
    """One Block-GD step with the output-perturbation clip (a_loss_clip = 0.95) on all rows of a
    full-width module (3072 or 14336 channels per token in the quantile) over the first mini-batch
    of 4096 tokens, from W = W0 with nothing locked, through realq_bgd_state_create /
    realq_bgd_step: the clip couples every channel of a token, so a sweep cannot be followed on
    sampled rows, but one step can be checked whole.  Against the oracle's clip_factor,
    clipped_grad and first Adam step over the same tokens, with Adam's eps set to the median |G| so
    that the update -lr G / (|G| + eps) carries the gradient's size and not only its sign: the
    clipped loss within 1e-5 and at least 99.9% of the updates within 1e-3 (of lr)."""
    torch = _torch()
    L = synth.make_module(cfg, module, T=8192)
    m, n = L.W0.shape
    batch, q, lr = 4096, 0.95, L.lr
    _banner(f"clipped step {cfg} {module} {m}x{n}, batch {batch}")
    X, Xh = L.X.astype(np.float64), L.Xhat.astype(np.float64)
    sl = oracle.minibatch(1, X.shape[0], batch)
    sb = L.s[sl] if L.s is not None else None
    R = oracle.residual(L.W0.astype(np.float64), L.W0.astype(np.float64), X[sl], Xh[sl])
    c = oracle.clip_factor(R, q)
    G = oracle.clipped_grad(R, c, sb, None, Xh[sl], batch)
    loss_ref = oracle.surrogate_loss(c * R, sb, None, batch)
    eps = float(np.median(np.abs(G)))
    W_ref, _, _ = oracle.adam_update(L.W0.astype(np.float64), G, np.zeros_like(G), np.zeros_like(G), 1, lr, eps=eps)
    clipped = float(np.mean(c < 1.0))
    print("clipped fraction", clipped, "eps", eps, flush=True)
    assert 0.03 <= clipped <= 0.07
    W0, Xd, Xhd, s, _ = P.to_device(L, torch)
    st = rq.BgdState(ctx, W0, Xd, Xhd, s, params=rq.bgd_params(steps=1, lr=lr, eps=eps, batch=batch, loss_clip=q))
    W = W0.double().contiguous()
    loss = torch.zeros((1,), dtype=torch.float64, device="cuda")
    rq.bgd_step(ctx, st, W, 0, 1.0, loss)
    torch.cuda.synchronize()
    st.close()
    lg = float(loss.item())
    print("clipped loss", lg, loss_ref, flush=True)
    assert abs(lg - loss_ref) <= 1e-5 * abs(loss_ref)
    W64 = L.W0.astype(np.float64)
    du_g = (W64 - W.cpu().numpy()) / lr
    du_o = (W64 - W_ref) / lr
    close = np.abs(du_g - du_o) <= 1e-3
    print("updates within 1e-3:", float(close.mean()), "max diff", float(np.abs(du_g - du_o).max()), flush=True)
    assert close.mean() >= 0.999
