"""GPU parity of the Gram-form BGD (loss and gradient through the calibration Gram matrices)
against the float64 oracle, which evaluates them over tokens: same bars as the token-streamed
path, plus agreement of the two GPU forms with each other."""
import numpy as np
import pytest

import oracle
import synth
from oracle.realq_oracle import QParams
from tests import parity as P

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


def _banner(msg):
    print(f"\n[gpu-case] {msg}", flush=True)


def _run(rq, ctx, L, steps, lr, form, M=None, P_=None, window=None):
    torch = _torch()
    W0, X, Xh, s, Md = P.to_device(L, torch)
    if M is not None:
        Md = torch.from_numpy(M).cuda()
    Pd = None if P_ is None else torch.from_numpy(P_).cuda()
    res = rq.quantize_layer(ctx, W0, X, Xh, s, Md, Pd, qp=rq.qparams(),
                            bgd=rq.bgd_params(steps=steps, lr=lr, form=form), window=window)
    torch.cuda.synchronize()
    return res


def _assert_parity(met, loss_gpu, loss_ref):
    print(met, "loss", loss_gpu, loss_ref, flush=True)
    assert met["code_identity"] >= P.CODE_IDENTITY
    assert met["first_group_agreement"] >= P.CODE_IDENTITY
    assert met["group_param_agreement"] >= P.GROUP_AGREEMENT_AFTER_BGD
    assert abs(loss_gpu - loss_ref) <= P.LOSS_RTOL * abs(loss_ref)


@pytest.mark.parametrize("case", ["single_512", "ragged"])
def test_gram_form_matches_oracle(rq, ctx, case):
    if case == "single_512":
        L = synth.make_module("single_512")
        steps, lr = L.steps, L.lr
    else:
        L = synth.make_module("single_512", m=70, n=300, T=1000)
        steps, lr = 2, 1e-3
    _banner(f"gram form {case}")
    g = _run(rq, ctx, L, steps, lr, rq.BGD_GRAM)
    o = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=steps, lr=lr)
    _assert_parity(P.compare(g, o), g.loss_final, o.loss_final)
    # the per-step losses of the first block come before any divergence is possible
    tr = g.loss_trace.cpu().numpy().reshape(-1, steps)[:-1]
    ref = np.array([v for (_, _, v) in o.loss_trace]).reshape(-1, steps)
    np.testing.assert_allclose(tr[0], ref[0], rtol=1e-4)


def test_gram_and_token_forms_agree(rq, ctx):
    L = synth.make_module("qwen3_0.6b_mlp", "gate", m=256, n=512, T=8192)
    _banner("gram vs token form")
    a = _run(rq, ctx, L, L.steps, L.lr, rq.BGD_TOKENS)
    b = _run(rq, ctx, L, L.steps, L.lr, rq.BGD_GRAM)
    ident = (a.codes.cpu() == b.codes.cpu()).float().mean().item()
    print("identity", ident, "loss", a.loss_final, b.loss_final, flush=True)
    assert ident >= P.CODE_IDENTITY
    assert abs(a.loss_final - b.loss_final) <= 1e-4 * abs(a.loss_final)
    ta = a.loss_trace.cpu().numpy()
    tb = b.loss_trace.cpu().numpy()
    np.testing.assert_allclose(tb[:L.steps], ta[:L.steps], rtol=1e-5)


def _wishart(m, seed):
    r = np.random.default_rng(seed)
    A = r.standard_normal((m, 2 * m))
    return (A @ A.T / (2 * m)).astype(np.float32)


def test_gram_form_dense_metric(rq, ctx):
    L = synth.make_module("qwen3_32b_layer", "q", m=256, n=384, T=2048)
    M = _wishart(256, 11)
    _banner("gram form dense metric")
    lr = 2e-4
    g = _run(rq, ctx, L, 4, lr, rq.BGD_GRAM, M=M)
    o = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, M=M, steps=4, lr=lr)
    _assert_parity(P.compare(g, o), g.loss_final, o.loss_final)


@pytest.mark.parametrize("window", [(0, 3), (2, 6)])
def test_gram_form_sliding_window(rq, ctx, window):
    L = synth.make_module("llama3.1_8b_layer", "q", m=256, n=384, T=2048)
    r = np.random.default_rng(12)
    Wn = (r.standard_normal((192, 256)) * 0.05).astype(np.float32)
    Pm = oracle.pullback_metric(Wn).astype(np.float32)
    _banner(f"gram form window {window}")
    g = _run(rq, ctx, L, 3, L.lr, rq.BGD_GRAM, P_=Pm, window=window)
    o = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, P=Pm, steps=3, lr=L.lr, window=window)
    _assert_parity(P.compare(g, o), g.loss_final, o.loss_final)


def test_gram_form_llama_gate_shape_sampled_rows(rq, ctx):
    """14336x4096 gate projection at 8192 tokens (full m and n) in Gram form, oracle on sampled rows."""
    L = synth.make_module("llama3.1_8b_layer", "gate", T=8192)
    _banner("gram form llama3.1-8b gate 14336x4096 T=8192")
    g = _run(rq, ctx, L, L.steps, L.lr, rq.BGD_GRAM)
    rows = np.random.default_rng(8).choice(L.W0.shape[0], 6, replace=False)
    o = oracle.quantize_layer(L.W0[rows], L.X, L.Xhat, L.s, steps=L.steps, lr=L.lr)
    lg = P.row_loss(g.W_hat.cpu().numpy()[rows], L.W0[rows], L.X, L.Xhat)
    _assert_parity(P.compare(g, o, rows=rows), lg, o.loss_final)


def test_gram_form_invalid_value_is_rejected(rq, ctx):
    torch = _torch()
    L = synth.make_module("single_512", m=8, n=128, T=64)
    W0, X, Xh, s, _ = P.to_device(L, torch)
    with pytest.raises(rq.RealqError) as ei:
        rq.quantize_layer(ctx, W0, X, Xh, qp=rq.qparams(), bgd=rq.bgd_params(steps=1, form=7))
    assert ei.value.code == -1
