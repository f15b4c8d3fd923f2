"""GPU parity of the increments (realq_bgd_params.resid_increment): within a column block,
Block-GD steps after the first take the residual as R_0 + Q with Q = bf16(W_k - W_0) Xhat^T and
the gradient as G_0 + bf16(Q o s)^T Xhat (Sec. 4.3: both are linear in the weights), where
Adam's displacement bound keeps the weight change within rms(W0) / 32, n <= 8192 and T >= 16 n.
The float64 oracle computes every step from scratch; the GPU runs with the increments allowed and
forbidden on the same inputs.  Bars as in test_gpu_parity.py."""
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


def _run(rq, ctx, L, steps, lr, inc, chunk=0):
    torch = _torch()
    W0, X, Xh, s, M = P.to_device(L, torch)
    res = rq.quantize_layer(ctx, W0, X, Xh, s, M, qp=rq.qparams(),
                            bgd=rq.bgd_params(steps=steps, lr=lr, tok_chunk=chunk, resid_increment=inc))
    torch.cuda.synchronize()
    return res


def _assert_parity(met, loss_gpu, loss_ref):
    print(met, "loss", loss_gpu, loss_ref, flush=True)
    assert met["code_identity"] >= P.CODE_IDENTITY
    assert met["first_group_agreement"] >= P.CODE_IDENTITY
    assert met["group_param_agreement"] >= P.GROUP_AGREEMENT_AFTER_BGD
    assert abs(loss_gpu - loss_ref) <= P.LOSS_RTOL * abs(loss_ref)


@pytest.mark.parametrize("m,n,T,chunk", [(300, 300, 4803, 0), (256, 384, 6144, 2048), (33, 200, 3200, 0)])
def test_increment_matches_oracle(rq, ctx, m, n, T, chunk):
    """LLaMA-3.1-8B-shaped inputs (weights N(0, 0.02^2), lr 1e-5, 8 steps per block: the bound holds)
    at ragged row, column and token counts (T >= 16 n), and with the tokens streamed in chunks."""
    L = synth.make_module("llama3.1_8b_layer", "gate", m=m, n=n, T=T, seed=11)
    _banner(f"increment m={m} n={n} T={T} chunk={chunk}")
    on = _run(rq, ctx, L, L.steps, L.lr, 1, chunk)
    off = _run(rq, ctx, L, L.steps, L.lr, 0, chunk)
    o = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=L.steps, lr=L.lr)
    _assert_parity(P.compare(on, o), on.loss_final, o.loss_final)
    _assert_parity(P.compare(off, o), off.loss_final, o.loss_final)
    # the increment ran: the scales (searched on the stepped weights) or the loss differ in their
    # last bits; the codes agree to the parity bar
    assert on.loss_final != off.loss_final or not (on.W_hat.cpu() == off.W_hat.cpu()).all()
    assert (on.codes.cpu() == off.codes.cpu()).float().mean().item() >= P.CODE_IDENTITY
    # the per-step losses of the later steps come from L0 + <G0, Delta> + sum s Q^2 / 2T: the first
    # block's match the oracle's trace, every block's the two-pass run's
    steps = L.steps
    tr_on = on.loss_trace.cpu().numpy().reshape(-1, steps)[:-1]
    tr_off = off.loss_trace.cpu().numpy().reshape(-1, steps)[:-1]
    ref = np.array([v for (_, _, v) in o.loss_trace]).reshape(-1, steps)
    np.testing.assert_allclose(tr_on[0], ref[0], rtol=1e-4)
    np.testing.assert_allclose(tr_on, tr_off, rtol=1e-4)


@pytest.mark.parametrize("case", ["lr", "tokens"])
def test_increment_not_taken_where_the_gate_fails(rq, ctx, case):
    """lr 1e-3 on weights of rms 0.02 (the displacement bound exceeds rms(W0) / 32), or the
    workload's lr with fewer than 16 tokens per input column: the two settings run the same
    launches and agree bitwise."""
    if case == "lr":
        L = synth.make_module("single_512", m=64, n=384, T=6144, seed=12)
        steps, lr = 4, 1e-3
    else:
        L = synth.make_module("llama3.1_8b_layer", "gate", m=64, n=384, T=6143, seed=12)
        steps, lr = L.steps, L.lr
    _banner(f"increment gated off ({case})")
    on = _run(rq, ctx, L, steps, lr, 1)
    off = _run(rq, ctx, L, steps, lr, 0)
    assert (on.W_hat.cpu() == off.W_hat.cpu()).all() and on.loss_final == off.loss_final


def test_five_calls_compose_to_the_layer_call_with_increment(rq, ctx):
    """The public calls (quantize_block, bgd_step) reproduce realq_quantize_layer bitwise with the
    increment taken: quantize_block restarts it at every column block."""
    torch = _torch()
    L = synth.make_module("llama3.1_8b_layer", "gate", m=96, n=384, T=6144, seed=13)
    _banner("five-call composition with the increment")
    W0, X, Xh, s, _ = P.to_device(L, torch)
    m, n, T = L.shape
    steps, lr = 4, 1e-5
    prm = rq.bgd_params(steps=steps, lr=lr)
    ref = rq.quantize_layer(ctx, W0, X, Xh, s, qp=rq.qparams(), bgd=prm)
    off = rq.quantize_layer(ctx, W0, X, Xh, s, qp=rq.qparams(), bgd=rq.bgd_params(steps=steps, lr=lr,
                                                                                   resid_increment=0))
    Hacc = torch.zeros((n, n), dtype=torch.float64, device="cuda")
    rq.hessian_accum(ctx, Xh, s, Hacc)
    U = torch.empty((n, n), dtype=torch.float32, device="cuda")
    dead = torch.empty((n,), dtype=torch.uint8, device="cuda")
    rq.chol_inverse(ctx, Hacc, T, 0.01, U, None, dead)
    st = rq.BgdState(ctx, W0, X, Xh, s, params=prm)
    W = W0.double()
    codes = torch.empty((m, n), dtype=torch.uint8, device="cuda")
    scales = torch.empty((m, n // 128), dtype=torch.float32, device="cuda")
    zeros = torch.empty((m, n // 128), dtype=torch.uint8, device="cuda")
    qp = rq.qparams()
    for c0 in range(0, n, 128):
        rq.quantize_block(ctx, W, c0, 128, U, dead, qp, codes, scales, zeros, st)
        if c0 + 128 < n:
            for _ in range(steps):
                rq.bgd_step(ctx, st, W, c0 + 128, 1.0)
    torch.cuda.synchronize()
    st.close()
    assert (codes.cpu() == ref.codes.cpu()).all()
    assert (W.float().cpu() == ref.W_hat.cpu()).all()
    assert ref.loss_final != off.loss_final or not (ref.W_hat.cpu() == off.W_hat.cpu()).all()


@pytest.mark.parametrize("case", ["dense_metric", "window_partner"])
def test_increment_with_a_metric(rq, ctx, case):
    """The gradient through a dense metric M (Eq. fisher_loss) or blended with the window partner's
    pull-back P (Eq. slide_window): the block's first gradient sum is added back before M_a is
    applied.  256 x 256 at 4096 tokens (16 per column), the workload's lr, 4 steps per block."""
    torch = _torch()
    L = synth.make_module("llama3.1_8b_layer", "q", m=256, n=256, T=4096, seed=14)
    r = np.random.default_rng(15)
    M = Pm = None
    window = None
    if case == "dense_metric":
        A = r.standard_normal((256, 512))
        M = (A @ A.T / 512).astype(np.float32)
    else:
        Wn = (r.standard_normal((192, 256)) * 0.05).astype(np.float32)
        Pm = oracle.pullback_metric(Wn).astype(np.float32)
        window = (1, 3)     # alpha = 1/2 at the one Block-GD block
    steps, lr = 4, L.lr
    _banner(f"increment with {case}")
    W0, X, Xh, s, _ = P.to_device(L, torch)
    Md = None if M is None else torch.from_numpy(M).cuda()
    Pd = None if Pm is None else torch.from_numpy(Pm).cuda()
    res = {}
    for inc in (1, 0):
        res[inc] = rq.quantize_layer(ctx, W0, X, Xh, s, Md, Pd, qp=rq.qparams(),
                                     bgd=rq.bgd_params(steps=steps, lr=lr, resid_increment=inc), window=window)
    torch.cuda.synchronize()
    o = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, M=M, P=Pm, steps=steps, lr=lr, window=window)
    for inc in (1, 0):
        _assert_parity(P.compare(res[inc], o), res[inc].loss_final, o.loss_final)
    assert res[1].loss_final != res[0].loss_final or not (res[1].W_hat.cpu() == res[0].W_hat.cpu()).all()


def test_increment_with_row_groups(rq, ctx):
    """N_g = 3 row groups, each with its own saliency Hessian (Alg. 1, Stage 1): the increments
    restart at every group's quantization of a block and at the lock."""
    torch = _torch()
    L = synth.make_module("llama3.1_8b_layer", "gate", m=200, n=256, T=4096, seed=16)
    S = synth.make_group_weights(3, 4096, seed=17)
    _banner("increment with 3 row groups")
    W0, X, Xh, s, _ = P.to_device(L, torch)
    Sd = torch.from_numpy(S).cuda()
    res = {}
    for inc in (1, 0):
        res[inc] = rq.quantize_layer(ctx, W0, X, Xh, s, qp=rq.qparams(),
                                     bgd=rq.bgd_params(steps=L.steps, lr=L.lr, resid_increment=inc), s_groups=Sd)
    torch.cuda.synchronize()
    o = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=L.steps, lr=L.lr, s_groups=S)
    for inc in (1, 0):
        _assert_parity(P.compare(res[inc], o), res[inc].loss_final, o.loss_final)
    assert res[1].loss_final != res[0].loss_final or not (res[1].W_hat.cpu() == res[0].W_hat.cpu()).all()


def test_increment_loss_when_alpha_changes_within_a_block(rq, ctx):
    """Through the public calls a caller may change the window's alpha between the steps of one
    column block: a first step through the blended metric (its loss is NaN) followed by identity
    steps, whose losses come from the block's first loss and gradient; they equal the two-pass run's."""
    import math
    torch = _torch()
    L = synth.make_module("llama3.1_8b_layer", "q", m=128, n=256, T=4096, seed=18)
    r = np.random.default_rng(19)
    Wn = (r.standard_normal((96, 128)) * 0.05).astype(np.float32)
    Pd = torch.from_numpy(oracle.pullback_metric(Wn).astype(np.float32)).cuda()
    W0, X, Xh, s, _ = P.to_device(L, torch)
    m, n, T = L.shape
    _banner("increment: alpha changes within a block")
    Hacc = torch.zeros((n, n), dtype=torch.float64, device="cuda")
    rq.hessian_accum(ctx, Xh, s, Hacc)
    U = torch.empty((n, n), dtype=torch.float32, device="cuda")
    dead = torch.empty((n,), dtype=torch.uint8, device="cuda")
    rq.chol_inverse(ctx, Hacc, T, 0.01, U, None, dead)
    qp = rq.qparams()
    out = {}
    for inc in (1, 0):
        st = rq.BgdState(ctx, W0, X, Xh, s, None, Pd, params=rq.bgd_params(steps=4, lr=L.lr, resid_increment=inc))
        W = W0.double()
        codes = torch.empty((m, n), dtype=torch.uint8, device="cuda")
        scales = torch.empty((m, n // 128), dtype=torch.float32, device="cuda")
        zeros = torch.empty((m, n // 128), dtype=torch.uint8, device="cuda")
        rq.quantize_block(ctx, W, 0, 128, U, dead, qp, codes, scales, zeros, st)
        losses = []
        for alpha in (0.5, 1.0, 1.0, 1.0):
            lo = torch.empty((1,), dtype=torch.float64, device="cuda")
            rq.bgd_step(ctx, st, W, 128, alpha, lo)
            losses.append(lo.item())
        torch.cuda.synchronize()
        st.close()
        out[inc] = losses
    print(out, flush=True)
    assert math.isnan(out[1][0]) and math.isnan(out[0][0])
    np.testing.assert_allclose(out[1][1:], out[0][1:], rtol=1e-6)


def test_increment_restarts_after_steps_minus_one_later_steps(rq, ctx):
    """A caller may take more Block-GD steps at one c1 than the parameters' `steps`: the state takes a
    fresh first step (two passes) after steps - 1 increments, so the displacement bound holds; the
    losses of 10 steps with steps = 4 equal the two-pass run's."""
    torch = _torch()
    L = synth.make_module("llama3.1_8b_layer", "gate", m=128, n=256, T=4096, seed=20)
    W0, X, Xh, s, _ = P.to_device(L, torch)
    m, n, T = L.shape
    _banner("increment: more steps than `steps` at one c1")
    Hacc = torch.zeros((n, n), dtype=torch.float64, device="cuda")
    rq.hessian_accum(ctx, Xh, s, Hacc)
    U = torch.empty((n, n), dtype=torch.float32, device="cuda")
    dead = torch.empty((n,), dtype=torch.uint8, device="cuda")
    rq.chol_inverse(ctx, Hacc, T, 0.01, U, None, dead)
    out = {}
    for inc in (1, 0):
        ctx.set_timing(True)
        ctx.reset_timing()
        st = rq.BgdState(ctx, W0, X, Xh, s, params=rq.bgd_params(steps=4, lr=L.lr, resid_increment=inc))
        W = W0.double()
        codes = torch.empty((m, n), dtype=torch.uint8, device="cuda")
        scales = torch.empty((m, n // 128), dtype=torch.float32, device="cuda")
        zeros = torch.empty((m, n // 128), dtype=torch.uint8, device="cuda")
        rq.quantize_block(ctx, W, 0, 128, U, dead, rq.qparams(), codes, scales, zeros, st)
        losses = []
        for _ in range(10):
            lo = torch.empty((1,), dtype=torch.float64, device="cuda")
            rq.bgd_step(ctx, st, W, 128, 1.0, lo)
            losses.append(lo.item())
        torch.cuda.synchronize()
        st.close()
        out[inc] = (losses, ctx.kernel_time("resid")[0], ctx.kernel_time("resid_inc")[0])
        ctx.set_timing(False)
    print(out, flush=True)
    assert out[1][1:] == (3, 7) and out[0][1:] == (10, 0)     # first steps at 0, 4, 8
    np.testing.assert_allclose(out[1][0], out[0][0], rtol=1e-6)
