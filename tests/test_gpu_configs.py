"""GPU parity at the full widths of the workloads that only the benchmark's extra legs ran before:
the dense surrogate metric of Eq. fisher_loss at the Qwen3-32B model width (5120 rows coupled
through a Wishart metric), the sliding-window partner of Eq. slide_window at the LLaMA-3.1-8B width
(q blended with the pull-back of o), and the down projections (LLaMA-3.1-8B 4096x14336, whose
inverse factor is a 14336-wide Cholesky, and Qwen3-0.6B 1024x3072 at its full 131072 tokens).

The oracle follows the sweep through its Gram-form surrogate (oracle.gram_surrogate, pinned equal
to the token form in the CPU suite), all rows when a dense metric couples them, sampled rows when
the identity metric leaves them independent.  Bars as in test_gpu_parity.py.
"""
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


def _assert_parity(met):
    print(met, flush=True)
    assert met["code_identity"] >= P.CODE_IDENTITY
    assert met["first_group_agreement"] >= P.CODE_IDENTITY
    assert met["group_param_agreement"] >= P.GROUP_AGREEMENT_AFTER_BGD


def _gpu(rq, ctx, L, steps, lr, M=None, Pm=None, window=None):
    torch = _torch()
    W0, X, Xh, s, _ = P.to_device(L, torch)
    Md = None if M is None else torch.from_numpy(np.ascontiguousarray(M, dtype=np.float32)).cuda()
    Pd = None if Pm is None else torch.from_numpy(np.ascontiguousarray(Pm, dtype=np.float32)).cuda()
    res = rq.quantize_layer(ctx, W0, X, Xh, s, Md, Pd, qp=rq.qparams(), bgd=rq.bgd_params(steps=steps, lr=lr),
                            window=window, want_H=True)
    torch.cuda.synchronize()
    return res


def test_dense_metric_at_model_width(rq, ctx):
    """Qwen3-32B q rows (5120, the width the Wishart metric F = A A^T / 10240 couples) over 512 input
    columns and 4096 tokens with Student-t (nu = 3) activations, 4 Block-GD steps per block at 10x
    the workload's learning rate so the metric moves the weights."""
    L = synth.make_module("qwen3_32b_layer", "q", m=5120, n=512, T=4096)
    assert L.M is not None and L.M.shape == (5120, 5120)
    steps, lr = 4, 10 * L.lr
    _banner(f"dense metric m=5120 n=512 T=4096 lr={lr}")
    g = _gpu(rq, ctx, L, steps, lr, M=L.M)
    grad_fn, loss_fn = oracle.gram_surrogate(L.W0, L.X, L.Xhat, L.s, trace_loss=False, M=L.M)
    o = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, M=L.M, steps=steps, lr=lr, grad_fn=grad_fn,
                              loss_fn=loss_fn, H=2.0 * grad_fn.Hs)
    _assert_parity(P.compare(g, o))
    print("loss gpu", g.loss_final, "oracle", o.loss_final, flush=True)
    assert abs(g.loss_final - o.loss_final) <= P.LOSS_RTOL * abs(o.loss_final)
    # and it is the dense-metric loss of the weights the GPU returned
    lg = loss_fn(g.W_hat.cpu().numpy().astype(np.float64))
    assert abs(g.loss_final - lg) <= 1e-5 * abs(lg)


def test_window_partner_at_model_width(rq, ctx):
    """LLaMA-3.1-8B q rows (4096) with the pull-back P = W0_o^T W0_o of the o projection (4096 x
    4096), window over the module's own 4 blocks (alpha 1, 2/3, 1/3 at the three Block-GD blocks),
    512 input columns, 4096 tokens, 4 steps per block at 10x the workload's learning rate."""
    L = synth.make_module("llama3.1_8b_layer", "q", m=4096, n=512, T=4096)
    Lo = synth.make_module("llama3.1_8b_layer", "o", m=4096, n=4096, T=8)
    Pm = oracle.pullback_metric(Lo.W0).astype(np.float32)
    steps, lr = 4, 10 * L.lr
    nb = 512 // 128
    _banner(f"window partner m=4096 n=512 T=4096 lr={lr}")
    g = _gpu(rq, ctx, L, steps, lr, Pm=Pm, window=(0, nb))
    grad_fn, loss_fn = oracle.gram_surrogate(L.W0, L.X, L.Xhat, L.s, trace_loss=False, P=Pm)
    o = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, P=Pm, steps=steps, lr=lr, window=(0, nb), grad_fn=grad_fn,
                              loss_fn=loss_fn, H=2.0 * grad_fn.Hs)
    _assert_parity(P.compare(g, o))
    print("loss gpu", g.loss_final, "oracle", o.loss_final, flush=True)
    assert abs(g.loss_final - o.loss_final) <= P.LOSS_RTOL * abs(o.loss_final)


def test_llama_down_full_width_sampled_rows(rq, ctx):
    """LLaMA-3.1-8B down projection at its full 4096 x 14336 (a 14336-wide Hessian and Cholesky,
    112 column blocks) with 8192 tokens, 8 Block-GD steps per block at the workload's learning rate;
    the oracle follows 32 rows (one in each 256-row tile, 16 more at random) and the whole Hessian
    is held to the relative-Frobenius bar."""
    import time
    t0 = time.time()
    L = synth.make_module("llama3.1_8b_layer", "down", T=8192)
    m, n, T = L.shape
    assert (m, n) == (4096, 14336)
    _banner(f"llama down {m}x{n} T={T}: inputs drawn in {time.time() - t0:.0f} s")
    g = _gpu(rq, ctx, L, L.steps, L.lr)
    _banner(f"GPU sweep {g.ms_total:.0f} ms")
    rows = P.tile_rows(m, per_tile=1, extra=16, seed=21)
    X, Xh = L.X.astype(np.float64), L.Xhat.astype(np.float64)
    grad_fn, loss_fn = oracle.gram_surrogate(L.W0[rows], X, Xh, L.s, trace_loss=False)
    herr = P.rel_fro(g.H.cpu().numpy().astype(np.float64), 2.0 * grad_fn.Hs)
    print("Hessian rel Frobenius", herr, flush=True)
    assert herr <= P.HESS_RTOL
    o = oracle.quantize_layer(L.W0[rows], X, Xh, L.s, steps=L.steps, lr=L.lr, grad_fn=grad_fn, loss_fn=loss_fn,
                              H=2.0 * grad_fn.Hs)
    _banner(f"oracle rows done at {time.time() - t0:.0f} s")
    met = P.compare(g, o, rows=rows, tie_cascade=True)
    _assert_parity(met)
    assert met["tie_cascade_rows"] <= 1, met
    lg = loss_fn(g.W_hat.cpu().numpy()[rows].astype(np.float64))
    print("row loss", lg, o.loss_final, flush=True)
    assert abs(lg - o.loss_final) <= P.LOSS_RTOL * abs(o.loss_final)


def test_qwen_down_full_size_sampled_rows(rq, ctx):
    """Qwen3-0.6B down projection at its full 1024 x 3072 with all 131072 calibration tokens (Student-t
    nu = 4 activations, log-normal per-token weights), 8 Block-GD steps per block at lr 3e-4; the
    oracle follows 24 rows (one in each 256-row tile, 20 more at random)."""
    L = synth.make_module("qwen3_0.6b_mlp", "down")
    m, n, T = L.shape
    assert (m, n, T) == (1024, 3072, 131072)
    _banner(f"qwen down {m}x{n} T={T}")
    g = _gpu(rq, ctx, L, L.steps, L.lr)
    rows = P.tile_rows(m, per_tile=1, extra=20, seed=22)
    X, Xh = L.X.astype(np.float64), L.Xhat.astype(np.float64)
    grad_fn, loss_fn = oracle.gram_surrogate(L.W0[rows], X, Xh, L.s, trace_loss=False)
    herr = P.rel_fro(g.H.cpu().numpy().astype(np.float64), 2.0 * grad_fn.Hs)
    print("Hessian rel Frobenius", herr, flush=True)
    assert herr <= P.HESS_RTOL
    o = oracle.quantize_layer(L.W0[rows], X, Xh, L.s, steps=L.steps, lr=L.lr, grad_fn=grad_fn, loss_fn=loss_fn,
                              H=2.0 * grad_fn.Hs)
    met = P.compare(g, o, rows=rows, tie_cascade=True)
    _assert_parity(met)
    assert met["tie_cascade_rows"] <= 1, met
    lg = loss_fn(g.W_hat.cpu().numpy()[rows].astype(np.float64))
    print("row loss", lg, o.loss_final, flush=True)
    assert abs(lg - o.loss_final) <= P.LOSS_RTOL * abs(o.loss_final)
