"""GPU parity of the block-output surrogate sweep of a pre-norm SwiGLU MLP block
(realq_mlp_block_sweep) against the float64 oracle (oracle/block_oracle.py): gate, up and down
quantized in order with GPTQ on each module's input in the quantized path and Block-GD on the
Fisher loss at the block output, optionally blended with the next block over b_global."""
import numpy as np
import pytest

import synth
from oracle import block_oracle as B
from tests import parity as P

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


def _banner(msg):
    print(f"\n[gpu-case] {msg}", flush=True)


def _dev(a, bf16=False):
    torch = _torch()
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    return t.to(torch.bfloat16) if bf16 else t


def _blk(inp):
    return B.MLPBlock(gamma=inp.gamma, Wg=inp.Wg, Wu=inp.Wu, Wd=inp.Wd, F=inp.F)


def _run(rq, ctx, inp, steps, lr, nxt=None, window=False, batch=0):
    torch = _torch()
    nx = None
    if nxt is not None:
        nx = (_dev(nxt.gamma), _dev(nxt.Wg), _dev(nxt.Wu), _dev(nxt.Wd), None if nxt.F is None else _dev(nxt.F))
    res = rq.mlp_block_sweep(ctx, _dev(inp.X, True), _dev(inp.Xhat, True), _dev(inp.gamma), _dev(inp.Wg),
                             _dev(inp.Wu), _dev(inp.Wd), None if inp.F is None else _dev(inp.F), nx,
                             window=window, qp=rq.qparams(), bgd=rq.bgd_params(steps=steps, lr=lr, batch=batch))
    torch.cuda.synchronize()
    return res


# The down projection's input z = bf16(silu(a) b) is rounded from float32 products on the GPU and
# from float64 ones in the oracle; about 25 of the 524288 entries of the 1024 x 512 case land on
# the other side of a bf16 rounding boundary.  The oracle with 25 random entries of z moved one
# bf16 step keeps 99.98% of down's codes, all of its first groups and 99.80% of its groups, so
# down's group bar without Block-GD is 99.5%.
DOWN_GROUP_AGREEMENT = 0.995

# The block surrogate makes Block-GD far more sensitive to rounding than the module-level one:
# the oracle against itself, with its module gradients perturbed by a bf16 hi/lo split's
# remainder (2^-17 of each token product), keeps at lr = 1e-3 only 85-86% of down's codes and
# 98.4-98.7% of up's (99.96-100% at lr = 1e-5, the paper's rate for 8B-class models), so the
# full code bars are held at lr = 1e-5 and at lr = 1e-3 the loss and the first steps are compared.
# Even at lr = 1e-5 the down projection is the sensitive one: every Adam step moves a weight by
# about lr, a weight within that distance of a rounding boundary flips, and GPTQ carries the flip
# along the rest of its 512-column row.  The oracle with the ~25 z entries that the GPU rounds the
# other way (fixed, in every forward) keeps 98.4-99.9% of down's codes and 86-99.6% of its groups
# with the identity metric (99.93-99.99% and 99.7-99.8% with a dense one).  Down is therefore held
# to its first groups (searched before any of its Block-GD steps), to 98% of its codes, and to the
# loss bar.
DOWN_CODE_IDENTITY_AFTER_BGD = 0.98


def _check(g, o, bgd):
    for name in B.MODULES:
        met = P.compare(g.modules[name], o.modules[name])
        print(name, met, flush=True)
        assert met["first_group_agreement"] >= P.CODE_IDENTITY, name
        if bgd and name == "down":
            assert met["code_identity"] >= DOWN_CODE_IDENTITY_AFTER_BGD, name
            continue
        assert met["code_identity"] >= P.CODE_IDENTITY, name
        bar = P.GROUP_AGREEMENT_AFTER_BGD if bgd else (DOWN_GROUP_AGREEMENT if name == "down" else P.CODE_IDENTITY)
        assert met["group_param_agreement"] >= bar, name
    print("loss", g.loss_final, o.loss_final, flush=True)
    assert abs(g.loss_final - o.loss_final) <= P.LOSS_RTOL * abs(o.loss_final)


def test_block_sweep_without_bgd(rq, ctx):
    inp = synth.make_mlp_block(1024, 256, 512, seed=1)
    _banner("mlp block T=1024 d=256 f=512, no Block-GD")
    g = _run(rq, ctx, inp, 0, 1e-3)
    o = B.mlp_block_sweep(inp.X, inp.Xhat, _blk(inp), steps=0)
    _check(g, o, False)


@pytest.mark.parametrize("dense", [True, False])
def test_block_sweep_with_bgd(rq, ctx, dense):
    inp = synth.make_mlp_block(1024, 256, 512, seed=2, dense_F=dense)
    _banner(f"mlp block Block-GD lr 1e-5, dense F={dense}")
    steps, lr = 3, 1e-5
    g = _run(rq, ctx, inp, steps, lr)
    o = B.mlp_block_sweep(inp.X, inp.Xhat, _blk(inp), steps=steps, lr=lr)
    _check(g, o, True)
    # the first Block-GD step of the gate comes before any divergence is possible
    tr = g.loss_trace.cpu().numpy()
    assert tr[0] == pytest.approx(o.modules["gate"].loss_trace[0][2], rel=1e-4)


def test_block_sweep_large_step_loss(rq, ctx):
    inp = synth.make_mlp_block(1024, 256, 512, seed=2, dense_F=False)
    _banner("mlp block Block-GD lr 1e-3: loss and first step")
    steps, lr = 3, 1e-3
    g = _run(rq, ctx, inp, steps, lr)
    o = B.mlp_block_sweep(inp.X, inp.Xhat, _blk(inp), steps=steps, lr=lr)
    print("loss", g.loss_final, o.loss_final, flush=True)
    assert abs(g.loss_final - o.loss_final) <= P.LOSS_RTOL * abs(o.loss_final)
    tr = g.loss_trace.cpu().numpy()
    ref = [v for (_, _, v) in o.modules["gate"].loss_trace]
    np.testing.assert_allclose(tr[:steps], ref[:steps], rtol=1e-4)


def test_block_sweep_sliding_window(rq, ctx):
    inp = synth.make_mlp_block(768, 256, 384, seed=3)
    nx = synth.make_mlp_block(8, 256, 384, seed=4)
    _banner("mlp block Block-GD with the next block over b_global")
    steps, lr = 2, 1e-5
    g = _run(rq, ctx, inp, steps, lr, nxt=nx, window=True)
    o = B.mlp_block_sweep(inp.X, inp.Xhat, _blk(inp), steps=steps, lr=lr, nxt=_blk(nx), window=True)
    _check(g, o, True)
    tr = g.loss_trace.cpu().numpy()
    # step 2 of the window (alpha < 1) before any divergence: the gate's second column block
    # has not been quantized yet when the first step runs, so compare the first step only
    assert tr[0] == pytest.approx(o.modules["gate"].loss_trace[0][2], rel=1e-4)
    assert np.isnan(tr[steps * 1]) and np.isnan(tr[steps * 3])     # last blocks of gate and up


def test_block_sweep_minibatch_with_window(rq, ctx):
    inp = synth.make_mlp_block(1024, 256, 384, seed=7)
    nx = synth.make_mlp_block(8, 256, 384, seed=8)
    batch, steps, lr = 384, 3, 1e-5                 # batches of 384, 384 and a ragged 256
    _banner(f"mlp block mini-batch Block-GD, batch {batch}, with the next block over b_global")
    g = _run(rq, ctx, inp, steps, lr, nxt=nx, window=True, batch=batch)
    o = B.mlp_block_sweep(inp.X, inp.Xhat, _blk(inp), steps=steps, lr=lr, nxt=_blk(nx), window=True,
                          batch=batch)
    _check(g, o, True)
    # the gate's first column block takes one step on each batch; steps of lr 1e-5 keep the
    # two sides together, so each batch's own loss is compared
    tr = g.loss_trace.cpu().numpy()
    ref = [v for (_, _, v) in o.modules["gate"].loss_trace]
    np.testing.assert_allclose(tr[:steps], ref[:steps], rtol=1e-4)
    assert len({round(v, 6) for v in ref[:steps]}) == steps


def test_block_sweep_rejects_bad_arguments(rq, ctx):
    torch = _torch()
    inp = synth.make_mlp_block(64, 128, 256, seed=5)
    for bgd in (rq.bgd_params(steps=1, loss_clip=0.9),
                rq.bgd_params(steps=1, form=rq.BGD_GRAM)):
        with pytest.raises(rq.RealqError) as ei:
            rq.mlp_block_sweep(ctx, _dev(inp.X, True), _dev(inp.Xhat, True), _dev(inp.gamma), _dev(inp.Wg),
                               _dev(inp.Wu), _dev(inp.Wd), bgd=bgd)
        assert ei.value.code == -1
    bad = synth.make_mlp_block(64, 100, 256, seed=6)
    with pytest.raises(rq.RealqError) as ei:
        rq.mlp_block_sweep(ctx, _dev(bad.X, True), _dev(bad.Xhat, True), _dev(bad.gamma), _dev(bad.Wg),
                           _dev(bad.Wu), _dev(bad.Wd), qp=rq.qparams(group=0))
    assert ei.value.code == -2
    torch.cuda.synchronize()
