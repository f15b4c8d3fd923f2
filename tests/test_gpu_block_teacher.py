"""Teacher-forced parity of the block-output surrogate sweeps (Sec. 4.2-4.4, Alg. 1 module order):
each module of the MLP block and of the full decoder block is swept alone by the GPU
(realq_mlp_block_sweep / realq_decoder_block_sweep with start_module = k, n_modules = 1) on the
oracle's quantized weights of the modules before it and on the oracle's input activations of that
module (the bf16 roundings of u, z, O and the projections fall either way between the GPU's float32
sums and the oracle's float64 ones, and a GPTQ sweep carries one such difference along a row), and
compared with the oracle's own result for that module.  The GPU takes the oracle's outputs as inputs, never the reverse; the
free-running sweeps (tests/test_gpu_block.py, tests/test_gpu_decoder.py) remain as diagnostics of
how far the two sides drift apart over a whole block."""
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


def _report(name, met, loss_g, loss_o):
    print(name, {k: met[k] for k in ("code_identity", "code_mismatches", "tie_cascade_rows", "group_param_agreement",
                                     "first_group_agreement", "search_near_ties", "group_mismatch_at_near_ties")},
          "loss", loss_g, loss_o, flush=True)


# ---------------------------------------------------------------- MLP block

def _mlp_blk(inp):
    return B.MLPBlock(gamma=inp.gamma, Wg=inp.Wg, Wu=inp.Wu, Wd=inp.Wd, F=inp.F)


def _mlp_loss(inp, W, nxt=None):
    """Own-block surrogate (alpha = 1) at weights W (dict), the oracle's forward."""
    f = B.mlp_forward(inp.Xhat, inp.gamma, W["gate"], W["up"], W["down"])
    ys = B.mlp_forward(inp.X, inp.gamma, inp.Wg, inp.Wu, inp.Wd).y
    return B.fisher_loss(f.y - ys, inp.F, inp.X.shape[0])


@pytest.mark.parametrize("case", ["dense", "window_batch"])
def test_mlp_block_modules_teacher_forced(rq, ctx, case):
    torch = _torch()
    if case == "dense":
        inp = synth.make_mlp_block(1024, 256, 512, seed=2, dense_F=True)
        nx, window, batch = None, False, 0
    else:
        inp = synth.make_mlp_block(1024, 256, 384, seed=7)
        nx, window, batch = synth.make_mlp_block(8, 256, 384, seed=8), True, 384
    steps, lr = 3, 1e-5
    _banner(f"mlp block teacher-forced {case}")
    o = B.mlp_block_sweep(inp.X, inp.Xhat, _mlp_blk(inp), steps=steps, lr=lr,
                          nxt=None if nx is None else _mlp_blk(nx), window=window, batch=batch or None)
    W0 = {"gate": inp.Wg, "up": inp.Wu, "down": inp.Wd}
    for k, name in enumerate(B.MODULES):
        fixed = {m: _dev(o.modules[m].W_hat) for m in B.MODULES[:k]}
        Wk = {m: (o.modules[m].W_hat if j < k else W0[m]) for j, m in enumerate(B.MODULES)}
        fw = B.mlp_forward(inp.Xhat, inp.gamma, Wk["gate"], Wk["up"], Wk["down"])
        x_in = fw.z if name == "down" else fw.u            # the oracle's input of this module
        nxt = None
        if nx is not None:
            nxt = (_dev(nx.gamma), _dev(nx.Wg), _dev(nx.Wu), _dev(nx.Wd), None if nx.F is None else _dev(nx.F))
        g = rq.mlp_block_sweep(ctx, _dev(inp.X, True), _dev(inp.Xhat, True), _dev(inp.gamma), _dev(inp.Wg),
                               _dev(inp.Wu), _dev(inp.Wd), None if inp.F is None else _dev(inp.F), nxt,
                               window=window, qp=rq.qparams(), bgd=rq.bgd_params(steps=steps, lr=lr, batch=batch),
                               start=k, n_modules=1, fixed=fixed, x_fixed=_dev(x_in, True))
        torch.cuda.synchronize()
        W = {m: (o.modules[m].W_hat if j <= k else W0[m]) for j, m in enumerate(B.MODULES)}
        loss_o = _mlp_loss(inp, W)
        met = P.compare(g.modules[name], o.modules[name], tie_cascade=True)
        _report(name, met, g.loss_final, loss_o)
        for m in B.MODULES[:k]:
            assert (g.modules[m].W_hat.cpu().numpy() == np.asarray(o.modules[m].W_hat, np.float32)).all()
        assert met["code_identity"] >= P.CODE_IDENTITY, name
        assert met["tie_cascade_rows"] <= 1, name
        assert met["first_group_agreement"] >= P.CODE_IDENTITY, name
        assert met["group_param_agreement"] >= P.GROUP_AGREEMENT_AFTER_BGD, name
        assert abs(g.loss_final - loss_o) <= P.LOSS_RTOL * abs(loss_o), name


# ---------------------------------------------------------------- decoder block

DEC = dict(T=1024, d=256, f=384, n_heads=4, n_kv=2, head_dim=64, seq_len=64)


def _dec_inputs(seed, dense=True):
    s = DEC
    return synth.make_decoder_block(s["T"], s["d"], s["f"], s["n_heads"], s["n_kv"], s["head_dim"], s["seq_len"],
                                    seed=seed, dense_F=dense)


def _dec_blk(inp):
    w = inp.w
    return B.DecoderBlock(gamma1=w["gamma1"], Wq=w["Wq"], Wk=w["Wk"], Wv=w["Wv"], Wo=w["Wo"], gamma2=w["gamma2"],
                          Wg=w["Wg"], Wu=w["Wu"], Wd=w["Wd"], n_heads=inp.n_heads, n_kv=inp.n_kv,
                          head_dim=inp.head_dim, seq_len=inp.seq_len, F=w["F"])


KEYS = {"q": "Wq", "k": "Wk", "v": "Wv", "o": "Wo", "gate": "Wg", "up": "Wu", "down": "Wd"}


@pytest.mark.parametrize("seed,dense", [(1, True), (2, False)])
def test_decoder_block_modules_teacher_forced(rq, ctx, seed, dense):
    torch = _torch()
    inp = _dec_inputs(seed, dense)
    steps, lr = 2, 1e-5
    _banner(f"decoder block teacher-forced seed {seed} dense {dense}")
    blk = _dec_blk(inp)
    o = B.decoder_block_sweep(inp.X, inp.Xhat, blk, steps=steps, lr=lr)
    dev_w = {k: (None if v is None else _dev(v)) for k, v in inp.w.items()}
    for k, name in enumerate(B.DECODER_MODULES):
        fixed = {m: _dev(o.modules[m].W_hat) for m in B.DECODER_MODULES[:k]}
        Wk = {m: (o.modules[m].W_hat if j < k else np.asarray(inp.w[KEYS[m]], np.float64))
              for j, m in enumerate(B.DECODER_MODULES)}
        fw = B.decoder_forward(inp.Xhat, blk, Wk)
        x_in = {"q": fw.h1, "k": fw.h1, "v": fw.h1, "o": fw.O, "gate": fw.mlp.u, "up": fw.mlp.u,
                "down": fw.mlp.z}[name]                     # the oracle's input of this module
        g = rq.decoder_block_sweep(ctx, _dev(inp.X, True), _dev(inp.Xhat, True), dev_w, None, n_heads=inp.n_heads,
                                   n_kv=inp.n_kv, head_dim=inp.head_dim, seq_len=inp.seq_len, qp=rq.qparams(),
                                   bgd=rq.bgd_params(steps=steps, lr=lr), start=k, n_modules=1, fixed=fixed,
                                   x_fixed=_dev(x_in, True))
        torch.cuda.synchronize()
        W = {m: (o.modules[m].W_hat if j <= k else np.asarray(inp.w[KEYS[m]], np.float64))
             for j, m in enumerate(B.DECODER_MODULES)}
        ys = o.ystar
        loss_o = B.fisher_loss(B.decoder_forward(inp.Xhat, blk, W).y - ys, blk.F, inp.X.shape[0])
        met = P.compare(g.modules[name], o.modules[name], tie_cascade=True)
        _report(name, met, g.loss_final, loss_o)
        assert met["code_identity"] >= P.CODE_IDENTITY, name
        assert met["tie_cascade_rows"] <= 1, name
        assert met["first_group_agreement"] >= P.CODE_IDENTITY, name
        assert met["group_param_agreement"] >= P.GROUP_AGREEMENT_AFTER_BGD, name
        assert abs(g.loss_final - loss_o) <= P.LOSS_RTOL * abs(loss_o), name
