"""GPU parity of the window partner metric, the module hand-off and a whole synthetic decoder layer
(q, k, v, o, gate, up, down) swept in order with the sliding window, against the oracle."""
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


def _dev(a, torch, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    return t.to(dtype) if dtype is not None else t


def test_pullback_metric(rq, ctx):
    torch = _torch()
    _banner("pullback metric")
    r = np.random.default_rng(90)
    Wn = (r.standard_normal((300, 200)) * 0.05).astype(np.float32)
    A = r.standard_normal((300, 600)).astype(np.float32)
    Mn = (A @ A.T / 600).astype(np.float32)
    Wn2 = (r.standard_normal((150, 200)) * 0.05).astype(np.float32)
    P1 = torch.empty((200, 200), dtype=torch.float32, device="cuda")
    rq.pullback_metric(ctx, _dev(Wn, torch), P1)
    rq.pullback_metric(ctx, _dev(Wn2, torch), P1, accumulate=True)
    P2 = torch.empty((200, 200), dtype=torch.float32, device="cuda")
    rq.pullback_metric(ctx, _dev(Wn, torch), P2, M_next=_dev(Mn, torch))
    torch.cuda.synchronize()
    ref1 = oracle.pullback_metric(Wn) + oracle.pullback_metric(Wn2)
    ref2 = oracle.pullback_metric(Wn, Mn)
    assert P.rel_fro(P1.cpu().numpy().astype(np.float64), ref1) < 1e-5
    assert P.rel_fro(P2.cpu().numpy().astype(np.float64), ref2) < 1e-5


@pytest.mark.parametrize("swiglu", [False, True])
def test_handoff(rq, ctx, swiglu):
    torch = _torch()
    _banner(f"handoff swiglu={swiglu}")
    L = synth.make_module("llama3.1_8b_layer", "q", m=320, n=256, T=1000)
    r = np.random.default_rng(91)
    Wb = (r.standard_normal((320, 256)) * 0.02).astype(np.float32)
    X = _dev(L.Xhat, torch, torch.bfloat16)
    Y = torch.empty((1000, 320), dtype=torch.bfloat16, device="cuda")
    rq.handoff(ctx, _dev(L.W0, torch), X, Y, Wb=_dev(Wb, torch) if swiglu else None)
    torch.cuda.synchronize()
    ref = oracle.handoff(L.W0, L.Xhat, Wb if swiglu else None)
    got = Y.float().cpu().numpy().astype(np.float64)
    same = (got == ref)
    # float32 accumulation against the float64 definition: values next to a bf16 rounding
    # boundary may land on the neighbouring bf16 value, and sums that cancel carry the
    # accumulation error (bounded by 2^-20 of the sum of absolute products) into the result
    Xd = L.Xhat.astype(np.float64)
    a = Xd @ L.W0.astype(np.float64).T
    ea = 2.0 ** -20 * (np.abs(Xd) @ np.abs(L.W0.astype(np.float64)).T)
    if swiglu:
        b = Xd @ Wb.astype(np.float64).T
        eb = 2.0 ** -20 * (np.abs(Xd) @ np.abs(Wb.astype(np.float64)).T)
        err = 1.1 * np.abs(b) * ea + np.abs(oracle.silu(a)) * eb
    else:
        err = ea
    ulp = np.abs(ref) * 2.0 ** -7
    assert same.mean() >= 0.99, same.mean()
    assert (np.abs(got - ref) <= ulp + 2 * err + 1e-30).all()


D_MODEL, D_FF, D_KV, T_CHAIN = 512, 1024, 256, 1024
SHAPES = {"q": (D_MODEL, D_MODEL), "k": (D_KV, D_MODEL), "v": (D_KV, D_MODEL), "o": (D_MODEL, D_MODEL),
          "gate": (D_FF, D_MODEL), "up": (D_FF, D_MODEL), "down": (D_MODEL, D_FF)}
PARTNERS = {"q": ["o"], "o": ["gate", "up"]}
ORDER = ("q", "k", "v", "o", "gate", "up", "down")
# A module downstream of a hand-off in the free-running chain reads inputs that differ from the
# oracle's: float32 vs float64 sums land on neighbouring bf16 values for a small fraction of
# entries, and a handful of differing codes upstream change Xhat on every token.  The sequential
# sweep amplifies such differences, so there only the final loss is compared, to this bar.
FREE_CHAIN_LOSS_RTOL = 5e-2


@pytest.fixture(scope="module")
def chain_case():
    _banner("oracle decoder layer chain (about a minute on the CPU)")
    r = np.random.default_rng(92)
    W0s = {k: synth.bf16_round((r.standard_normal(s) * 0.02).astype(np.float32)) for k, s in SHAPES.items()}
    L = synth.make_module("llama3.1_8b_layer", "q", m=D_MODEL, n=D_MODEL, T=T_CHAIN)
    steps, lr = 8, L.lr
    ref, inputs = oracle.layer_chain(W0s, L.X, L.Xhat, steps=steps, lr=lr, return_inputs=True)
    return W0s, L.X, L.Xhat, steps, lr, ref, inputs


def _sweep_module(rq, ctx, torch, dW, name, X, Xh, steps, lr):
    m, n = SHAPES[name]
    Pm, window = None, None
    if name in PARTNERS:
        Pm = torch.empty((m, m), dtype=torch.float32, device="cuda")
        for i, p in enumerate(PARTNERS[name]):
            rq.pullback_metric(ctx, dW[p], Pm, accumulate=i > 0)
        window = (0, -(-n // 128))
    return rq.quantize_layer(ctx, dW[name], X, Xh, None, None, Pm, qp=rq.qparams(),
                             bgd=rq.bgd_params(steps=steps, lr=lr), window=window)


def _handoffs(rq, torch, ctx, dW, name, res, X, Xh, gate_state):
    """GPU hand-off after module ``name``: {next module: (X, Xhat)} (empty when none)."""
    bf = torch.bfloat16
    Tn = X.shape[0]
    if name in ("q", "o"):
        Y = torch.empty((Tn, SHAPES[name][0]), dtype=bf, device="cuda")
        Yh = torch.empty_like(Y)
        rq.handoff(ctx, dW[name], X, Y)
        rq.handoff(ctx, res.W_hat, Xh, Yh)
        return {"o": (Y, Yh)} if name == "q" else {"gate": (Y, Yh), "up": (Y, Yh)}
    if name == "up":
        Xg, Xhg, What_g = gate_state
        Y = torch.empty((Tn, D_FF), dtype=bf, device="cuda")
        Yh = torch.empty_like(Y)
        rq.handoff(ctx, dW["gate"], Xg, Y, Wb=dW["up"])
        rq.handoff(ctx, What_g, Xhg, Yh, Wb=res.W_hat)
        return {"down": (Y, Yh)}
    return {}


def test_decoder_layer_chain_teacher_forced(rq, ctx, chain_case):
    """Every module of a reduced LLaMA-shaped layer swept on the GPU from the oracle chain's own
    inputs (q and o with their window partners), and every GPU hand-off computed from the oracle's
    quantized weights, each held to the single-module bars."""
    torch = _torch()
    _banner("decoder layer chain, teacher forced")
    W0s, _, _, steps, lr, ref, inputs = chain_case
    dW = {k: _dev(v, torch) for k, v in W0s.items()}
    bf = torch.bfloat16
    for name in ORDER:
        X, Xh = (_dev(a, torch, bf) for a in inputs[name])
        res = _sweep_module(rq, ctx, torch, dW, name, X, Xh, steps, lr)
        torch.cuda.synchronize()
        met = P.compare(res, ref[name])
        loss_rel = abs(res.loss_final - ref[name].loss_final) / abs(ref[name].loss_final)
        print(name, met, "loss_rel", loss_rel, flush=True)
        assert met["code_identity"] >= P.CODE_IDENTITY, name
        assert met["first_group_agreement"] >= P.CODE_IDENTITY, name
        assert met["group_param_agreement"] >= P.GROUP_AGREEMENT_AFTER_BGD, name
        assert loss_rel <= P.LOSS_RTOL, name
        # hand-off of the oracle's quantized weights and inputs vs the oracle's next inputs
        Xg, Xhg = inputs["gate"]
        gate_state = (_dev(Xg, torch, bf), _dev(Xhg, torch, bf), _dev(ref["gate"].W_hat, torch))
        What_ref = type("W", (), {"W_hat": _dev(ref[name].W_hat, torch)})
        for nxt, (Y, Yh) in _handoffs(rq, torch, ctx, dW, name, What_ref, X, Xh, gate_state).items():
            torch.cuda.synchronize()
            for got, want in ((Y, inputs[nxt][0]), (Yh, inputs[nxt][1])):
                same = (got.float().cpu().numpy().astype(np.float64) == want).mean()
                assert same >= 0.99, (name, nxt, same)


def test_decoder_layer_chain_free_running(rq, ctx, chain_case):
    """The whole layer chained on the GPU alone, each module reading the GPU's own hand-offs."""
    torch = _torch()
    _banner("decoder layer chain, free running")
    W0s, X0, Xh0, steps, lr, ref, _ = chain_case
    dW = {k: _dev(v, torch) for k, v in W0s.items()}
    bf = torch.bfloat16
    X_in = {k: (_dev(X0, torch, bf), _dev(Xh0, torch, bf)) for k in ("q", "k", "v")}
    out = {}
    for name in ORDER:
        X, Xh = X_in[name]
        res = out[name] = _sweep_module(rq, ctx, torch, dW, name, X, Xh, steps, lr)
        gate_state = (*X_in["gate"], out["gate"].W_hat) if name == "up" else None
        X_in.update(_handoffs(rq, torch, ctx, dW, name, res, X, Xh, gate_state))
    torch.cuda.synchronize()
    for name in ORDER:
        met = P.compare(out[name], ref[name])
        loss_rel = abs(out[name].loss_final - ref[name].loss_final) / abs(ref[name].loss_final)
        print(name, met, "loss_rel", loss_rel, flush=True)
        if name in ("q", "k", "v"):
            # same layer input on both sides: the single-module bars hold
            assert met["code_identity"] >= P.CODE_IDENTITY, name
            assert loss_rel <= P.LOSS_RTOL, name
        else:
            assert loss_rel <= FREE_CHAIN_LOSS_RTOL, name


@pytest.mark.parametrize("swiglu", [False, True])
def test_handoff_at_model_width_sampled_tokens(rq, ctx, swiglu):
    """The hand-off at the LLaMA-3.1-8B widths and all 262144 calibration tokens: q's output
    (4096 x 4096, the o projection's input) and the SwiGLU input of the down projection from gate
    and up (14336 x 4096 each; the output, 262144 x 14336, has more elements than a 32-bit index
    reaches).  Checked against the oracle's definition on 48 sampled tokens (the last ones
    included), to the bound of the small-shape hand-off test."""
    torch = _torch()
    T = 262144
    m = 14336 if swiglu else 4096
    L = synth.make_module("llama3.1_8b_layer", "gate" if swiglu else "q", T=T)
    assert L.W0.shape == (m, 4096)
    r = np.random.default_rng(93)
    Wb = (r.standard_normal((m, 4096)) * 0.02).astype(np.float32) if swiglu else None
    _banner(f"handoff at model width m={m} T={T} swiglu={swiglu}")
    X = _dev(L.Xhat, torch, torch.bfloat16)
    Y = torch.empty((T, m), dtype=torch.bfloat16, device="cuda")
    rq.handoff(ctx, _dev(L.W0, torch), X, Y, Wb=_dev(Wb, torch) if swiglu else None)
    torch.cuda.synchronize()
    toks = np.sort(np.concatenate([r.choice(T - 8, 40, replace=False), np.arange(T - 8, T)]))
    got = Y[torch.from_numpy(toks).cuda()].float().cpu().numpy().astype(np.float64)
    del X, Y
    Xd = L.Xhat[toks].astype(np.float64)
    ref = oracle.handoff(L.W0, Xd, Wb)
    a = Xd @ L.W0.astype(np.float64).T
    ea = 2.0 ** -20 * (np.abs(Xd) @ np.abs(L.W0.astype(np.float64)).T)
    if swiglu:
        b = Xd @ Wb.astype(np.float64).T
        eb = 2.0 ** -20 * (np.abs(Xd) @ np.abs(Wb.astype(np.float64)).T)
        err = 1.1 * np.abs(b) * ea + np.abs(oracle.silu(a)) * eb
    else:
        err = ea
    ulp = np.abs(ref) * 2.0 ** -7
    same = float((got == ref).mean())
    print("identical entries", same, flush=True)
    assert same >= 0.99
    assert (np.abs(got - ref) <= ulp + 2 * err + 1e-30).all()
