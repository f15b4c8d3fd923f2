"""GPU parity of the block-output surrogate sweep of a full pre-norm decoder block
(realq_decoder_block_sweep: rotary causal attention with grouped key/value heads, then a SwiGLU
MLP) against the float64 oracle (oracle/block_oracle.py): q, k, v, o, gate, up and down quantized
in order with GPTQ on each module's input in the quantized path and Block-GD on the Fisher loss
at the block output, optionally blended with the next decoder block over b_global."""
import numpy as np
import pytest

import synth
from oracle import block_oracle as B
from tests import parity as P

pytestmark = pytest.mark.gpu

SHAPE = dict(T=1024, d=256, f=384, n_heads=4, n_kv=2, head_dim=64, seq_len=64)


def _torch():
    import torch
    return torch


def _banner(msg):
    print(f"\n[gpu-case] {msg}", flush=True)


def _dev(a, bf16=False):
    torch = _torch()
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    return t.to(torch.bfloat16) if bf16 else t


def _inputs(seed, T=None, dense=True):
    s = dict(SHAPE)
    if T is not None:
        s["T"] = T
    return synth.make_decoder_block(s["T"], s["d"], s["f"], s["n_heads"], s["n_kv"], s["head_dim"], s["seq_len"],
                                    seed=seed, dense_F=dense)


def _oracle_blk(inp):
    w = inp.w
    return B.DecoderBlock(gamma1=w["gamma1"], Wq=w["Wq"], Wk=w["Wk"], Wv=w["Wv"], Wo=w["Wo"], gamma2=w["gamma2"],
                          Wg=w["Wg"], Wu=w["Wu"], Wd=w["Wd"], n_heads=inp.n_heads, n_kv=inp.n_kv,
                          head_dim=inp.head_dim, seq_len=inp.seq_len, F=w["F"])


def _dev_blk(inp):
    return {k: (None if v is None else _dev(v)) for k, v in inp.w.items()}


def _run(rq, ctx, inp, steps, lr, nxt=None, window=False, batch=0):
    torch = _torch()
    res = rq.decoder_block_sweep(ctx, _dev(inp.X, True), _dev(inp.Xhat, True), _dev_blk(inp),
                                 None if nxt is None else _dev_blk(nxt), n_heads=inp.n_heads, n_kv=inp.n_kv,
                                 head_dim=inp.head_dim, seq_len=inp.seq_len, window=window, qp=rq.qparams(),
                                 bgd=rq.bgd_params(steps=steps, lr=lr, batch=batch))
    torch.cuda.synchronize()
    return res


# The GPU path accumulates every projection in float32 (weights split into three bf16 terms, so
# they enter with all 24 bits) before its bf16 rounding and keeps the attention probabilities as
# float32; the oracle rounds float64 values.  At the 1024-token shape about 5-25 of the
# 65536-262144 entries of each of q, k, v land on the other side of a bf16 rounding boundary, each
# q or k flip moves a row (or, for k, a causal column) of attention probabilities, and O -- the
# o projection's input -- ends up with 60-400 flipped entries (the GPU's own forward shows
# 168-341, within that range).  The oracle with every one of these roundings done in float32, in
# several summation orders (seeds 1, 2, 6, 7 and 8, with and without Block-GD at lr = 1e-5, dense
# and identity metric), against itself keeps all of q, k and v's codes, 99.74-99.98% of o's codes
# and 99.2-100% of its groups, 99.95-100% of gate's and up's codes and 99.35-100% of their
# groups, all first groups everywhere, and the loss within 2e-4; down, which sees every flip
# upstream and carries each along its 384-column rows through GPTQ, keeps only 96.9-99.3% of its
# codes and 52-89% of its groups.  With the next block in the window (512 tokens) the down
# projection's Block-GD follows mostly the next block's loss (its blocks have b_global 13 and 14
# of 15) and the same emulation keeps 89.4-91.8% of its codes and 39-44% of its groups (96.9-97.3%
# and 52-56% at 1024 tokens), gate and up 99.85-99.97% and 98.96-99.61%.  Hence: q, k and v at
# the module-level bars; o at 99.5% of codes and the Block-GD group bar; gate and up at 99.8% of
# codes and the Block-GD group bar; down at its first groups and 95% of its codes (85% with the
# window), with no group bar; the loss at the module-level tolerance.
O_CODE_IDENTITY = 0.995
GATE_UP_CODE_IDENTITY = 0.998
DOWN_CODE_IDENTITY = 0.95
DOWN_CODE_IDENTITY_WINDOW = 0.85


def _metrics(g, o):
    mets = {}
    for name in B.DECODER_MODULES:
        mets[name] = P.compare(g.modules[name], o.modules[name])
        print(name, mets[name], flush=True)
    print("loss", g.loss_final, o.loss_final, flush=True)
    return mets


def _check(g, o, bgd, window=False):
    mets = _metrics(g, o)
    for name, met in mets.items():
        assert met["first_group_agreement"] >= P.CODE_IDENTITY, name
        if name == "down":
            assert met["code_identity"] >= (DOWN_CODE_IDENTITY_WINDOW if window else DOWN_CODE_IDENTITY), name
            continue
        code_bar = {"o": O_CODE_IDENTITY, "gate": GATE_UP_CODE_IDENTITY, "up": GATE_UP_CODE_IDENTITY}.get(
            name, P.CODE_IDENTITY)
        assert met["code_identity"] >= code_bar, name
        group_bar = P.GROUP_AGREEMENT_AFTER_BGD if bgd or name in ("o", "gate", "up") else P.CODE_IDENTITY
        assert met["group_param_agreement"] >= group_bar, name
    assert abs(g.loss_final - o.loss_final) <= P.LOSS_RTOL * abs(o.loss_final)


def _bf16_ulp(a):
    a = np.abs(a)
    return np.where(a > 0, 2.0 ** (np.floor(np.log2(np.where(a > 0, a, 1.0))) - 7), 0.0)


@pytest.mark.parametrize("seed,which", [(1, "X"), (2, "Xhat")])
def test_decoder_forward_matches_oracle(rq, ctx, seed, which):
    """realq_decoder_forward element by element: h1 is rounded from the same float64 value on both
    sides (bit-exact); q, k and v are float32 dot products of length d before their bf16
    rounding, so an entry may differ from the oracle's by one bf16 step plus twice the dot
    product's float32 error bound d 2^-24 sum_k |h1_k W_k| (a few entries per 10^4); O inherits each
    flipped q/k entry across a row or causal column of attention (under 0.3%); x2 and y differ
    by the o and down outputs' bf16 roundings that fall the other way, each one bf16 step, so
    normwise by a few 10^-6 (bar 2e-5)."""
    torch = _torch()
    inp = _inputs(seed)
    X = getattr(inp, which)
    _banner(f"decoder forward seed {seed} on {which}")
    r = rq.decoder_forward(ctx, _dev(X, True), _dev_blk(inp), n_heads=inp.n_heads, n_kv=inp.n_kv,
                           head_dim=inp.head_dim, seq_len=inp.seq_len, intermediates=True)
    torch.cuda.synchronize()
    g = {k: v.float().cpu().numpy().astype(np.float64) for k, v in r.items()}
    blk = _oracle_blk(inp)
    o = B.decoder_forward(X, blk)
    assert (g["h1"] == o.h1).all()
    d = X.shape[1]
    for name, W in (("q", blk.Wq), ("k", blk.Wk), ("v", blk.Wv)):
        ref = getattr(o, name)
        bound = _bf16_ulp(ref) + 2 * d * 2.0 ** -24 * (np.abs(o.h1) @ np.abs(np.asarray(W, np.float64)).T)
        diff = np.abs(g[name] - ref)
        frac = float((diff > 0).mean())
        print(name, "flipped", frac, flush=True)
        assert frac <= 5e-4, name
        assert (diff <= bound).all(), name
    frac_O = float((g["O"] != o.O).mean())
    print("O flipped", frac_O, flush=True)
    assert frac_O <= 3e-3
    for name, ref in (("x2", o.x2), ("y", o.y)):
        rel = np.linalg.norm(g[name] - ref) / np.linalg.norm(ref)
        print(name, "normwise", rel, flush=True)
        assert rel <= 2e-5, name


def _blk_for(blk, n_heads, n_kv, head_dim, **_):
    """The block's tensors with the attention weights re-shaped (zero) to the given head layout, so
    that the binding's shape checks pass and the library's own checks decide."""
    torch = _torch()
    d = blk["Wq"].shape[1]
    out = dict(blk)
    out["Wq"] = torch.zeros((n_heads * head_dim, d), device="cuda")
    out["Wk"] = torch.zeros((n_kv * head_dim, d), device="cuda")
    out["Wv"] = torch.zeros((n_kv * head_dim, d), device="cuda")
    out["Wo"] = torch.zeros((d, n_heads * head_dim), device="cuda")
    return out


def test_decoder_forward_rejects_bad_arguments(rq, ctx):
    torch = _torch()
    inp = _inputs(5, T=128)
    X, blk = _dev(inp.X, True), _dev_blk(inp)
    for kw in (dict(seq_len=48), dict(seq_len=16), dict(n_kv=3), dict(head_dim=63), dict(head_dim=48)):
        args = dict(dict(n_heads=4, n_kv=2, head_dim=64, seq_len=64), **kw)
        with pytest.raises(rq.RealqError) as ei:
            rq.decoder_forward(ctx, X, _blk_for(blk, **args), **args)
        assert ei.value.code == -2, kw
    with pytest.raises(ValueError):           # weights that do not match the head layout
        rq.decoder_forward(ctx, X, blk, n_heads=4, n_kv=3, head_dim=64, seq_len=64)
    with pytest.raises(rq.RealqError) as ei:
        rq.decoder_forward(ctx, X, blk, n_heads=4, n_kv=2, head_dim=64, seq_len=64, eps=0.0)
    assert ei.value.code == -1
    torch.cuda.synchronize()


def test_decoder_sweep_without_bgd(rq, ctx):
    inp = _inputs(1)
    _banner("decoder block T=1024 d=256 f=384 H=4 Hkv=2 hd=64 L=64, no Block-GD")
    g = _run(rq, ctx, inp, 0, 1e-3)
    o = B.decoder_block_sweep(inp.X, inp.Xhat, _oracle_blk(inp), steps=0)
    _check(g, o, False)


@pytest.mark.parametrize("dense", [True, False])
def test_decoder_sweep_with_bgd(rq, ctx, dense):
    inp = _inputs(2, dense=dense)
    _banner(f"decoder block Block-GD lr 1e-5, dense F={dense}")
    steps, lr = 2, 1e-5
    g = _run(rq, ctx, inp, steps, lr)
    o = B.decoder_block_sweep(inp.X, inp.Xhat, _oracle_blk(inp), steps=steps, lr=lr)
    tr = g.loss_trace.cpu().numpy()
    print("trace0", tr[0], o.modules["q"].loss_trace[0][2], flush=True)
    _check(g, o, True)
    # the first Block-GD step of q comes before any divergence is possible
    assert tr[0] == pytest.approx(o.modules["q"].loss_trace[0][2], rel=1e-4)


def test_decoder_sweep_sliding_window(rq, ctx):
    inp = _inputs(3, T=512)
    nx = _inputs(4, T=64)
    _banner("decoder block Block-GD with the next decoder block over b_global")
    steps, lr = 2, 1e-5
    g = _run(rq, ctx, inp, steps, lr, nxt=nx, window=True)
    o = B.decoder_block_sweep(inp.X, inp.Xhat, _oracle_blk(inp), steps=steps, lr=lr, nxt=_oracle_blk(nx),
                              window=True)
    tr = g.loss_trace.cpu().numpy()
    print("trace0", tr[0], o.modules["q"].loss_trace[0][2], flush=True)
    _check(g, o, True, window=True)
    assert tr[0] == pytest.approx(o.modules["q"].loss_trace[0][2], rel=1e-4)
    assert np.isnan(tr[steps * 1])      # q has two column blocks; its last one takes no step


def test_decoder_sweep_rejects_bad_arguments(rq, ctx):
    torch = _torch()
    inp = _inputs(5, T=128)
    X, Xh, blk = _dev(inp.X, True), _dev(inp.Xhat, True), _dev_blk(inp)
    base = dict(n_heads=4, n_kv=2, head_dim=64, seq_len=64)
    for kw in (dict(seq_len=48), dict(seq_len=16), dict(n_kv=3), dict(seq_len=8192), dict(head_dim=63),
               dict(head_dim=48)):
        args = dict(base, **kw)
        with pytest.raises(rq.RealqError) as ei:
            rq.decoder_block_sweep(ctx, X, Xh, _blk_for(blk, **args), **args)
        assert ei.value.code == -2, kw
    for bgd in (rq.bgd_params(steps=1, loss_clip=0.9), rq.bgd_params(steps=1, form=rq.BGD_GRAM)):
        with pytest.raises(rq.RealqError) as ei:
            rq.decoder_block_sweep(ctx, X, Xh, blk, **base, bgd=bgd)
        assert ei.value.code == -1
    # a mini-batch must hold whole sequences
    with pytest.raises(rq.RealqError) as ei:
        rq.decoder_block_sweep(ctx, X, Xh, blk, **base, bgd=rq.bgd_params(steps=1, batch=96))
    assert ei.value.code == -2
    torch.cuda.synchronize()


def test_decoder_sweep_minibatch(rq, ctx):
    inp = _inputs(6)
    batch, steps, lr = 384, 3, 1e-5                 # six sequences, six, and a ragged four
    _banner(f"decoder block mini-batch Block-GD, batch {batch}")
    g = _run(rq, ctx, inp, steps, lr, batch=batch)
    o = B.decoder_block_sweep(inp.X, inp.Xhat, _oracle_blk(inp), steps=steps, lr=lr, batch=batch)
    tr = g.loss_trace.cpu().numpy()
    ref = [v for (_, _, v) in o.modules["q"].loss_trace]
    print("trace", tr[:steps], ref[:steps], flush=True)
    _check(g, o, True)
    # q's first column block takes one step on each batch
    np.testing.assert_allclose(tr[:steps], ref[:steps], rtol=1e-4)


def test_decoder_forward_llama8b_shape_one_sequence(rq, ctx):
    """realq_decoder_forward at the LLaMA-3.1-8B block shape the benchmark times (d 4096, 32 query
    heads over 8 key/value heads of 128, f 14336) on one 2048-token sequence: 64 attention tiles
    per side and every value-column tile of the MFMA kernels.  At this shape the bf16 roundings
    cascade further: a flipped key moves a causal column of up to 2048 queries, and flips of O,
    x2 and u feed each other through the MLP.  The oracle with every product in float32 (scores
    included) against itself flips 2.0e-4 of q, k, v and 0.43% of O, with x2 and y normwise
    4.2e-4 and 2.0e-3 off; the GPU's MFMA sums flip about a third more of q, k, v and about twice
    as much of O.  Bars: q, k, v as in test_decoder_forward_matches_oracle; O flips under 2%; x2 and
    y normwise within 2e-3 and 6e-3.  A wrong head, mask or scale moves most entries instead."""
    torch = _torch()
    inp = synth.make_decoder_block(2048, 4096, 14336, 32, 8, 128, 2048, seed=11)
    _banner("decoder forward at the 8B block shape, one 2048-token sequence")
    r = rq.decoder_forward(ctx, _dev(inp.Xhat, True), _dev_blk(inp), n_heads=32, n_kv=8, head_dim=128,
                           seq_len=2048, intermediates=True)
    torch.cuda.synchronize()
    g = {k: v.float().cpu().numpy().astype(np.float64) for k, v in r.items()}
    blk = _oracle_blk(inp)
    o = B.decoder_forward(inp.Xhat, blk)
    d = 4096
    frac, within = {}, {}
    for name, W in (("q", blk.Wq), ("k", blk.Wk), ("v", blk.Wv)):
        ref = getattr(o, name)
        bound = _bf16_ulp(ref) + 2 * d * 2.0 ** -24 * (np.abs(o.h1) @ np.abs(np.asarray(W, np.float64)).T)
        diff = np.abs(g[name] - ref)
        frac[name] = float((diff > 0).mean())
        within[name] = bool((diff <= bound).all())
    frac_O = float((g["O"] != o.O).mean())
    rel = {name: float(np.linalg.norm(g[name] - ref) / np.linalg.norm(ref)) for name, ref in (("x2", o.x2), ("y", o.y))}
    print("flipped", frac, "within bound", within, "O flipped", frac_O, "normwise", rel, flush=True)
    assert (g["h1"] == o.h1).all()
    for name in ("q", "k", "v"):
        assert frac[name] <= 5e-4 and within[name], name
    assert frac_O <= 2e-2
    assert rel["x2"] <= 2e-3 and rel["y"] <= 6e-3


def test_decoder_first_steps_with_wide_heads(rq, ctx):
    """Block-GD through attention with head_dim 128, 8 query heads over 2 key/value heads (4 per
    group) and 8 tiles per 256-token sequence, at lr 1e-4.  The first Adam step of each module's
    first column block lowers the loss by about lr sum |g| (a step far smaller than the weights),
    so that decrease checks the magnitude and sign of the gradient through the attention backward:
    within 1% of the oracle's for q (both sides at the same weights; the loss itself agrees to about
    1e-5 of its value) and within 5% for k, v and o, whose states carry the small differences of
    the modules before them.  Over the whole sweep at this rate the oracle with every product in
    float32 (three summation orders) ends 1.0e-3 to 3.5e-3 away from itself in its final loss, so
    that is held to 5e-3."""
    inp = synth.make_decoder_block(512, 512, 768, 8, 2, 128, 256, seed=12, dense_F=False)
    _banner("decoder block, head_dim 128, 8 over 2 heads, 256-token sequences, lr 1e-4")
    steps, lr = 2, 1e-4
    g = _run(rq, ctx, inp, steps, lr)
    o = B.decoder_block_sweep(inp.X, inp.Xhat, _oracle_blk(inp), steps=steps, lr=lr)
    tr = g.loss_trace.cpu().numpy()
    off = 0
    for name in B.DECODER_MODULES:
        ref = o.modules[name].loss_trace
        d_g, d_o = tr[off + 1] - tr[off], ref[1][2] - ref[0][2]
        print(name, "first-step decrease", d_g, d_o, flush=True)
        if name in ("q", "k", "v", "o"):
            tol = (0.01 if name == "q" else 0.05) * abs(d_o) + 2e-5 * abs(ref[0][2])
            assert abs(d_g - d_o) <= tol, name
        off += steps * -(-o.modules[name].codes.shape[1] // 128)
    assert tr[0] == pytest.approx(o.modules["q"].loss_trace[0][2], rel=1e-4)
    print("loss", g.loss_final, o.loss_final, flush=True)
    assert abs(g.loss_final - o.loss_final) <= 5e-3 * abs(o.loss_final)


def test_decoder_ragged_and_degenerate_shapes(rq, ctx):
    """Edge shapes in one block: plain multi-head attention (n_kv = n_heads), head_dim 32 (one
    value-column tile), 32-token sequences (one attention tile each), d = 264 and f = 392 (column
    blocks of 128, 128 and 8; 128, 128, 128 and 8) and an o projection of 64 columns (one partial
    block, so o takes no Block-GD step).  Without Block-GD every module is GPTQ on its own input
    (module-level bars, down at its no-BGD bar of the decoder tests); with Block-GD the first step
    and the final loss are compared."""
    inp = synth.make_decoder_block(96, 264, 392, 2, 2, 32, 32, seed=13)
    _banner("decoder block, ragged widths, MHA, head_dim 32, 32-token sequences")
    g = _run(rq, ctx, inp, 0, 1e-5)
    o = B.decoder_block_sweep(inp.X, inp.Xhat, _oracle_blk(inp), steps=0)
    _check(g, o, False)
    g = _run(rq, ctx, inp, 2, 1e-5)
    o = B.decoder_block_sweep(inp.X, inp.Xhat, _oracle_blk(inp), steps=2, lr=1e-5)
    tr = g.loss_trace.cpu().numpy()
    print("trace0", tr[0], o.modules["q"].loss_trace[0][2], "loss", g.loss_final, o.loss_final, flush=True)
    assert tr[0] == pytest.approx(o.modules["q"].loss_trace[0][2], rel=1e-4)
    assert abs(g.loss_final - o.loss_final) <= P.LOSS_RTOL * abs(o.loss_final)
    # o (one partial block) and the last block of every module take no Block-GD step
    off = 3 * 2 * 3
    assert np.isnan(tr[off:off + 2]).all()


def test_decoder_lds_attention_ragged_tile_count(rq, ctx):
    """The LDS-staged attention kernels (forward, dS, dQ and dK/dV, which take 4 consecutive
    32-token tiles per block) at a tile count that is not a multiple of 4: 160-token sequences
    (5 tiles, so every sequence's second block has 3 idle waves), 16 sequences of 16 query heads
    over 4 key/value heads of 64, enough blocks that every LDS kernel's launch condition holds.
    q (its gradient through dS and dQ) and then k (through dS and dK), each with one Block-GD step
    per block; k runs teacher-forced on the oracle's quantized q and its input h1, so that q's
    own rounding differences do not reach it.  Module-level bars."""
    inp = synth.make_decoder_block(2560, 1024, 256, 16, 4, 64, 160, seed=17, dense_F=False)
    S, nt = inp.X.shape[0] // inp.seq_len, inp.seq_len // 32
    assert S * inp.n_heads * -(-nt // 4) >= 512 and nt % 4 != 0
    _banner("decoder block, 5-tile sequences on the LDS-staged attention kernels, q and k")
    torch = _torch()
    blk = _oracle_blk(inp)
    o = B.decoder_block_sweep(inp.X, inp.Xhat, blk, steps=1, lr=1e-5, modules=("q", "k"))
    W = {k: np.asarray(v, np.float64) for k, v in blk.weights().items()}
    W["q"] = o.modules["q"].W_hat
    h1 = B.decoder_forward(inp.Xhat, blk, W).h1
    for k, name in enumerate(("q", "k")):
        g = rq.decoder_block_sweep(ctx, _dev(inp.X, True), _dev(inp.Xhat, True), _dev_blk(inp), None,
                                   n_heads=inp.n_heads, n_kv=inp.n_kv, head_dim=inp.head_dim, seq_len=inp.seq_len,
                                   qp=rq.qparams(), bgd=rq.bgd_params(steps=1, lr=1e-5), start=k, n_modules=1,
                                   fixed={"q": _dev(o.modules["q"].W_hat)} if k else None,
                                   x_fixed=_dev(h1, True) if k else None)
        torch.cuda.synchronize()
        met = P.compare(g.modules[name], o.modules[name])
        print(name, met, flush=True)
        assert met["code_identity"] >= P.CODE_IDENTITY, name
        assert met["first_group_agreement"] >= P.CODE_IDENTITY, name
        assert met["group_param_agreement"] >= P.GROUP_AGREEMENT_AFTER_BGD, name
    print("loss", g.loss_final, o.loss_final, flush=True)
    assert abs(g.loss_final - o.loss_final) <= P.LOSS_RTOL * abs(o.loss_final)
