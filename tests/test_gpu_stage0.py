"""GPU parity of the Stage-0 accumulators and of the row-group sweep against the float64 oracle:
the aggregated Fisher (Eq. fisher_full), per-token saliency of each row group with the
Hessian-side clip (Eq. saliency_hessian, Appendix D.1), and quantization with one Hessian per
row group (Alg. 1, Stage 1)."""
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


def _bf16_dev(a):
    torch = _torch()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16).cuda()


def _f32_dev(a):
    torch = _torch()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def _assert_parity(met, loss_gpu, loss_ref, bgd):
    print(met, "loss", loss_gpu, loss_ref, flush=True)
    assert met["code_identity"] >= P.CODE_IDENTITY
    assert met["first_group_agreement"] >= P.CODE_IDENTITY
    assert met["group_param_agreement"] >= (P.GROUP_AGREEMENT_AFTER_BGD if bgd else P.CODE_IDENTITY)
    assert abs(loss_gpu - loss_ref) <= P.LOSS_RTOL * abs(loss_ref)


# ============================================================================ Fisher and saliency

def test_fisher_accumulates_over_token_chunks(rq, ctx):
    torch = _torch()
    T, m = 3001, 300
    G = synth.make_output_grads(T, m, seed=1)
    _banner(f"fisher T={T} m={m}")
    Gd = _bf16_dev(G)
    Facc = torch.zeros((m, m), dtype=torch.float64, device="cuda")
    rq.fisher_accum(ctx, Gd[:1700].contiguous(), Facc)
    rq.fisher_accum(ctx, Gd[1700:].contiguous(), Facc)
    F = torch.empty((m, m), dtype=torch.float32, device="cuda")
    rq.fisher_finish(ctx, Facc, T, F)
    torch.cuda.synchronize()
    ref = oracle.fisher(G.astype(np.float64))
    d = np.sqrt(np.diag(ref))
    # bf16 products are exact; tiles accumulate in float32 over the token chunk
    err = np.abs(F.cpu().numpy().astype(np.float64) - ref) / np.outer(d, d)
    print("max scaled error", err.max(), flush=True)
    assert err.max() <= 3e-5


@pytest.mark.parametrize("T,m,ng,q", [(5000, 300, 4, 0.99), (5000, 300, 4, 0.0), (777, 10, 4, 0.9),
                                      (64, 5, 4, 0.5), (1, 7, 7, 0.99), (4097, 4096, 1, 1.0),
                                      (20000, 1024, 4, 0.99)])
def test_saliency_matches_oracle(rq, ctx, T, m, ng, q):
    G = synth.make_output_grads(T, m, seed=2)
    _banner(f"saliency T={T} m={m} groups={ng} clip={q}")
    got = rq.saliency(ctx, _bf16_dev(G), ng, q).cpu().numpy()
    # the library takes the quantile from the float32 clip_q: the oracle gets the same number
    ref = oracle.saliency(G.astype(np.float64), ng, clip_q=float(np.float32(q)) if q > 0 else None)
    nr = ref.shape[0]
    assert nr == len(oracle.row_groups(m, ng))
    np.testing.assert_array_equal(got[nr:], 0.0)        # empty groups
    # float64 sums in another order, then rounded to float32: at most one float32 step apart
    np.testing.assert_allclose(got[:nr], ref.astype(np.float32), rtol=2.0 ** -23, atol=0)
    if q > 0:
        k = int(np.ceil(np.float64(np.float32(q)) * T))
        for g in range(nr):
            tau = got[g].max()
            assert (got[g] >= tau).sum() >= T - k + 1    # the clipped tail sits on the k-th value


def test_saliency_rejects_bad_arguments(rq, ctx):
    Gd = _bf16_dev(synth.make_output_grads(16, 8, seed=3))
    for ng, q in [(0, 0.9), (9, 0.9), (2, 1.5), (2, -0.1)]:
        with pytest.raises(rq.RealqError) as ei:
            rq.saliency(ctx, Gd, ng, q)
        assert ei.value.code == -1


# ============================================================================ one Hessian per row group

def _layer(rq, ctx, L, steps, lr, S, want=False):
    torch = _torch()
    W0, Xd, Xh, sd, _ = P.to_device(L, torch)
    res = rq.quantize_layer(ctx, W0, Xd, Xh, sd, qp=rq.qparams(), bgd=rq.bgd_params(steps=steps, lr=lr),
                            s_groups=None if S is None else _f32_dev(S), want_H=want, want_U=want)
    torch.cuda.synchronize()
    return res


@pytest.mark.parametrize("steps", [0, 3])
def test_row_groups_match_oracle(rq, ctx, steps):
    L = synth.make_module("single_512", m=200, n=384, T=2048)   # 3 groups of 67, 67, 66 rows
    S = synth.make_group_weights(3, 2048, seed=3)
    _banner(f"row groups m=200 N_g=3 steps={steps}")
    g = _layer(rq, ctx, L, steps, L.lr, S, want=True)
    o = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=steps, lr=L.lr, s_groups=S)
    _assert_parity(P.compare(g, o), g.loss_final, o.loss_final, steps > 0)
    for k in range(3):
        assert P.rel_fro(g.H[k].cpu().numpy().astype(np.float64), o.H[k]) <= P.HESS_RTOL
        np.testing.assert_array_equal(g.dead[k].cpu().numpy().astype(bool), o.dead[k])


def test_one_row_group_is_the_single_hessian_sweep(rq, ctx):
    L = synth.make_module("single_512", m=64, n=256, T=1024)
    _banner("one row group vs the single-Hessian sweep")
    a = _layer(rq, ctx, L, 2, L.lr, None)
    b = _layer(rq, ctx, L, 2, L.lr, L.s[None, :])
    assert (a.codes.cpu() == b.codes.cpu()).all()
    assert (a.W_hat.cpu() == b.W_hat.cpu()).all()
    assert a.loss_final == b.loss_final


def test_dead_column_of_one_row_group(rq, ctx):
    """Column 200 is dead for group 0 only (its saliency vanishes where the column is nonzero) while
    Block-GD (s = None) moves it before block 1: the group's rows still dequantize to exactly 0."""
    torch = _torch()
    L = synth.make_module("single_512", m=64, n=256, T=512)
    X, Xh = L.X.copy(), L.Xhat.copy()
    for a in (X, Xh):
        a[:, 200] = 0.0
        a[:20, 200] = 1.5
    S = np.ones((2, 512), dtype=np.float32)
    S[0, :20] = 0.0
    _banner("dead column in one row group")
    W0 = torch.from_numpy(L.W0).cuda()
    g = rq.quantize_layer(ctx, W0, _bf16_dev(X), _bf16_dev(Xh), None, qp=rq.qparams(),
                          bgd=rq.bgd_params(steps=4, lr=L.lr), s_groups=_f32_dev(S))
    torch.cuda.synchronize()
    o = oracle.quantize_layer(L.W0, X, Xh, None, steps=4, lr=L.lr, s_groups=S)
    assert o.dead[0][200] and not o.dead[1][200]
    assert (g.W_hat.cpu().numpy()[:32, 200] == 0.0).all()
    _assert_parity(P.compare(g, o), g.loss_final, o.loss_final, True)


def test_row_calls_compose_to_the_layer_call(rq, ctx):
    """realq_quantize_block_rows per row group + realq_bgd_lock_block + realq_bgd_step reproduce
    realq_quantize_layer with row groups bit for bit."""
    torch = _torch()
    L = synth.make_module("single_512", m=96, n=384, T=512)
    S = synth.make_group_weights(2, 512, seed=4)
    _banner("row-group calls vs the layer call")
    W0, X, Xh, s, _ = P.to_device(L, torch)
    m, n, T = L.shape
    steps, lr = 2, 1e-3
    ref = _layer(rq, ctx, L, steps, lr, S)
    Sd = _f32_dev(S)
    qp = rq.qparams()
    Us, deads = [], []
    for g in range(2):
        Hacc = torch.zeros((n, n), dtype=torch.float64, device="cuda")
        rq.hessian_accum(ctx, Xh, Sd[g].contiguous(), Hacc)
        U = torch.empty((n, n), dtype=torch.float32, device="cuda")
        dead = torch.empty((n,), dtype=torch.uint8, device="cuda")
        rq.chol_inverse(ctx, Hacc, T, 0.01, U, None, dead)
        Us.append(U)
        deads.append(dead)
    st = rq.BgdState(ctx, W0, X, Xh, s, params=rq.bgd_params(steps=steps, lr=lr))
    W = W0.double()
    codes = torch.empty((m, n), dtype=torch.uint8, device="cuda")
    scales = torch.empty((m, n // 128), dtype=torch.float32, device="cuda")
    zeros = torch.empty((m, n // 128), dtype=torch.uint8, device="cuda")
    groups = rq.row_groups(m, 2)
    for c0 in range(0, n, 128):
        for (r0, r1), U, dead in zip(groups, Us, deads):
            rq.quantize_block_rows(ctx, W, r0, r1, c0, 128, U, dead, qp, codes, scales, zeros, st)
        rq.bgd_lock_block(ctx, st, c0, 128)
        if c0 + 128 < n:
            for _ in range(steps):
                rq.bgd_step(ctx, st, W, c0 + 128, 1.0)
    torch.cuda.synchronize()
    assert (codes.cpu() == ref.codes.cpu()).all()
    assert (W.float().cpu() == ref.W_hat.cpu()).all()
    with pytest.raises(rq.RealqError) as ei:       # locking out of column order
        rq.bgd_lock_block(ctx, st, 0, 128)
    assert ei.value.code == -2
    with pytest.raises(rq.RealqError) as ei:       # rows past m
        rq.quantize_block_rows(ctx, W, 90, 97, 0, 128, Us[0], deads[0], qp, codes, scales, zeros)
    assert ei.value.code == -2
    st.close()


def test_row_groups_reject_more_groups_than_rows(rq, ctx):
    L = synth.make_module("single_512", m=8, n=128, T=64)
    S = synth.make_group_weights(9, 64, seed=5)
    with pytest.raises(rq.RealqError) as ei:
        _layer(rq, ctx, L, 0, 1e-3, S)
    assert ei.value.code == -1


# ============================================================================ Stage 0 into Stage 1

def test_saliency_feeds_the_row_group_sweep(rq, ctx):
    """Gradients -> clipped saliency (0.99) -> N_g = 4 row-group sweep with Block-GD, on the GPU
    and in the oracle from the same gradients."""
    L = synth.make_module("qwen3_0.6b_mlp", "gate", m=256, n=384, T=2048)
    G = synth.make_output_grads(2048, 256, seed=6)
    _banner("stage 0 -> row-group sweep, m=256 N_g=4")
    Sg = rq.saliency(ctx, _bf16_dev(G), 4, 0.99)
    torch = _torch()
    W0, X, Xh, s, _ = P.to_device(L, torch)
    g = rq.quantize_layer(ctx, W0, X, Xh, s, qp=rq.qparams(), bgd=rq.bgd_params(steps=3, lr=L.lr), s_groups=Sg)
    torch.cuda.synchronize()
    S_ref = oracle.saliency(G.astype(np.float64), 4, clip_q=float(np.float32(0.99)))
    o = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=3, lr=L.lr,
                              s_groups=S_ref.astype(np.float32).astype(np.float64))
    _assert_parity(P.compare(g, o), g.loss_final, o.loss_final, True)


def test_row_groups_llama_gate_shape_sampled_rows(rq, ctx):
    """14336x4096 gate projection at 8192 tokens with N_g = 4 saliency Hessians from 8192 x 14336
    gradients; the oracle runs sampled rows of two groups (rows are independent for M = I)."""
    L = synth.make_module("llama3.1_8b_layer", "gate", T=8192)
    m = L.W0.shape[0]
    G = synth.make_output_grads(8192, m, seed=7)
    _banner("row groups llama3.1-8b gate 14336x4096 T=8192 N_g=4")
    torch = _torch()
    Sg = rq.saliency(ctx, _bf16_dev(G), 4, 0.99)
    W0, X, Xh, s, _ = P.to_device(L, torch)
    g = rq.quantize_layer(ctx, W0, X, Xh, s, qp=rq.qparams(), bgd=rq.bgd_params(steps=L.steps, lr=L.lr),
                          s_groups=Sg)
    torch.cuda.synchronize()
    S_ref = oracle.saliency(G.astype(np.float64), 4, clip_q=float(np.float32(0.99))).astype(np.float32)
    np.testing.assert_allclose(Sg.cpu().numpy(), S_ref, rtol=2.0 ** -23, atol=0)
    del G
    rng = np.random.default_rng(9)
    groups = oracle.row_groups(m, 4)
    for k in (0, 3):
        sl = groups[k]
        rows = np.sort(rng.choice(np.arange(sl.start, sl.stop), 3, replace=False))
        o = oracle.quantize_layer(L.W0[rows], L.X, L.Xhat, L.s, steps=L.steps, lr=L.lr,
                                  s_groups=S_ref[k][None, :].astype(np.float64))
        met = P.compare(g, o, rows=rows)
        lg = P.row_loss(g.W_hat.cpu().numpy()[rows], L.W0[rows], L.X, L.Xhat)
        _assert_parity(met, lg, o.loss_final, True)


# ============================================================================ Stage 0 at the full workload sizes

def _device_grads(torch, T, m, seed, chunk=16384):
    """Seeded per-token output gradients [T, m] bf16 drawn on the device (Gaussian x LogNormal(0, 2.3)
    token scale x LogNormal(0, 1.15) channel scale x 1e-3, four tokens x 1e5): the distribution of the
    synthetic Stage-0 inputs at sizes the host would take minutes to draw.  Returns (G, outlier tokens)."""
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    chan = torch.exp(1.15 * torch.randn((1, m), generator=g, device="cuda"))
    G = torch.empty((T, m), dtype=torch.bfloat16, device="cuda")
    for t0 in range(0, T, chunk):
        t1 = min(T, t0 + chunk)
        tok = torch.exp(2.3 * torch.randn((t1 - t0, 1), generator=g, device="cuda"))
        G[t0:t1] = (torch.randn((t1 - t0, m), generator=g, device="cuda") * tok * chan * 1e-3).to(torch.bfloat16)
    idx = torch.randperm(T, generator=g, device="cuda")[:4]
    G[idx] = (G[idx].float() * 1e5).to(torch.bfloat16)
    torch.cuda.synchronize()
    return G, idx.cpu().numpy()


def test_fisher_at_block_output_width_sampled_entries(rq, ctx):
    """Aggregated Fisher of 65536 tokens at the 4096-wide LLaMA-3.1-8B block output in one call; the
    oracle computes the principal submatrix on 160 sampled channels (one in each 32-channel stripe of
    the contraction's tiles, 32 more at random), which spans every pair of output tiles."""
    torch = _torch()
    T, m = 65536, 4096
    _banner(f"fisher full width T={T} m={m}")
    Gd, _ = _device_grads(torch, T, m, seed=31)
    Facc = torch.zeros((m, m), dtype=torch.float64, device="cuda")
    rq.fisher_accum(ctx, Gd, Facc)
    F = torch.empty((m, m), dtype=torch.float32, device="cuda")
    rq.fisher_finish(ctx, Facc, T, F)
    torch.cuda.synchronize()
    idx = P.tile_rows(m, per_tile=1, extra=32, seed=32, tile=32)
    Gs = Gd[:, torch.from_numpy(idx).cuda()].float().cpu().numpy().astype(np.float64)
    del Gd, Facc
    ref = oracle.fisher(Gs)
    got = F.cpu().numpy()[np.ix_(idx, idx)].astype(np.float64)
    d = np.sqrt(np.diag(ref))
    err = np.abs(got - ref) / np.outer(d, d)
    print("max scaled error", err.max(), flush=True)
    # products of bf16 values are exact; each 32768-token chunk (128 Mi elements at 4096 channels)
    # sums in float32 over 2048 MFMA steps of 16 tokens, and |sum_t g_ti g_tj| <= T sqrt(F_ii F_jj)
    # (Cauchy-Schwarz), so the scaled error stays within the summation bound 2048 * 2^-24 plus the
    # final float32 rounding
    assert err.max() <= (32768 // 16 + 1) * 2.0 ** -24


def test_saliency_at_llama_gate_size_sampled_tokens(rq, ctx):
    """Saliency of the LLaMA-3.1-8B gate's 262144 x 14336 output gradients (3.8e9 bf16 values, past
    2^31) in 4 row groups.  Unclipped, 256 sampled tokens and the four outliers match the oracle;
    clipped at 0.99, every token holds min(unclipped, tau) with tau the nearest-rank quantile of the
    unclipped values over all tokens, so the selection is checked exactly at any size."""
    torch = _torch()
    T, m, ng, q = 262144, 14336, 4, 0.99
    _banner(f"saliency full size T={T} m={m} groups={ng}")
    Gd, outl = _device_grads(torch, T, m, seed=33)
    s0 = rq.saliency(ctx, Gd, ng, 0.0).cpu().numpy()
    sq = rq.saliency(ctx, Gd, ng, q).cpu().numpy()
    rng = np.random.default_rng(34)
    toks = np.unique(np.concatenate([rng.choice(T, 256, replace=False), outl, [0, T - 1]]))
    Gs = Gd[torch.from_numpy(toks).cuda()].float().cpu().numpy().astype(np.float64)
    del Gd
    ref = oracle.saliency(Gs, ng).astype(np.float32)
    np.testing.assert_allclose(s0[:, toks], ref, rtol=2.0 ** -23, atol=0)
    k = int(np.ceil(np.float64(np.float32(q)) * T))
    for g in range(ng):
        tau = np.sort(s0[g])[k - 1]
        assert sq[g].max() == tau
        np.testing.assert_array_equal(sq[g], np.minimum(s0[g], tau))
    assert (sq[:, outl] == sq.max(axis=1, keepdims=True)).all()       # the outliers sit on the clip
