"""Layer-sweep benchmark of the REAL-Q HIP library on one MI355X.

One step = one whole per-module sweep (Hessian, inverse factor, every 128-column
block with quantization, OBS compensation, lock and K Block-GD steps, final loss)
of the LLaMA-3.1-8B-shaped gate projection: W 14336 x 4096, 262144 calibration
tokens, W4 g128, 8 BGD steps per block.  Inputs are synthetic, generated on the
device with the workload's distributions, and resident in HBM before timing.
The Block-GD steps stream the residual and gradient GEMMs over all tokens; the
same sweep with the loss and gradient taken through the calibration Gram matrices
is timed once more afterwards and reported under "gram_form" (or, with
--form gram, as the line itself).

Prints one JSON line.  ``--gpus`` above 1 is refused: the build runs on one GPU.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16 = 2.5e15        # MI355X dense bf16 MFMA, FLOP/s
PEAK_HBM = 8.0e12         # MI355X HBM3E, B/s

WORKLOADS = {
    # name: (cfg, module, m, n, T, steps, lr)
    "llama3.1_8b_gate": ("llama3.1_8b_layer", "gate", 14336, 4096, 262144, 8, 1e-5),
    "qwen3_0.6b_gate": ("qwen3_0.6b_mlp", "gate", 3072, 1024, 131072, 8, 3e-4),
    "single_512": ("single_512", "linear", 512, 512, 4096, 4, 1e-3),
    "qwen3_32b_gate": ("qwen3_32b_layer", "gate", 25600, 5120, 262144, 8, 2e-6),
    "llama3.1_70b_gate": ("llama3.1_70b_layer", "gate", 28672, 8192, 262144, 8, 3e-6),
}
# residual and gradient GEMMs streamed over the tokens in chunks of this size (0: all at once)
TOKEN_CHUNK = {"llama3.1_70b_gate": 32768}


def f_alg(m, n, T, K, block=128, xhat_differs=True, Tb=None):
    """Algorithmic FLOPs of the token-streamed sweep (hi/lo split passes not counted); Tb: tokens per
    Block-GD step when each step takes a mini-batch (default all T)."""
    nb = -(-n // block)
    SJ = sum(n - min((b + 1) * block, n) for b in range(nb))
    hess = 2 * n * n * T
    init = 2 * m * n * T if xhat_differs else 0
    lock = 2 * m * (n - min(block, n)) * T
    bgd = K * 4 * m * (T if Tb is None else min(Tb, T)) * SJ
    obs = 2 * m * block * SJ
    return dict(total=hess + init + lock + bgd + obs, resid=K * 2 * m * T * SJ, grad=K * 2 * m * T * SJ, SJ=SJ)


def make_inputs(torch, wl, seed=0):
    """Device-side generation with the workload's distributions (torch Philox)."""
    cfg, module, m, n, T, steps, lr = WORKLOADS[wl]
    import synth
    c = synth.CONFIGS[cfg]
    g = torch.Generator(device="cuda")
    g.manual_seed(seed * 1000 + list(c["modules"]).index(module))
    wdt, wstd = c["w"]
    W0 = torch.randn((m, n), generator=g, device="cuda") * wstd
    if wdt == "bf16":
        W0 = W0.to(torch.bfloat16).float()
    spec = c["x"]
    if spec[0] == "student_t":
        # Student-t with integer nu: z / sqrt(chi2_nu / nu), chi2_nu a sum of nu squared normals, all
        # drawn from the seeded generator so the inputs do not depend on earlier random draws
        nu = int(spec[1])
        assert nu == spec[1], "integer degrees of freedom"
        z = torch.randn((T, n), generator=g, device="cuda")
        chi = (torch.randn((T, nu), generator=g, device="cuda") ** 2).sum(dim=1, keepdim=True)
        X32 = z * torch.sqrt(nu / chi)
    else:
        X32 = torch.randn((T, n), generator=g, device="cuda")
        k = int(spec[1]) if spec[0] == "outlier_count" else max(1, int(round(spec[1] * n)))
        idx = torch.randperm(n, generator=g, device="cuda")[:k]
        X32[:, idx] *= spec[2]
    noise = torch.randn((T, n), generator=g, device="cuda")
    kind, amp = c["xhat"]
    Xh32 = X32 + amp * noise if kind == "additive" else X32 * (1 + amp * noise)
    del noise
    X = X32.to(torch.bfloat16)
    del X32
    Xh = Xh32.to(torch.bfloat16)
    del Xh32
    s = None
    if c["s"] == "absnormal":
        s = torch.randn((T,), generator=g, device="cuda").abs()
    elif c["s"] == "lognormal":
        s = torch.randn((T,), generator=g, device="cuda").exp()
    torch.cuda.synchronize()
    return W0.contiguous(), X.contiguous(), Xh.contiguous(), s


def _host_info():
    """CPU model, usable cores and the BLAS numpy calls (recorded with the CPU baseline)."""
    import numpy as np
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    blas = "unknown"
    try:
        cfg = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        blas = f"{cfg.get('name')} {cfg.get('version')}"
    except Exception:
        pass
    threads = None
    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"),
                      default=None)
    except Exception:
        pass
    return model, len(os.sched_getaffinity(0)), blas, threads


def cpu_baseline(wl, hess_tokens=32768, rows=256, tokens=16384):
    """The oracle on the machine's host cores, timed phase by phase at the workload's shape: the
    Hessian on a slice of the calibration tokens (full n), damping and the inverse factor at full
    n, and column block 0 with its K Block-GD steps on a sample of rows and tokens (full n).  The
    oracle's own floating-point rate over these phases then prices the workload's algorithmic
    FLOPs: the result is an extrapolation (a full sweep is hours on a host)."""
    import numpy as np
    import synth
    import oracle
    cfg, module, m, n, T, steps, lr = WORKLOADS[wl]
    model, cores, blas, threads = _host_info()
    Th = min(hess_tokens, T)
    Ts = min(tokens, T)
    r = min(rows, m)
    L = synth.make_module(cfg, module, m=r, n=n, T=max(Th, Ts))
    X, Xh = L.X.astype(np.float64), L.Xhat.astype(np.float64)
    qp = oracle.QParams()
    # 1. Hessian (2 n^2 Th)
    t0 = time.perf_counter()
    H = oracle.hessian(Xh[:Th], None if L.s is None else L.s[:Th])
    t_h = time.perf_counter() - t0
    # 2. damping and the inverse factor (about 2 n^3 for the inverse, n^3 / 3 for the factor)
    t0 = time.perf_counter()
    Hd, _ = oracle.damp_hessian(H, qp.damp)
    oracle.inverse_factor(Hd)
    t_c = time.perf_counter() - t0
    # 3. column block 0 (search, GPTQ, trailing update) and its K Block-GD steps
    t0 = time.perf_counter()
    oracle.quantize_layer(L.W0, X[:Ts], Xh[:Ts], None if L.s is None else L.s[:Ts],
                          qp=oracle.QParams(block=n), steps=0)   # one block of n columns: search + GPTQ
    t_q = time.perf_counter() - t0
    t0 = time.perf_counter()
    sw = None if L.s is None else L.s[:Ts]
    W = L.W0.astype(np.float64)
    J = slice(qp.block, n)
    mA = np.zeros((r, n - qp.block))
    vA = np.zeros_like(mA)
    for k in range(steps):
        R = oracle.residual(W, L.W0, X[:Ts], Xh[:Ts])
        G = oracle.surrogate_grad(R, sw, None, Xh[:Ts, J], Ts)
        W[:, J], mA, vA = oracle.adam_update(W[:, J], G, mA, vA, k + 1, lr)
    t_b = time.perf_counter() - t0
    # floating-point work of the timed phases (the oracle's own: its residual is the full forward)
    nJ = n - qp.block
    fl = (2.0 * n * n * Th + 2.0 * n ** 3 + n ** 3 / 3.0
          + steps * (4.0 * r * n * Ts + 2.0 * r * Ts * nJ))
    t_timed = t_h + t_c + t_b
    rate = fl / t_timed
    # the search and GPTQ are not FLOP-shaped: scaled by rows and column blocks instead
    t_quant_full = t_q * (m / r)
    t_full = f_alg(m, n, T, steps)["total"] / rate + t_quant_full
    return {"value": n / t_full, "unit": "columns/s", "cores": int(cores), "kind": "oracle", "extrapolated": True,
            "cpu": model, "blas": blas, "blas_threads": threads,
            "sample": f"oracle phases at n={n}: Hessian on {Th} of {T} tokens {t_h:.1f} s; damping + inverse "
                      f"factor {t_c:.1f} s; block 0 of {r} of {m} rows: search + GPTQ of all {n} columns "
                      f"{t_q:.1f} s, {steps} Block-GD steps on {Ts} tokens {t_b:.1f} s; oracle rate "
                      f"{rate / 1e9:.1f} GFLOP/s fp64 over the FLOP-shaped phases, the algorithmic FLOPs of the "
                      f"full sweep priced at it plus the search and GPTQ scaled by rows: {t_full:.0f} s per "
                      f"sweep (extrapolated)"}


def output_grads(torch, T, m, seed=1, chunk=16384):
    """Device-side stand-in for per-token output gradients [T, m] bf16 with the distribution the
    synthetic Stage-0 inputs use: Gaussian x LogNormal(0, 2.3) token scale x LogNormal(0, 1.15)
    channel scale, four tokens x 1e5, scaled by 1e-3."""
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
    return G


def stage0(torch, rq, ctx, W0, X, Xh, s, qp, bgd, m, n, T, n_groups=4, fisher_tokens=65536, d_model=4096):
    """Stage-0 accumulators and the row-group sweep on the bench inputs:
    saliency of the module's output gradients over all T tokens (HBM-bound: 2 B read per gradient),
    the aggregated Fisher at the 4096-wide block output on a 65536-token batch (MFMA: 2 T d^2), and
    the sweep with N_g = 4 saliency Hessians."""
    out = {}
    G = output_grads(torch, T, m)
    S = rq.saliency(ctx, G, n_groups, 0.99)        # warm-up (workspaces)
    ctx.reset_timing()
    S = rq.saliency(ctx, G, n_groups, 0.99, out=S)
    torch.cuda.synchronize()
    _, ms = ctx.kernel_time("saliency")
    by = 2.0 * T * m
    out["saliency"] = {"tokens": T, "m": m, "groups": n_groups, "clip": 0.99, "ms": ms,
                       "GB_per_s": by / (ms / 1e3) / 1e9, "frac_hbm": by / (ms / 1e3) / PEAK_HBM}
    del G
    Gb = output_grads(torch, fisher_tokens, d_model, seed=2)
    F_acc = torch.zeros((d_model, d_model), dtype=torch.float64, device="cuda")
    rq.fisher_accum(ctx, Gb, F_acc)                 # warm-up
    F_acc.zero_()
    ctx.reset_timing()
    rq.fisher_accum(ctx, Gb, F_acc)
    torch.cuda.synchronize()
    _, ms = ctx.kernel_time("hessian")
    fl = 2.0 * fisher_tokens * d_model * d_model
    out["fisher"] = {"tokens": fisher_tokens, "d": d_model, "ms": ms, "TFLOP_per_s": fl / (ms / 1e3) / 1e12,
                     "frac_bf16_peak": fl / (ms / 1e3) / PEAK_BF16}
    del Gb, F_acc
    o = rq.quantize_layer(ctx, W0, X, Xh, s, qp=qp, bgd=bgd, s_groups=S)         # warm-up (workspaces)
    o = rq.quantize_layer(ctx, W0, X, Xh, s, qp=qp, bgd=bgd, s_groups=S, out=o)
    print(f"[bench] row-group sweep (N_g = {n_groups}): {o.ms_total:.1f} ms, loss {o.loss_final:.6g}",
          file=sys.stderr, flush=True)
    out["row_group_sweep"] = {"groups": n_groups, "ms_per_step": o.ms_total, "columns_per_s": n / (o.ms_total / 1e3),
                              "loss_final": o.loss_final}
    return out


def block_f_alg(T, d, f, block, steps, window, dense):
    """Algorithmic FLOPs of the Block-GD steps of realq_mlp_block_sweep (the block forward, the
    surrogate and the backward to one module's trailing columns; the next block's forward and
    backward when the window blends it in)."""
    tdf, tdd = 2.0 * T * d * f, 2.0 * T * d * d
    total = 0.0
    b_global = 0
    for mod, (rows, cols) in enumerate(((f, d), (f, d), (d, f))):
        nb = -(-cols // block)
        for b in range(nb):
            b_global += 1
            if b == nb - 1:
                continue
            nJ = cols - (b + 1) * block
            per = (tdf if mod < 2 else 0.0) + tdf + (tdd if dense else 0.0)   # a or b; out; F dy
            per += (tdf if mod < 2 else 0.0) + 2.0 * rows * nJ * T             # dz = g Wd; gradient
            if window and b_global > 1:                                         # alpha < 1
                per += 3 * tdf + (tdd if dense else 0.0) + tdf + 2 * tdf        # next block fwd, F, dz2, du2
            total += steps * per
    return total


def decoder_f_alg(T, d, f, H, Hkv, hd, L, block, steps, window, dense):
    """Algorithmic FLOPs of the Block-GD steps of realq_decoder_block_sweep, split into the
    projection and MLP GEMMs and the causal attention (QK^T and PV forward; dP, dQ, dK and dV
    backward, each 2 T H hd (L + 1) / 2; all on bf16 MFMA)."""
    Hq, Hk = H * hd, Hkv * hd
    tdf, tdd = 2.0 * T * d * f, 2.0 * T * d * d
    att = 2.0 * T * H * hd * (L + 1) / 2.0
    qkv = 2.0 * T * d * (Hq + 2 * Hk)
    oo = 2.0 * T * Hq * d
    proj = {"q": 2.0 * T * d * Hq, "k": 2.0 * T * d * Hk, "v": 2.0 * T * d * Hk}
    shapes = (("q", Hq, d), ("k", Hk, d), ("v", Hk, d), ("o", d, Hq), ("gate", f, d), ("up", f, d), ("down", d, f))
    gemm = attn = 0.0
    b_global = 0
    for name, rows, cols in shapes:
        nb = -(-cols // block)
        for b in range(nb):
            b_global += 1
            if b == nb - 1:
                continue
            nJ = cols - (b + 1) * block
            g = a = 0.0
            # forward from this module's stage
            if name in proj:
                g += proj[name] + oo + 3 * tdf
                a += 2 * att
            elif name == "o":
                g += oo + 3 * tdf
            elif name in ("gate", "up"):
                g += 2 * tdf
            else:
                g += tdf
            g += tdd if dense else 0.0                      # F dy
            # backward to this module's output
            if name in ("gate", "up"):
                g += tdf
            elif name == "o" or name in proj:
                g += 3 * tdf                                # dz, du
                if name in proj:
                    g += oo
                    a += 4 * att
            g += 2.0 * rows * nJ * T                        # the gradient of the trailing columns
            if window and b_global > 1:                     # the next block: forward, F, backward to x
                g += qkv + oo + 3 * tdf + (tdd if dense else 0.0) + 3 * tdf + oo + qkv
                a += 6 * att
            gemm += steps * g
            attn += steps * a
    return gemm, attn


def mlp_block(torch, rq, ctx, qp, T=8192, d=4096, f=14336, steps=8, lr=1e-5):
    """The block-output surrogate sweep of a LLaMA-3.1-8B-shaped MLP block (d 4096, f 14336) on
    8192 tokens with a dense 4096 x 4096 block-output metric and the next block blended in."""
    g = torch.Generator(device="cuda")
    g.manual_seed(77)

    def w(shape, std=0.02):
        return (torch.randn(shape, generator=g, device="cuda") * std).to(torch.bfloat16).float().contiguous()

    def metric():
        A = torch.randn((d, 2 * d), generator=g, device="cuda")
        return (A @ A.T / (2 * d)).contiguous()

    X = (torch.randn((T, d), generator=g, device="cuda")).to(torch.bfloat16).contiguous()
    Xh = (X.float() * (1 + 0.01 * torch.randn((T, d), generator=g, device="cuda"))).to(torch.bfloat16).contiguous()
    gamma = (1 + 0.1 * torch.randn((d,), generator=g, device="cuda")).contiguous()
    blk = (gamma, w((f, d)), w((f, d)), w((d, f)), metric())
    nxt = ((1 + 0.1 * torch.randn((d,), generator=g, device="cuda")).contiguous(), w((f, d)), w((f, d)),
           w((d, f)), metric())
    bgd = rq.bgd_params(steps=steps, lr=lr)
    ctx.reset_timing()
    r = rq.mlp_block_sweep(ctx, X, Xh, *blk, nxt, window=True, qp=qp, bgd=bgd)
    nst, st_ms = ctx.kernel_time("block_step")
    fl = block_f_alg(T, d, f, qp.block, steps, True, True)
    print(f"[bench] mlp block sweep: {r.ms_total:.1f} ms, loss {r.loss_final:.6g}", file=sys.stderr, flush=True)
    return {"tokens": T, "d": d, "f": f, "bgd_steps": steps, "window": True, "dense_metric": True,
            "ms_total": r.ms_total, "loss_final": r.loss_final, "block_steps": nst,
            "block_step_ms_total": st_ms, "block_step_tflops_alg": fl / (st_ms / 1e3) / 1e12 if st_ms > 0 else None,
            "frac_bf16_peak_alg": fl / (st_ms / 1e3) / PEAK_BF16 if st_ms > 0 else None,
            "columns_per_s": (2 * d + f) / (r.ms_total / 1e3)}


def decoder_block(torch, rq, ctx, qp, T=8192, d=4096, f=14336, H=32, Hkv=8, hd=128, L=2048, steps=2, lr=1e-5):
    """The block-output surrogate sweep of a LLaMA-3.1-8B-shaped decoder block (d 4096, 32 query
    and 8 key/value heads of 128, f 14336) on 8192 tokens in sequences of 2048, with a dense
    4096 x 4096 block-output metric, the next decoder block blended in, and 2 Block-GD steps per
    column block (8 for the MLP block: the decoder's 304 column blocks each take a forward and
    backward through attention and the next block)."""
    g = torch.Generator(device="cuda")
    g.manual_seed(78)
    Hq, Hk = H * hd, Hkv * hd

    def w(shape, std=0.02):
        return (torch.randn(shape, generator=g, device="cuda") * std).to(torch.bfloat16).float().contiguous()

    def block():
        A = torch.randn((d, 2 * d), generator=g, device="cuda")
        return {"gamma1": (1 + 0.1 * torch.randn((d,), generator=g, device="cuda")).contiguous(),
                "Wq": w((Hq, d), 0.04), "Wk": w((Hk, d), 0.04), "Wv": w((Hk, d)), "Wo": w((d, Hq)),
                "gamma2": (1 + 0.1 * torch.randn((d,), generator=g, device="cuda")).contiguous(),
                "Wg": w((f, d)), "Wu": w((f, d)), "Wd": w((d, f)), "F": (A @ A.T / (2 * d)).contiguous()}

    X = (torch.randn((T, d), generator=g, device="cuda")).to(torch.bfloat16).contiguous()
    Xh = (X.float() * (1 + 0.01 * torch.randn((T, d), generator=g, device="cuda"))).to(torch.bfloat16).contiguous()
    blk, nxt = block(), block()
    bgd = rq.bgd_params(steps=steps, lr=lr)
    ctx.reset_timing()
    r = rq.decoder_block_sweep(ctx, X, Xh, blk, nxt, n_heads=H, n_kv=Hkv, head_dim=hd, seq_len=L, window=True,
                               qp=qp, bgd=bgd)
    nst, st_ms = ctx.kernel_time("block_step")
    nat, at_ms = ctx.kernel_time("attention")
    fl_gemm, fl_att = decoder_f_alg(T, d, f, H, Hkv, hd, L, qp.block, steps, True, True)
    print(f"[bench] decoder block sweep: {r.ms_total:.1f} ms, loss {r.loss_final:.6g}", file=sys.stderr, flush=True)
    gemm_ms = st_ms - at_ms
    return {"tokens": T, "d": d, "f": f, "n_heads": H, "n_kv": Hkv, "head_dim": hd, "seq_len": L, "bgd_steps": steps,
            "window": True, "dense_metric": True, "ms_total": r.ms_total, "loss_final": r.loss_final,
            "block_steps": nst, "block_step_ms_total": st_ms, "attention_launch_groups": nat,
            "attention_ms_total": at_ms,
            "attention_tflops_alg": fl_att / (at_ms / 1e3) / 1e12 if at_ms > 0 else None,
            "attention_frac_bf16_peak_alg": fl_att / (at_ms / 1e3) / PEAK_BF16 if at_ms > 0 else None,
            "gemm_tflops_alg": fl_gemm / (gemm_ms / 1e3) / 1e12 if gemm_ms > 0 else None,
            "gemm_frac_bf16_peak_alg": fl_gemm / (gemm_ms / 1e3) / PEAK_BF16 if gemm_ms > 0 else None,
            "columns_per_s": (3 * d + Hq + 2 * d + f) / (r.ms_total / 1e3)}


# Further modules of the layer workloads, one sweep each at full size (name: cfg, module, T, token
# chunk, window partner module or None): the Qwen3-32B q projection with its dense Wishart metric,
# the LLaMA-3.1-8B q projection with o as its window partner, the LLaMA-3.1-8B down projection
# (inverse factor at n = 14336) at 8192 tokens, and the Qwen3-0.6B down projection at its full
# 131072 tokens.
CONFIG_LEGS = {
    "qwen3_32b_q_dense_metric": ("qwen3_32b_layer", "q", 262144, 0, None),
    "llama3.1_8b_q_window_o": ("llama3.1_8b_layer", "q", 262144, 0, "o"),
    "llama3.1_8b_down_T8192": ("llama3.1_8b_layer", "down", 8192, 0, None),
    "qwen3_0.6b_down": ("qwen3_0.6b_mlp", "down", 131072, 0, None),
}


def config_legs(torch, rq, ctx, qp):
    """One warm-up and one timed sweep of each CONFIG_LEGS module (inputs generated on the device
    with the workload's distributions); F_alg counts K 2 m^2 SJ per dense metric or partner term."""
    import synth
    out = {}
    for name, (cfg, module, T, chunk, partner) in CONFIG_LEGS.items():
        c = synth.CONFIGS[cfg]
        m, n = c["modules"][module]
        K, lr = c["steps"], c["lr"]
        WORKLOADS["_leg"] = (cfg, module, m, n, T, K, lr)
        W0, X, Xh, s = make_inputs(torch, "_leg")
        M = P = None
        window = None
        g = torch.Generator(device="cuda")
        g.manual_seed(4242)
        if c["M"] is not None and c["M"][1] == m:
            A = torch.randn((m, 2 * m), generator=g, device="cuda")
            M = (A @ A.T / (2 * m)).contiguous()
            del A
        if partner is not None:
            mp, _ = c["modules"][partner]
            Wn = (torch.randn((mp, m), generator=g, device="cuda") * c["w"][1]).to(torch.bfloat16).float().contiguous()
            P = torch.empty((m, m), dtype=torch.float32, device="cuda")
            rq.pullback_metric(ctx, Wn, P)
            del Wn
            window = (0, -(-n // qp.block))
        bgd = rq.bgd_params(steps=K, lr=lr, tok_chunk=chunk)
        o = rq.quantize_layer(ctx, W0, X, Xh, s, M, P, qp=qp, bgd=bgd, window=window)
        ctx.set_timing(True)
        ctx.reset_timing()
        o = rq.quantize_layer(ctx, W0, X, Xh, s, M, P, qp=qp, bgd=bgd, window=window, out=o)
        kt = {kn: ctx.kernel_time(kn)[1] for kn in ("resid", "grad", "resid_inc", "grad_inc", "metric", "adam",
                                                          "lock", "quantize", "chol", "init", "dense_loss")}
        fa = f_alg(m, n, T, K)
        dense_terms = (1 if M is not None else 0) + (1 if P is not None else 0)
        fl = fa["total"] + dense_terms * K * 2.0 * m * m * fa["SJ"]
        print(f"[bench] {name}: {m}x{n} T={T}: {o.ms_total:.1f} ms, loss {o.loss_final:.6g}", file=sys.stderr,
              flush=True)
        out[name] = {"m": m, "n": n, "tokens": T, "bgd_steps": K, "dense_metric": M is not None,
                     "window_partner": partner, "ms": o.ms_total, "columns_per_s": n / (o.ms_total / 1e3),
                     "tflops_alg": fl / (o.ms_total / 1e3) / 1e12, "frac_bf16_peak_alg": fl / (o.ms_total / 1e3) / PEAK_BF16,
                     "loss_final": o.loss_final, "kernel_ms": {k: round(v, 2) for k, v in kt.items() if v > 0}}
        if kt["metric"] > 0:
            # the dense-metric products: K 2 m^2 SJ algorithmic FLOPs, three bf16 MFMA passes executed
            fm = K * 2.0 * m * m * fa["SJ"]
            out[name]["metric_tflops_alg"] = fm / (kt["metric"] / 1e3) / 1e12
        del W0, X, Xh, s, M, P, o
        torch.cuda.empty_cache()
    WORKLOADS.pop("_leg", None)
    return out


def next_legs(torch, rq, ctx, W0, X, Xh, s, m, n, T, K, lr, workload, batch=65536):
    """One sweep each (after the headline, so the workspaces exist) of the extensions beyond the
    plain sweep, on the headline's own inputs: Block-GD on mini-batches of 65536 tokens per Adam
    step (Sec. 4.3; the paper's 32 calibration sequences of 2048 tokens), and the symmetric per-row
    W4 quantizer of the paper's main tables; then the Qwen3-0.6B gate (3072 x 1024, 131072 tokens)
    with mini-batches and the output-perturbation clip a_loss_clip = 0.95 (Appendix D.1's setting
    for the small Qwen3 models).  F_alg counts the Block-GD GEMMs over the tokens each step takes."""
    out = {}

    def one(name, W0_, X_, Xh_, s_, m_, n_, T_, K_, lr_, qp_, bgd_, Tb):
        o = rq.quantize_layer(ctx, W0_, X_, Xh_, s_, qp=qp_, bgd=bgd_)
        fl = f_alg(m_, n_, T_, K_, Tb=Tb)["total"]
        print(f"[bench] {name}: {o.ms_total:.1f} ms, loss {o.loss_final:.6g}", file=sys.stderr, flush=True)
        out[name] = {"m": m_, "n": n_, "tokens": T_, "tokens_per_step": min(Tb, T_), "bgd_steps": K_,
                     "ms": o.ms_total, "columns_per_s": n_ / (o.ms_total / 1e3),
                     "tflops_alg": fl / (o.ms_total / 1e3) / 1e12, "loss_final": o.loss_final}

    one(f"{workload}_minibatch{batch}", W0, X, Xh, s, m, n, T, K, lr, rq.qparams(),
        rq.bgd_params(steps=K, lr=lr, batch=batch), batch)
    one(f"{workload}_sym_per_row_w4", W0, X, Xh, s, m, n, T, K, lr, rq.qparams(sym=True, group=0),
        rq.bgd_params(steps=K, lr=lr), T)
    WORKLOADS["_leg"] = ("qwen3_0.6b_mlp", "gate", 3072, 1024, 131072, 8, 3e-4)
    try:
        W0q, Xq, Xhq, sq = make_inputs(torch, "_leg")
    finally:
        WORKLOADS.pop("_leg", None)
    one(f"qwen3_0.6b_gate_minibatch{batch}_clip0.95", W0q, Xq, Xhq, sq, 3072, 1024, 131072, 8, 3e-4, rq.qparams(),
        rq.bgd_params(steps=8, lr=3e-4, batch=batch, loss_clip=0.95), batch)
    return out


LAYER_ORDER = ("q", "k", "v", "o", "gate", "up", "down")
LAYER_PARTNERS = {"q": ("o",), "o": ("gate", "up")}


def whole_layer(torch, rq, ctx, qp, cfg="llama3.1_8b_layer"):
    """The seven modules of one synthetic decoder layer at full size, in the order q, k, v, o, gate,
    up, down, each on the hand-off of the module before it (X_o = X W_q^T, X_gate,up = X_o W_o^T,
    X_down = SiLU(X W_gate^T) * (X W_up^T), the quantized path with the quantized weights, all in
    bf16), q and o with their consumers' pull-back metric over the window of their own blocks.
    One pass; each module's time is the library's own (Hessian, factorisation, the whole sweep,
    final loss), the hand-offs are timed apart."""
    import synth
    c = synth.CONFIGS[cfg]
    T, K, lr = c["T"], c["steps"], c["lr"]
    shapes = {k: tuple(v) for k, v in c["modules"].items()}
    WORKLOADS["_leg"] = (cfg, "q", *shapes["q"], T, K, lr)
    W0q, X0, Xh0, s = make_inputs(torch, "_leg")
    WORKLOADS.pop("_leg", None)
    g = torch.Generator(device="cuda")
    g.manual_seed(777)
    W0 = {"q": W0q}
    for name in LAYER_ORDER[1:]:
        W = torch.randn(shapes[name], generator=g, device="cuda") * c["w"][1]
        W0[name] = W.to(torch.bfloat16).float().contiguous()
    bf = torch.bfloat16
    inputs = {k: (X0, Xh0) for k in ("q", "k", "v")}
    out, gate_hat = {}, None
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    handoff_ms = 0.0
    fl_total = 0.0
    for name in LAYER_ORDER:
        m, n = shapes[name]
        X, Xh = inputs[name]
        P, window = None, None
        if name in LAYER_PARTNERS:
            P = torch.empty((m, m), dtype=torch.float32, device="cuda")
            for i, partner in enumerate(LAYER_PARTNERS[name]):
                rq.pullback_metric(ctx, W0[partner], P, accumulate=i > 0)
            window = (0, -(-n // qp.block))
        bgd = rq.bgd_params(steps=K, lr=lr, tok_chunk=TOKEN_CHUNK.get(f"{cfg}:{name}", 0))
        r = rq.quantize_layer(ctx, W0[name], X, Xh, s, None, P, qp=qp, bgd=bgd, window=window)
        fa = f_alg(m, n, T, K)
        fl = fa["total"] + (K * 2.0 * m * m * fa["SJ"] if P is not None else 0.0)
        fl_total += fl
        out[name] = {"m": m, "n": n, "ms": r.ms_total, "tflops_alg": fl / (r.ms_total / 1e3) / 1e12,
                     "loss_final": r.loss_final}
        print(f"[bench] layer {name}: {m}x{n} {r.ms_total:.1f} ms, loss {r.loss_final:.6g}", file=sys.stderr,
              flush=True)
        ev0.record()
        if name in ("q", "o"):
            Y = torch.empty((T, m), dtype=bf, device="cuda")
            Yh = torch.empty_like(Y)
            rq.handoff(ctx, W0[name], X, Y)
            rq.handoff(ctx, r.W_hat, Xh, Yh)
            if name == "q":
                inputs["o"] = (Y, Yh)
            else:
                inputs["gate"] = inputs["up"] = (Y, Yh)
        elif name == "gate":
            gate_hat = r.W_hat
        elif name == "up":
            Xg, Xhg = inputs["gate"]
            Y = torch.empty((T, m), dtype=bf, device="cuda")
            Yh = torch.empty_like(Y)
            rq.handoff(ctx, W0["gate"], Xg, Y, Wb=W0["up"])
            rq.handoff(ctx, gate_hat, Xhg, Yh, Wb=r.W_hat)
            inputs["down"] = (Y, Yh)
            del inputs["gate"], inputs["up"]
        ev1.record()
        torch.cuda.synchronize()
        handoff_ms += ev0.elapsed_time(ev1)
        del r, P
        torch.cuda.empty_cache()
    total = sum(v["ms"] for v in out.values()) + handoff_ms
    return {"config": cfg, "tokens": T, "bgd_steps": K, "modules": out, "handoff_ms": handoff_ms,
            "ms_total": total, "flops_alg": fl_total, "tflops_alg": fl_total / (total / 1e3) / 1e12,
            "frac_bf16_peak_alg": fl_total / (total / 1e3) / PEAK_BF16}


GEMM_SOURCE = os.path.join(ROOT, "paper_2609_00049_amd", "csrc", "gemm_bf16.hip")
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "gemm_llama8b_gate_traffic.txt")


def gemm_source_sha1():
    import hashlib
    with open(GEMM_SOURCE, "rb") as f:
        return hashlib.sha1(f.read()).hexdigest()


def measured_traffic(workload, kernel):
    """HBM bytes per launch of the residual ("resid") or gradient ("grad") GEMM from the committed
    rocprofv3 counter summary, or None when the summary is missing, covers another workload, or
    predates the current GEMM source."""
    try:
        kv = {}
        for line in open(TRAFFIC_PROFILE):
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
        if kv.get("workload") != workload or kv.get("gemm_source_sha1") != gemm_source_sha1():
            return None
        return float(kv[f"traffic_bytes_per_launch.{kernel}"])
    except (OSError, KeyError, ValueError):
        return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="llama3.1_8b_gate", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--tok-chunk", type=int, default=None,
                    help="stream the tokens through the Block-GD GEMMs in chunks of this many (default: the "
                         "workload's own setting, 0 = all tokens at once)")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="run one plain device copy of this many bytes first (calibrates HBM byte counters)")
    ap.add_argument("--form", default="tokens", choices=("tokens", "gram"),
                    help="BGD evaluation: residual/gradient GEMMs over all tokens every step (the step of the "
                         "headline metric), or the same loss and gradient through the calibration Gram matrices")
    ap.add_argument("--no-increment", action="store_true",
                    help="run every Block-GD step with both passes (resid_increment = 0): the sweep without "
                         "the increments of a column block's later steps")
    ap.add_argument("--no-gram-line", action="store_true",
                    help="with --form tokens, skip the extra untimed Gram-form sweep reported under gram_form")
    ap.add_argument("--no-stage0", action="store_true",
                    help="skip the Stage-0 accumulator timings and the N_g = 4 row-group sweep (stage0)")
    ap.add_argument("--no-block", action="store_true",
                    help="skip the block-output surrogate sweep of a LLaMA-3.1-8B-shaped MLP block (mlp_block)")
    ap.add_argument("--no-decoder", action="store_true",
                    help="skip the block-output surrogate sweep of a LLaMA-3.1-8B-shaped decoder block "
                         "(decoder_block)")
    ap.add_argument("--no-next", action="store_true",
                    help="skip the mini-batch, symmetric-quantizer and clip sweeps (also skipped with --no-configs)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the sweeps of the further modules (dense metric, window partner, down projections)")
    ap.add_argument("--only", choices=("stage0", "block", "decoder", "configs", "layer"),
                    help="run only that part (for per-part kernel profiles) and print its object")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs the sweep on one GPU; --gpus {args.gpus} is not supported "
              f"(the row-sharded multi-GPU design is documented but not built)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_00049_amd import realq as rq

    torch.cuda.set_device(0)
    cfg, module, m, n, T, K, lr = WORKLOADS[args.workload]
    if args.only == "block":
        ctx = rq.Context()
        ctx.set_timing(True)
        print(json.dumps({"mlp_block": mlp_block(torch, rq, ctx, rq.qparams())}), flush=True)
        return
    if args.only == "decoder":
        ctx = rq.Context()
        ctx.set_timing(True)
        print(json.dumps({"decoder_block": decoder_block(torch, rq, ctx, rq.qparams())}), flush=True)
        return
    if args.only == "layer":
        ctx = rq.Context()
        print(json.dumps({"whole_layer": whole_layer(torch, rq, ctx, rq.qparams())}), flush=True)
        return
    if args.only == "configs":
        ctx = rq.Context()
        print(json.dumps({"configs": config_legs(torch, rq, ctx, rq.qparams())}), flush=True)
        return
    print(f"[bench] generating {args.workload}: m={m} n={n} T={T} K={K}", file=sys.stderr, flush=True)
    W0, X, Xh, s = make_inputs(torch, args.workload)
    if args.copy_bytes > 0:
        src = torch.ones(args.copy_bytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] calibration copy of {args.copy_bytes} bytes done", file=sys.stderr, flush=True)
        del src, dst
    ctx = rq.Context()
    qp = rq.qparams()
    form = rq.BGD_GRAM if args.form == "gram" else rq.BGD_TOKENS
    tok_chunk = TOKEN_CHUNK.get(args.workload, 0) if args.tok_chunk is None else args.tok_chunk
    bgd = rq.bgd_params(steps=K, lr=lr, form=form, tok_chunk=tok_chunk, resid_increment=0 if args.no_increment else 1)
    if args.only == "stage0":
        ctx.set_timing(True)
        print(json.dumps({"stage0": stage0(torch, rq, ctx, W0, X, Xh, s, qp, rq.bgd_params(steps=K, lr=lr), m, n,
                                           T)}), flush=True)
        return
    out = None
    for w in range(args.warmup):
        out = rq.quantize_layer(ctx, W0, X, Xh, s, qp=qp, bgd=bgd, out=out)
        print(f"[bench] warmup {w}: {out.ms_total:.1f} ms", file=sys.stderr, flush=True)
    ctx.set_timing(True)
    ctx.reset_timing()
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    sweep_ms = []
    for k in range(args.steps):
        out = rq.quantize_layer(ctx, W0, X, Xh, s, qp=qp, bgd=bgd, out=out)
        sweep_ms.append(out.ms_total)
        print(f"[bench] step {k}: {out.ms_total:.1f} ms, loss {out.loss_final:.6g}", file=sys.stderr, flush=True)
    ev1.record()
    torch.cuda.synchronize()
    total_ms = ev0.elapsed_time(ev1)
    ms_per_step = total_ms / args.steps

    fa = f_alg(m, n, T, K)
    kt = {name: ctx.kernel_time(name) for name in ("resid", "grad", "resid_inc", "grad_inc", "quantize", "obs",
                                                    "lock", "adam", "hessian", "chol", "init", "gram", "gram_step")}
    # the residual (gradient) GEMM: a column block's first step ("resid") and its later steps,
    # which take the residual as an increment where the library allows it ("resid_inc")
    both = {k: (kt[k][0] + kt[k + "_inc"][0], kt[k][1] + kt[k + "_inc"][1]) for k in ("resid", "grad")}
    increments = kt["resid_inc"][0] > 0
    if args.form == "tokens":
        # dominant kernel by total time over the timed steps
        dom = max(("resid", "grad"), key=lambda k: both[k][1])
        dom_flops = fa[dom] * args.steps
        launches, dom_ms = both[dom]
    else:
        # D G_hh over all n columns every step (the loss trace is recorded), m x n x n
        dom = "gram_step"
        dom_flops = 2.0 * m * n * n * kt[dom][0]
        launches, dom_ms = kt[dom]
    achieved = dom_flops / (dom_ms / 1e3) if dom_ms > 0 else math.nan
    # the achievable MFMA rate of this GPU (register-resident loop), beside the data-sheet peak;
    # executed MFMA work counts both halves of every hi/lo split operand: twice the algorithmic on
    # a block's first step, once on the later steps that take increments
    exec_factor = (2.0 + (K - 1)) / K if increments else 2.0
    peak_meas = rq.mfma_peak(ctx) * 1e12
    sweep_rate = fa["total"] / (ms_per_step / 1e3)
    res = {
        "metric": "layer-sweep time (ms) and quantized columns/sec; achieved TFLOP/s vs MFMA peak",
        "value": n / (ms_per_step / 1e3),
        "unit": "columns/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("bf16 MFMA (hi/lo split fp32 operands on a block's first step, bf16 increments on the later "
                  "steps), fp32/fp64 accumulate" if increments else
                  "bf16 MFMA (hi/lo split fp32 operands), fp32/fp64 accumulate"),
        "data": "synthetic (device-generated, workload distributions)",
        "config": {"workload": args.workload, "m": m, "n": n, "tokens": T, "bgd_steps": K, "bits": 4,
                   "group": 128, "block": 128, "bgd_form": args.form,
                   "token_chunk": tok_chunk},
        "weights_per_s": m * n / (ms_per_step / 1e3),
        "sweep_ms_each": [round(x, 1) for x in sweep_ms],
        "sweep_ms_median": float(sorted(sweep_ms)[len(sweep_ms) // 2]),
        "loss_final": out.loss_final,
        "tflops_alg": sweep_rate / 1e12,
        "frac_bf16_peak_alg": sweep_rate / PEAK_BF16,
        "mfma_peak_measured_tflops": peak_meas / 1e12,
        "frac_measured_peak_alg": sweep_rate / peak_meas,
        "kernel_ms_per_step": {k: v[1] / args.steps for k, v in kt.items()},
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": achieved / 1e12, "peak": PEAK_BF16 / 1e12,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16,
                     "traffic": (measured_traffic(args.workload, dom) if args.form == "tokens"
                                 and tok_chunk == TOKEN_CHUNK.get(args.workload, 0) else None),
                     "launches": launches, "avg_launch_ms": dom_ms / max(1, launches),
                     "measured_peak": peak_meas / 1e12, "frac_measured_peak": achieved / peak_meas,
                     "executed_frac": exec_factor * achieved / PEAK_BF16 if args.form == "tokens" else None,
                     "executed_frac_measured_peak": (exec_factor * achieved / peak_meas if args.form == "tokens"
                                                     else None),
                     "increment_launches": kt[dom + "_inc"][0] if args.form == "tokens" else 0},
    }
    if args.form == "tokens" and not args.no_gram_line:
        # one untimed-region Gram-form sweep of the same inputs, reported beside the headline
        gb = rq.bgd_params(steps=K, lr=lr, form=rq.BGD_GRAM)
        og = rq.quantize_layer(ctx, W0, X, Xh, s, qp=qp, bgd=gb)      # warm-up (workspaces)
        og = rq.quantize_layer(ctx, W0, X, Xh, s, qp=qp, bgd=gb, out=og)
        print(f"[bench] gram form: {og.ms_total:.1f} ms, loss {og.loss_final:.6g}", file=sys.stderr, flush=True)
        res["gram_form"] = {"ms_per_step": og.ms_total, "columns_per_s": n / (og.ms_total / 1e3),
                            "loss_final": og.loss_final, "loss_final_tokens": out.loss_final,
                            "note": "same loss and gradient through the calibration Gram matrices "
                                    "(bench.py --form gram for its own line)"}
    if not args.no_stage0:
        res["stage0"] = stage0(torch, rq, ctx, W0, X, Xh, s, qp, rq.bgd_params(steps=K, lr=lr), m, n, T)
    if not (args.no_next or args.no_configs) and args.form == "tokens":
        res["next"] = next_legs(torch, rq, ctx, W0, X, Xh, s, m, n, T, K, lr, args.workload)
    if not (args.no_block and args.no_decoder and args.no_configs):
        del W0, X, Xh, s
        torch.cuda.empty_cache()
    if not args.no_configs:
        res["configs"] = config_legs(torch, rq, ctx, qp)
    if not args.no_block:
        res["mlp_block"] = mlp_block(torch, rq, ctx, qp)
    if not args.no_decoder:
        res["decoder_block"] = decoder_block(torch, rq, ctx, qp)
    ctx.close()
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on a sample", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(args.workload)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
