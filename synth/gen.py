"""Seeded generators for the five calibration workloads of the layer sweep.

Each workload stands in for the WikiText-2 calibration activations of a named
model (the paper calibrates on 2048-token WikiText-2 sequences, Sec. 6.1); the
generators keep the 2048-token sequence structure in their token counts and
model outlier channels and heavy tails with simple distributions.

Draw order for one module is fixed: W, then X, then outlier channel indices,
then the X-hat noise, then the per-token weights s, then the metric M.  The
generator seed of module k of a workload is ``seed * 1000 + k``.

bf16 values are produced by round-to-nearest-even of the float32 draw and are
returned as float32 arrays holding bf16-exact values (``bf16_bits`` gives the
raw 16-bit patterns that device code consumes).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, Optional, Tuple

import numpy as np


# ----------------------------------------------------------------------------- bf16 storage

def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> uint16 bf16 bit patterns, round to nearest, ties to even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_from_bits(b: np.ndarray) -> np.ndarray:
    """uint16 bf16 bit patterns -> float32 values (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 values rounded to the nearest bf16 value (returned as float32)."""
    return bf16_from_bits(bf16_bits(x))


# ----------------------------------------------------------------------------- workloads

# Learning rates of cfg 2-5 are the paper's scheduled (non-final-block) W4A16 values from Table realq_lr
# (Appendix D.3) for the model each workload is shaped after; cfg 1 states its own.
CONFIGS: Dict[str, dict] = {
    "single_512": dict(
        desc="single linear layer 512x512, 4096 tokens",
        modules={"linear": (512, 512)}, T=4096,
        w=("f32", 0.02), x=("outlier_count", 4, 20.0), xhat=("additive", 0.01),
        s="absnormal", M=None, steps=4, lr=1e-3),
    "qwen3_0.6b_mlp": dict(
        desc="Qwen3-0.6B-shaped MLP projections, 131072 tokens (64 x 2048)",
        modules={"gate": (3072, 1024), "up": (3072, 1024), "down": (1024, 3072)}, T=131072,
        w=("bf16", 0.02), x=("student_t", 4.0), xhat=("relative", 0.01),
        s="lognormal", M=None, steps=8, lr=3e-4),
    "llama3.1_8b_layer": dict(
        desc="LLaMA-3.1-8B-shaped decoder layer, 262144 tokens (128 x 2048)",
        modules={"q": (4096, 4096), "k": (1024, 4096), "v": (1024, 4096), "o": (4096, 4096),
                 "gate": (14336, 4096), "up": (14336, 4096), "down": (4096, 14336)}, T=262144,
        w=("bf16", 0.02), x=("outlier_frac", 0.01, 50.0), xhat=("relative", 0.01),
        s=None, M=None, steps=8, lr=1e-5),
    "qwen3_32b_layer": dict(
        desc="Qwen3-32B-shaped decoder layer, 262144 tokens, dense Wishart surrogate metric",
        modules={"q": (5120, 5120), "k": (1024, 5120), "v": (1024, 5120), "o": (5120, 5120),
                 "gate": (25600, 5120), "up": (25600, 5120), "down": (5120, 25600)}, T=262144,
        w=("bf16", 0.02), x=("student_t", 3.0), xhat=("relative", 0.01),
        s=None, M=("wishart", 5120), steps=8, lr=2e-6),
    "llama3.1_70b_layer": dict(
        desc="LLaMA-3.1-70B-shaped decoder layer, 262144 tokens in 32768-token chunks",
        modules={"q": (8192, 8192), "k": (1024, 8192), "v": (1024, 8192), "o": (8192, 8192),
                 "gate": (28672, 8192), "up": (28672, 8192), "down": (8192, 28672)}, T=262144,
        w=("bf16", 0.015), x=("outlier_frac", 0.01, 50.0), xhat=("relative", 0.01),
        s=None, M=None, steps=8, lr=3e-6),
}


def module_names(cfg: str):
    return list(CONFIGS[cfg]["modules"].keys())


@dataclass
class LayerInputs:
    cfg: str
    module: str
    W0: np.ndarray              # float32 [m, n]
    X: np.ndarray               # float32, bf16-exact [T, n]   original-model layer input
    Xhat: np.ndarray            # float32, bf16-exact [T, n]   input seen by the quantized model
    s: Optional[np.ndarray]     # float32 [T] per-token weights, or None (all ones)
    M: Optional[np.ndarray]     # float32 [m, m] surrogate metric, or None (identity)
    steps: int
    lr: float

    @property
    def shape(self) -> Tuple[int, int, int]:
        return self.W0.shape[0], self.W0.shape[1], self.X.shape[0]


def _activations(rng, T, n, spec):
    kind = spec[0]
    if kind == "student_t":
        x = rng.standard_t(spec[1], size=(T, n)).astype(np.float32)
        return x
    x = rng.standard_normal((T, n), dtype=np.float32)
    if kind == "outlier_count":
        k = int(spec[1])
    elif kind == "outlier_frac":
        k = max(1, int(round(spec[1] * n)))
    else:
        raise ValueError(kind)
    idx = rng.choice(n, size=min(k, n), replace=False)
    x[:, idx] *= np.float32(spec[2])
    return x


def make_module(cfg: str, module: Optional[str] = None, seed: int = 0, *,
                m: Optional[int] = None, n: Optional[int] = None, T: Optional[int] = None,
                with_metric: bool = True) -> LayerInputs:
    """Draw one module's inputs for workload ``cfg``.

    ``m``, ``n`` and ``T`` override the workload's sizes (the distributions stay
    the same), which the parity tests use for reduced-size cases.
    """
    c = CONFIGS[cfg]
    names = list(c["modules"].keys())
    module = module or names[0]
    idx = names.index(module)
    m0, n0 = c["modules"][module]
    m = m0 if m is None else m
    n = n0 if n is None else n
    T = c["T"] if T is None else T
    rng = np.random.default_rng(seed * 1000 + idx)

    wdt, wstd = c["w"]
    W = (rng.standard_normal((m, n), dtype=np.float32) * np.float32(wstd))
    if wdt == "bf16":
        W = bf16_round(W)

    X32 = _activations(rng, T, n, c["x"])
    xh_kind, xh_amp = c["xhat"]
    noise = rng.standard_normal((T, n), dtype=np.float32)
    if xh_kind == "additive":
        Xh32 = X32 + np.float32(xh_amp) * noise
    else:
        Xh32 = X32 * (np.float32(1.0) + np.float32(xh_amp) * noise)
    X = bf16_round(X32)
    Xhat = bf16_round(Xh32)
    del X32, Xh32, noise

    s = None
    if c["s"] == "absnormal":
        s = np.abs(rng.standard_normal(T, dtype=np.float32))
    elif c["s"] == "lognormal":
        s = rng.lognormal(0.0, 1.0, size=T).astype(np.float32)

    M = None
    if with_metric and c["M"] is not None and c["M"][0] == "wishart" and m0 == c["M"][1]:
        # the dense metric belongs to the modules whose output width is the model width
        d = m
        A = rng.standard_normal((d, 2 * d), dtype=np.float32)
        M = (A @ A.T) / np.float32(2 * d)
    return LayerInputs(cfg=cfg, module=module, W0=W, X=X, Xhat=Xhat, s=s, M=M,
                       steps=c["steps"], lr=c["lr"])


# ----------------------------------------------------------------------------- Stage-0 inputs

def make_output_grads(T: int, m: int, seed: int = 0, outlier_tokens: int = 4,
                      outlier_scale: float = 1e5) -> np.ndarray:
    """Per-token gradients of a module's output, [T, m] bf16-exact float32.

    Token magnitudes are log-normal (about one decade of spread), channel magnitudes
    log-normal (half a decade), and ``outlier_tokens`` tokens are scaled up by
    ``outlier_scale``: end-to-end gradients in deep layers reach many orders of magnitude
    above the median (Appendix D.1), which the saliency clip exists for.
    """
    rng = np.random.default_rng(seed * 1000 + 900)
    g = rng.standard_normal((T, m), dtype=np.float32)
    g *= rng.lognormal(0.0, 2.3, size=(T, 1)).astype(np.float32)
    g *= rng.lognormal(0.0, 1.15, size=(1, m)).astype(np.float32)
    if outlier_tokens > 0 and T > 0:
        idx = rng.choice(T, size=min(outlier_tokens, T), replace=False)
        g[idx] *= np.float32(outlier_scale)
    return bf16_round(g * np.float32(1e-3))


def make_group_weights(n_groups: int, T: int, seed: int = 0) -> np.ndarray:
    """Positive per-token weights of ``n_groups`` row groups, [n_groups, T] float32, log-normal
    with a shared per-token factor (groups of one module see correlated saliency)."""
    rng = np.random.default_rng(seed * 1000 + 901)
    common = rng.lognormal(0.0, 1.0, size=(1, T))
    own = rng.lognormal(0.0, 0.5, size=(n_groups, T))
    return (common * own).astype(np.float32)


# ----------------------------------------------------------------------------- MLP block inputs

@dataclass
class MLPBlockInputs:
    X: np.ndarray        # [T, d] bf16-exact float32, block input of the full-precision model
    Xhat: np.ndarray     # [T, d] bf16-exact float32, block input of the quantized model
    gamma: np.ndarray    # [d] float32 RMSNorm weight
    Wg: np.ndarray       # [f, d] bf16-exact float32
    Wu: np.ndarray       # [f, d]
    Wd: np.ndarray       # [d, f]
    F: Optional[np.ndarray]   # [d, d] float32 Wishart metric at the block output, or None


def make_mlp_block(T: int, d: int, f: int, seed: int = 0, dense_F: bool = True, wstd: float = 0.02,
                   xhat_rel: float = 0.01) -> MLPBlockInputs:
    """One pre-norm SwiGLU MLP block with its calibration inputs: Student-t (nu = 4) block inputs
    with four outlier channels x 10, Xhat = X (1 + xhat_rel xi), gamma = 1 + 0.1 N(0, 1), bf16
    N(0, wstd^2) weights, and a Wishart (2d degrees of freedom) metric at the block output."""
    rng = np.random.default_rng(seed * 1000 + 950)
    X32 = rng.standard_t(4.0, size=(T, d)).astype(np.float32)
    idx = rng.choice(d, size=min(4, d), replace=False)
    X32[:, idx] *= np.float32(10.0)
    Xh32 = X32 * (np.float32(1.0) + np.float32(xhat_rel) * rng.standard_normal((T, d), dtype=np.float32))
    gamma = (1.0 + 0.1 * rng.standard_normal(d)).astype(np.float32)
    Wg = bf16_round(rng.standard_normal((f, d), dtype=np.float32) * np.float32(wstd))
    Wu = bf16_round(rng.standard_normal((f, d), dtype=np.float32) * np.float32(wstd))
    Wd = bf16_round(rng.standard_normal((d, f), dtype=np.float32) * np.float32(wstd))
    F = None
    if dense_F:
        A = rng.standard_normal((d, 2 * d), dtype=np.float32)
        F = (A @ A.T) / np.float32(2 * d)
    return MLPBlockInputs(X=bf16_round(X32), Xhat=bf16_round(Xh32), gamma=gamma, Wg=Wg, Wu=Wu, Wd=Wd, F=F)


@dataclass
class DecoderBlockInputs:
    X: np.ndarray        # [T, d] bf16-exact float32, block input of the full-precision model
    Xhat: np.ndarray     # [T, d] bf16-exact float32, block input of the quantized model
    w: dict              # gamma1, Wq, Wk, Wv, Wo, gamma2, Wg, Wu, Wd, F (float32 numpy; F may be None)
    n_heads: int
    n_kv: int
    head_dim: int
    seq_len: int


def make_decoder_block(T: int, d: int, f: int, n_heads: int, n_kv: int, head_dim: int, seq_len: int,
                       seed: int = 0, dense_F: bool = True, wstd: float = 0.02, qk_std: float = 0.04,
                       xhat_rel: float = 0.01) -> DecoderBlockInputs:
    """One pre-norm decoder block (attention, then a SwiGLU MLP) with its calibration inputs: the
    MLP half and the inputs as make_mlp_block draws them, gamma1 = 1 + 0.1 N(0, 1), bf16
    N(0, qk_std^2) query and key weights (sharper attention than wstd gives) and bf16
    N(0, wstd^2) value and output weights."""
    m = make_mlp_block(T, d, f, seed=seed, dense_F=dense_F, wstd=wstd, xhat_rel=xhat_rel)
    rng = np.random.default_rng(seed * 1000 + 951)
    Hq, Hk = n_heads * head_dim, n_kv * head_dim
    w = dict(gamma1=(1.0 + 0.1 * rng.standard_normal(d)).astype(np.float32),
             Wq=bf16_round(rng.standard_normal((Hq, d), dtype=np.float32) * np.float32(qk_std)),
             Wk=bf16_round(rng.standard_normal((Hk, d), dtype=np.float32) * np.float32(qk_std)),
             Wv=bf16_round(rng.standard_normal((Hk, d), dtype=np.float32) * np.float32(wstd)),
             Wo=bf16_round(rng.standard_normal((d, Hq), dtype=np.float32) * np.float32(wstd)),
             gamma2=m.gamma, Wg=m.Wg, Wu=m.Wu, Wd=m.Wd, F=m.F)
    return DecoderBlockInputs(X=m.X, Xhat=m.Xhat, w=w, n_heads=n_heads, n_kv=n_kv, head_dim=head_dim,
                              seq_len=seq_len)
