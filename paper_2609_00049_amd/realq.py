"""Python binding of librealq.so (include/realq.h): argument marshalling only.

Every function takes torch tensors that live on the GPU, passes their device
pointers and sizes to the C ABI, and enqueues the work on torch's current stream.
All arithmetic of the sweep runs in the HIP kernels of the library; if the library
is not built this module raises on import.
"""
from __future__ import annotations

import ctypes
import math
from dataclasses import dataclass
from pathlib import Path
from typing import Optional

import torch

_LIB_PATH = Path(__file__).resolve().parent / "librealq.so"

OK = 0
ERRORS = {
    -1: "REALQ_ERR_INVALID_ARG",
    -2: "REALQ_ERR_SHAPE",
    -3: "REALQ_ERR_NOT_SPD",
    -4: "REALQ_ERR_HIP",
    -5: "REALQ_ERR_OOM",
    -6: "REALQ_ERR_NONFINITE",
}

EXPORTS = [
    "realq_qparams_default", "realq_bgd_params_default",
    "realq_ctx_create", "realq_ctx_destroy", "realq_last_error",
    "realq_ctx_set_timing", "realq_ctx_kernel_time", "realq_ctx_reset_timing",
    "realq_fisher_accum", "realq_fisher_finish", "realq_saliency",
    "realq_hessian_accum", "realq_chol_inverse",
    "realq_bgd_state_create", "realq_bgd_state_destroy",
    "realq_quantize_block", "realq_quantize_block_rows", "realq_bgd_lock_block",
    "realq_bgd_step", "realq_bgd_loss", "realq_quantize_layer",
    "realq_pullback_metric", "realq_handoff", "realq_mlp_block_sweep",
    "realq_decoder_block_sweep", "realq_decoder_forward",
]


class RealqError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


# ----------------------------------------------------------------------------- C structs

class QParams(ctypes.Structure):
    _fields_ = [("bits", ctypes.c_int32), ("group", ctypes.c_int32), ("block", ctypes.c_int32),
                ("grid", ctypes.c_int32), ("damp", ctypes.c_float), ("sym", ctypes.c_int32)]


class BgdParams(ctypes.Structure):
    _fields_ = [("steps", ctypes.c_int32), ("lr", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("eps", ctypes.c_float), ("tok_chunk", ctypes.c_int64),
                ("form", ctypes.c_int32), ("loss_clip", ctypes.c_float), ("batch", ctypes.c_int64)]


BGD_TOKENS = 0   # residual and gradient GEMMs over all tokens every step
BGD_GRAM = 1     # the same loss and gradient through the calibration Gram matrices


class LayerDesc(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int64), ("n", ctypes.c_int64), ("T", ctypes.c_int64),
                ("W0", ctypes.c_void_p), ("X", ctypes.c_void_p), ("Xhat", ctypes.c_void_p),
                ("s", ctypes.c_void_p), ("M", ctypes.c_void_p), ("P", ctypes.c_void_p),
                ("window_offset", ctypes.c_int32), ("window_total", ctypes.c_int32),
                ("q", QParams), ("bgd", BgdParams),
                ("s_groups", ctypes.c_void_p), ("n_groups", ctypes.c_int32)]


class LayerOut(ctypes.Structure):
    _fields_ = [("codes", ctypes.c_void_p), ("scales", ctypes.c_void_p), ("zeros", ctypes.c_void_p),
                ("W_hat", ctypes.c_void_p), ("H", ctypes.c_void_p), ("U", ctypes.c_void_p),
                ("dead", ctypes.c_void_p), ("loss_trace", ctypes.c_void_p),
                ("loss_final", ctypes.c_double), ("ms_total", ctypes.c_double)]


class MLPBlock(ctypes.Structure):
    _fields_ = [("gamma", ctypes.c_void_p), ("Wg", ctypes.c_void_p), ("Wu", ctypes.c_void_p),
                ("Wd", ctypes.c_void_p), ("F", ctypes.c_void_p)]


class MLPDesc(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("d", ctypes.c_int64), ("f", ctypes.c_int64),
                ("X", ctypes.c_void_p), ("Xhat", ctypes.c_void_p), ("blk", MLPBlock), ("next", MLPBlock),
                ("eps", ctypes.c_float), ("window", ctypes.c_int32), ("q", QParams), ("bgd", BgdParams)]


class MLPOut(ctypes.Structure):
    _fields_ = [("codes", ctypes.c_void_p * 3), ("scales", ctypes.c_void_p * 3), ("zeros", ctypes.c_void_p * 3),
                ("W_hat", ctypes.c_void_p * 3), ("loss_trace", ctypes.c_void_p),
                ("loss_final", ctypes.c_double), ("ms_total", ctypes.c_double)]


class DecoderBlock(ctypes.Structure):
    _fields_ = [("gamma1", ctypes.c_void_p), ("Wq", ctypes.c_void_p), ("Wk", ctypes.c_void_p),
                ("Wv", ctypes.c_void_p), ("Wo", ctypes.c_void_p), ("mlp", MLPBlock)]


class DecoderDesc(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("d", ctypes.c_int64), ("f", ctypes.c_int64), ("seq_len", ctypes.c_int64),
                ("n_heads", ctypes.c_int32), ("n_kv", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("rope_base", ctypes.c_float), ("eps", ctypes.c_float),
                ("X", ctypes.c_void_p), ("Xhat", ctypes.c_void_p), ("blk", DecoderBlock), ("next", DecoderBlock),
                ("window", ctypes.c_int32), ("q", QParams), ("bgd", BgdParams)]


class DecoderOut(ctypes.Structure):
    _fields_ = [("codes", ctypes.c_void_p * 7), ("scales", ctypes.c_void_p * 7), ("zeros", ctypes.c_void_p * 7),
                ("W_hat", ctypes.c_void_p * 7), ("loss_trace", ctypes.c_void_p),
                ("loss_final", ctypes.c_double), ("ms_total", ctypes.c_double)]


class DecoderFwdOut(ctypes.Structure):
    _fields_ = [("h1", ctypes.c_void_p), ("q", ctypes.c_void_p), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("O", ctypes.c_void_p), ("x2", ctypes.c_void_p), ("y", ctypes.c_void_p)]


def _load():
    if not _LIB_PATH.exists():
        raise ImportError(f"{_LIB_PATH} is not built; run paper_2609_00049_amd.build.build() first")
    lib = ctypes.CDLL(str(_LIB_PATH))
    vp, i64, i32, f32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float
    sig = {
        "realq_qparams_default": (None, [ctypes.POINTER(QParams)]),
        "realq_bgd_params_default": (None, [ctypes.POINTER(BgdParams)]),
        "realq_ctx_create": (ctypes.c_int, [ctypes.POINTER(vp), vp]),
        "realq_ctx_destroy": (None, [vp]),
        "realq_last_error": (ctypes.c_char_p, [vp]),
        "realq_ctx_set_timing": (ctypes.c_int, [vp, ctypes.c_int]),
        "realq_ctx_kernel_time": (ctypes.c_int, [vp, ctypes.c_char_p, ctypes.POINTER(i64),
                                                 ctypes.POINTER(ctypes.c_double)]),
        "realq_ctx_reset_timing": (ctypes.c_int, [vp]),
        "realq_fisher_accum": (ctypes.c_int, [vp, vp, i64, i64, vp]),
        "realq_fisher_finish": (ctypes.c_int, [vp, vp, i64, i64, vp]),
        "realq_saliency": (ctypes.c_int, [vp, vp, i64, i64, i32, f32, vp]),
        "realq_hessian_accum": (ctypes.c_int, [vp, vp, vp, i64, i64, vp]),
        "realq_chol_inverse": (ctypes.c_int, [vp, vp, i64, i64, f32, vp, vp, vp]),
        "realq_bgd_state_create": (ctypes.c_int, [vp, ctypes.POINTER(vp), vp, vp, vp, vp, vp, vp, i64, i64, i64,
                                                  ctypes.POINTER(BgdParams)]),
        "realq_bgd_state_destroy": (None, [vp]),
        "realq_quantize_block": (ctypes.c_int, [vp, vp, i64, i64, i64, i64, vp, vp, ctypes.POINTER(QParams),
                                                vp, vp, vp, vp]),
        "realq_quantize_block_rows": (ctypes.c_int, [vp, vp, i64, i64, i64, i64, i64, i64, vp, vp,
                                                     ctypes.POINTER(QParams), vp, vp, vp, vp]),
        "realq_bgd_lock_block": (ctypes.c_int, [vp, vp, i64, i64]),
        "realq_bgd_step": (ctypes.c_int, [vp, vp, vp, i64, f32, vp]),
        "realq_bgd_loss": (ctypes.c_int, [vp, vp, vp, vp]),
        "realq_quantize_layer": (ctypes.c_int, [vp, ctypes.POINTER(LayerDesc), ctypes.POINTER(LayerOut)]),
        "realq_pullback_metric": (ctypes.c_int, [vp, vp, vp, i64, i64, ctypes.c_int, vp]),
        "realq_handoff": (ctypes.c_int, [vp, vp, vp, vp, i64, i64, i64, vp]),
        "realq_mlp_block_sweep": (ctypes.c_int, [vp, ctypes.POINTER(MLPDesc), ctypes.POINTER(MLPOut)]),
        "realq_decoder_block_sweep": (ctypes.c_int, [vp, ctypes.POINTER(DecoderDesc), ctypes.POINTER(DecoderOut)]),
        "realq_decoder_forward": (ctypes.c_int, [vp, ctypes.POINTER(DecoderDesc), ctypes.POINTER(DecoderFwdOut)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def lib():
    return _lib


# ----------------------------------------------------------------------------- helpers

def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("realq expects device tensors")
    if not t.is_contiguous():
        raise ValueError("realq expects contiguous tensors")
    return ctypes.c_void_p(t.data_ptr())


def _f64(t: torch.Tensor) -> torch.Tensor:
    """The sweep's working weights are float64."""
    if t.dtype != torch.float64:
        raise ValueError("working weights W must be float64")
    return t


def _bits(t: torch.Tensor) -> torch.Tensor:
    """bf16 tensor -> same storage viewed as int16 bit patterns."""
    if t.dtype != torch.bfloat16:
        raise ValueError("calibration inputs must be bfloat16")
    return t


def qparams(bits=4, group=128, block=128, grid=80, damp=0.01, sym=False) -> QParams:
    """group = 0: one group per row; sym: symmetric range with the zero fixed at 2^(bits-1)."""
    return QParams(bits, group, block, grid, damp, int(bool(sym)))


def bgd_params(steps=0, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, tok_chunk=0, form=BGD_TOKENS, loss_clip=0.0,
               batch=0) -> BgdParams:
    return BgdParams(steps, lr, beta1, beta2, eps, tok_chunk, form, loss_clip, batch)


class Context:
    """A realq_ctx bound to a torch stream (default: the current stream)."""

    def __init__(self, stream: Optional[torch.cuda.Stream] = None):
        stream = stream or torch.cuda.current_stream()
        self.stream = stream
        h = ctypes.c_void_p()
        rc = _lib.realq_ctx_create(ctypes.byref(h), ctypes.c_void_p(stream.cuda_stream))
        if rc != OK:
            raise RealqError(rc, "realq_ctx_create failed")
        self.h = h

    def check(self, rc: int):
        if rc != OK:
            raise RealqError(rc, _lib.realq_last_error(self.h).decode())

    def close(self):
        if getattr(self, "h", None):
            _lib.realq_ctx_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_timing(self, on: bool):
        self.check(_lib.realq_ctx_set_timing(self.h, int(on)))

    def reset_timing(self):
        self.check(_lib.realq_ctx_reset_timing(self.h))

    def kernel_time(self, name: str):
        n = ctypes.c_int64()
        ms = ctypes.c_double()
        self.check(_lib.realq_ctx_kernel_time(self.h, name.encode(), ctypes.byref(n), ctypes.byref(ms)))
        return n.value, ms.value


# ----------------------------------------------------------------------------- the calls

def row_groups(m: int, n_groups: int):
    """(r0, r1) of the row groups that hold rows: contiguous ranges of ceil(m / n_groups) rows."""
    r = -(-m // n_groups)
    return [(g * r, min(m, (g + 1) * r)) for g in range(n_groups) if g * r < m]


def fisher_accum(ctx: Context, G: torch.Tensor, F_acc: torch.Tensor):
    """F_acc += sum_t g_t g_t^T (float64 [m,m]); G [T,m] bf16 output gradients."""
    T, m = G.shape
    ctx.check(_lib.realq_fisher_accum(ctx.h, _ptr(_bits(G)), T, m, _ptr(F_acc)))


def fisher_finish(ctx: Context, F_acc: torch.Tensor, T_total: int, F: torch.Tensor):
    """F = float32(F_acc / T_total)."""
    m = F_acc.shape[0]
    ctx.check(_lib.realq_fisher_finish(ctx.h, _ptr(F_acc), m, T_total, _ptr(F)))


def saliency(ctx: Context, G: torch.Tensor, n_groups: int, clip_q: float = 0.0, out: Optional[torch.Tensor] = None):
    """[n_groups, T] float32 per-token squared gradient norms of each row group, clipped per group
    at the nearest-rank clip_q quantile over tokens (0 = no clip)."""
    T, m = G.shape
    if out is None:
        out = torch.empty((n_groups, T), dtype=torch.float32, device=G.device)
    ctx.check(_lib.realq_saliency(ctx.h, _ptr(_bits(G)), T, m, n_groups, clip_q, _ptr(out)))
    return out


def hessian_accum(ctx: Context, Xhat: torch.Tensor, s: Optional[torch.Tensor], H_acc: torch.Tensor):
    """H_acc += sum_t s_t xhat_t xhat_t^T (float64 [n,n])."""
    T, n = Xhat.shape
    ctx.check(_lib.realq_hessian_accum(ctx.h, _ptr(_bits(Xhat)), _ptr(s), T, n, _ptr(H_acc)))


def chol_inverse(ctx: Context, H_acc: torch.Tensor, T_total: int, damp: float, U: torch.Tensor,
                 H_out: Optional[torch.Tensor] = None, dead: Optional[torch.Tensor] = None):
    n = H_acc.shape[0]
    ctx.check(_lib.realq_chol_inverse(ctx.h, _ptr(H_acc), n, T_total, damp, _ptr(H_out), _ptr(U), _ptr(dead)))


class BgdState:
    def __init__(self, ctx: Context, W0, X, Xhat, s=None, M=None, P=None, params: Optional[BgdParams] = None):
        self.ctx = ctx
        self._keep = (W0, X, Xhat, s, M, P)
        m, n = W0.shape
        T = X.shape[0]
        params = params or bgd_params()
        h = ctypes.c_void_p()
        ctx.check(_lib.realq_bgd_state_create(ctx.h, ctypes.byref(h), _ptr(W0), _ptr(_bits(X)), _ptr(_bits(Xhat)),
                                              _ptr(s), _ptr(M), _ptr(P), m, n, T, ctypes.byref(params)))
        self.h = h

    def close(self):
        if getattr(self, "h", None):
            _lib.realq_bgd_state_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def quantize_block(ctx: Context, W, c0: int, bs: int, U, dead, qp: QParams, codes, scales, zeros,
                   state: Optional[BgdState] = None):
    m, n = W.shape
    ctx.check(_lib.realq_quantize_block(ctx.h, _ptr(_f64(W)), m, n, c0, bs, _ptr(U), _ptr(dead), ctypes.byref(qp),
                                        _ptr(codes), _ptr(scales), _ptr(zeros), state.h if state else None))


def quantize_block_rows(ctx: Context, W, r0: int, r1: int, c0: int, bs: int, U, dead, qp: QParams, codes, scales,
                        zeros, state: Optional[BgdState] = None):
    m, n = W.shape
    ctx.check(_lib.realq_quantize_block_rows(ctx.h, _ptr(_f64(W)), m, n, r0, r1, c0, bs, _ptr(U), _ptr(dead),
                                             ctypes.byref(qp), _ptr(codes), _ptr(scales), _ptr(zeros),
                                             state.h if state else None))


def bgd_lock_block(ctx: Context, state: BgdState, c0: int, bs: int):
    ctx.check(_lib.realq_bgd_lock_block(ctx.h, state.h, c0, bs))


def bgd_step(ctx: Context, state: BgdState, W, c1: int, alpha: float = 1.0, loss_out=None):
    ctx.check(_lib.realq_bgd_step(ctx.h, state.h, _ptr(_f64(W)), c1, alpha, _ptr(loss_out)))


def bgd_loss(ctx: Context, state: BgdState, W, loss_out):
    ctx.check(_lib.realq_bgd_loss(ctx.h, state.h, _ptr(_f64(W)), _ptr(loss_out)))


def pullback_metric(ctx: Context, W_next, P, M_next=None, accumulate=False):
    """P (+)= W_next^T M_next W_next."""
    m_next, m = W_next.shape
    ctx.check(_lib.realq_pullback_metric(ctx.h, _ptr(W_next), _ptr(M_next), m_next, m, int(accumulate), _ptr(P)))


def handoff(ctx: Context, Wa, X, Y, Wb=None):
    """Y = bf16(X Wa^T), or bf16(silu(X Wa^T) * (X Wb^T)) when Wb is given."""
    T, n = X.shape
    m = Wa.shape[0]
    ctx.check(_lib.realq_handoff(ctx.h, _ptr(Wa), _ptr(Wb), _ptr(_bits(X)), T, n, m, _ptr(Y)))


@dataclass
class LayerResult:
    codes: torch.Tensor
    scales: torch.Tensor
    zeros: torch.Tensor
    W_hat: torch.Tensor
    H: Optional[torch.Tensor]
    U: Optional[torch.Tensor]
    dead: Optional[torch.Tensor]
    loss_trace: Optional[torch.Tensor]
    loss_final: float
    ms_total: float


def quantize_layer(ctx: Context, W0, X, Xhat, s=None, M=None, P=None, *, qp: Optional[QParams] = None,
                   bgd: Optional[BgdParams] = None, window=None, want_H=False, want_U=False,
                   want_trace=True, s_groups=None, out: Optional[LayerResult] = None) -> LayerResult:
    """Whole-module sweep; allocates the outputs unless ``out`` supplies them.  ``s_groups``
    [N_g, T] float32: one Hessian per row group (H, U and dead then carry a leading N_g axis)."""
    qp = qp or qparams()
    bgd = bgd or bgd_params()
    m, n = W0.shape
    T = X.shape[0]
    dev = W0.device
    n_groups = 0 if s_groups is None else s_groups.shape[0]
    lead = () if s_groups is None else (n_groups,)
    if out is None:
        ng = -(-n // (qp.group or n))
        nb = -(-n // qp.block)
        out = LayerResult(
            codes=torch.empty((m, n), dtype=torch.uint8, device=dev),
            scales=torch.empty((m, ng), dtype=torch.float32, device=dev),
            zeros=torch.empty((m, ng), dtype=torch.uint8, device=dev),
            W_hat=torch.empty((m, n), dtype=torch.float32, device=dev),
            H=torch.empty(lead + (n, n), dtype=torch.float32, device=dev) if want_H else None,
            U=torch.empty(lead + (n, n), dtype=torch.float32, device=dev) if want_U else None,
            dead=torch.empty(lead + (n,), dtype=torch.uint8, device=dev),
            loss_trace=torch.empty((max(1, nb * bgd.steps),), dtype=torch.float64, device=dev)
            if want_trace else None,
            loss_final=math.nan, ms_total=math.nan)
    woff, wtot = (0, 0) if window is None else window
    desc = LayerDesc(m, n, T, _ptr(W0), _ptr(_bits(X)), _ptr(_bits(Xhat)), _ptr(s), _ptr(M), _ptr(P),
                     woff, wtot, qp, bgd, _ptr(s_groups), n_groups)
    lo = LayerOut(_ptr(out.codes), _ptr(out.scales), _ptr(out.zeros), _ptr(out.W_hat), _ptr(out.H), _ptr(out.U),
                  _ptr(out.dead), _ptr(out.loss_trace), math.nan, math.nan)
    ctx.check(_lib.realq_quantize_layer(ctx.h, ctypes.byref(desc), ctypes.byref(lo)))
    out.loss_final = lo.loss_final
    out.ms_total = lo.ms_total
    return out


# ----------------------------------------------------------------------------- block-output surrogate

MLP_MODULES = ("gate", "up", "down")


@dataclass
class BlockResult:
    modules: dict            # name -> LayerResult (codes, scales, zeros, W_hat; the rest None)
    loss_trace: Optional[torch.Tensor]
    loss_final: float
    ms_total: float


def _mlp_block(gamma, Wg, Wu, Wd, F=None) -> MLPBlock:
    return MLPBlock(_ptr(gamma), _ptr(Wg), _ptr(Wu), _ptr(Wd), _ptr(F))


def mlp_block_sweep(ctx: Context, X, Xhat, gamma, Wg, Wu, Wd, F=None, nxt=None, *, eps=1e-6, window=False,
                    qp: Optional[QParams] = None, bgd: Optional[BgdParams] = None, want_trace=True) -> BlockResult:
    """Quantize gate, up and down of one pre-norm SwiGLU MLP block with Block-GD on the block-output
    surrogate.  X, Xhat [T, d] bf16; gamma [d]; Wg, Wu [f, d]; Wd [d, f]; F [d, d] or None;
    nxt = (gamma, Wg, Wu, Wd, F) of the next block or None."""
    qp = qp or qparams()
    bgd = bgd or bgd_params()
    T, d = X.shape
    f = Wg.shape[0]
    dev = X.device
    nb = [-(-d // qp.block), -(-d // qp.block), -(-f // qp.block)]
    mods = {}
    for name, (rows, cols) in zip(MLP_MODULES, ((f, d), (f, d), (d, f))):
        ng = -(-cols // (qp.group or cols))
        mods[name] = LayerResult(codes=torch.empty((rows, cols), dtype=torch.uint8, device=dev),
                                 scales=torch.empty((rows, ng), dtype=torch.float32, device=dev),
                                 zeros=torch.empty((rows, ng), dtype=torch.uint8, device=dev),
                                 W_hat=torch.empty((rows, cols), dtype=torch.float32, device=dev),
                                 H=None, U=None, dead=None, loss_trace=None, loss_final=math.nan, ms_total=math.nan)
    trace = torch.empty((max(1, sum(nb) * bgd.steps),), dtype=torch.float64, device=dev) if want_trace else None
    nx = _mlp_block(*nxt) if nxt is not None else MLPBlock()
    desc = MLPDesc(T, d, f, _ptr(_bits(X)), _ptr(_bits(Xhat)), _mlp_block(gamma, Wg, Wu, Wd, F), nx, eps,
                   int(bool(window)), qp, bgd)
    o = MLPOut()
    for k, name in enumerate(MLP_MODULES):
        o.codes[k] = _ptr(mods[name].codes)
        o.scales[k] = _ptr(mods[name].scales)
        o.zeros[k] = _ptr(mods[name].zeros)
        o.W_hat[k] = _ptr(mods[name].W_hat)
    o.loss_trace = _ptr(trace)
    ctx.check(_lib.realq_mlp_block_sweep(ctx.h, ctypes.byref(desc), ctypes.byref(o)))
    return BlockResult(modules=mods, loss_trace=trace, loss_final=o.loss_final, ms_total=o.ms_total)


DECODER_MODULES = ("q", "k", "v", "o", "gate", "up", "down")


def _decoder_block(w: dict) -> DecoderBlock:
    return DecoderBlock(_ptr(w["gamma1"]), _ptr(w["Wq"]), _ptr(w["Wk"]), _ptr(w["Wv"]), _ptr(w["Wo"]),
                        _mlp_block(w["gamma2"], w["Wg"], w["Wu"], w["Wd"], w.get("F")))


def decoder_block_sweep(ctx: Context, X, Xhat, blk: dict, nxt: Optional[dict] = None, *, n_heads, n_kv, head_dim,
                        seq_len, rope_base=10000.0, eps=1e-6, window=False, qp: Optional[QParams] = None,
                        bgd: Optional[BgdParams] = None, want_trace=True) -> BlockResult:
    """Quantize q, k, v, o, gate, up and down of one pre-norm decoder block (rotary causal
    attention with grouped key/value heads, then a SwiGLU MLP) with Block-GD on the block-output
    surrogate.  X, Xhat [T, d] bf16; blk and nxt are dicts of float32 device tensors with keys
    gamma1 [d], Wq [H hd, d], Wk and Wv [Hkv hd, d], Wo [d, H hd], gamma2 [d], Wg and Wu [f, d],
    Wd [d, f] and optionally F [d, d]; nxt is the next block (window partner) or None."""
    qp = qp or qparams()
    bgd = bgd or bgd_params()
    T, d = X.shape
    f = blk["Wg"].shape[0]
    dev = X.device
    shapes = [tuple(blk[k].shape) for k in ("Wq", "Wk", "Wv", "Wo", "Wg", "Wu", "Wd")]
    nb = [-(-cols // qp.block) for (_, cols) in shapes]
    mods = {}
    for name, (rows, cols) in zip(DECODER_MODULES, shapes):
        ng = -(-cols // (qp.group or cols))
        mods[name] = LayerResult(codes=torch.empty((rows, cols), dtype=torch.uint8, device=dev),
                                 scales=torch.empty((rows, ng), dtype=torch.float32, device=dev),
                                 zeros=torch.empty((rows, ng), dtype=torch.uint8, device=dev),
                                 W_hat=torch.empty((rows, cols), dtype=torch.float32, device=dev),
                                 H=None, U=None, dead=None, loss_trace=None, loss_final=math.nan, ms_total=math.nan)
    trace = torch.empty((max(1, sum(nb) * bgd.steps),), dtype=torch.float64, device=dev) if want_trace else None
    nx = _decoder_block(nxt) if nxt is not None else DecoderBlock()
    desc = DecoderDesc(T, d, f, seq_len, n_heads, n_kv, head_dim, rope_base, eps, _ptr(_bits(X)), _ptr(_bits(Xhat)),
                       _decoder_block(blk), nx, int(bool(window)), qp, bgd)
    o = DecoderOut()
    for k, name in enumerate(DECODER_MODULES):
        o.codes[k] = _ptr(mods[name].codes)
        o.scales[k] = _ptr(mods[name].scales)
        o.zeros[k] = _ptr(mods[name].zeros)
        o.W_hat[k] = _ptr(mods[name].W_hat)
    o.loss_trace = _ptr(trace)
    ctx.check(_lib.realq_decoder_block_sweep(ctx.h, ctypes.byref(desc), ctypes.byref(o)))
    return BlockResult(modules=mods, loss_trace=trace, loss_final=o.loss_final, ms_total=o.ms_total)


def decoder_forward(ctx: Context, X, blk: dict, *, n_heads, n_kv, head_dim, seq_len, rope_base=10000.0, eps=1e-6,
                    intermediates=False) -> dict:
    """One forward of the decoder block (weights as for decoder_block_sweep) on X [T, d] (bf16):
    {'y': [T, d] float32} and, with intermediates=True, h1, q, k, v, O (bf16) and x2 (float32)."""
    T, d = X.shape
    f = blk["Wg"].shape[0]
    dev = X.device
    Hq, Hk = n_heads * head_dim, n_kv * head_dim
    res = {"y": torch.empty((T, d), dtype=torch.float32, device=dev)}
    if intermediates:
        for name, w in (("h1", d), ("q", Hq), ("k", Hk), ("v", Hk), ("O", Hq)):
            res[name] = torch.empty((T, w), dtype=torch.bfloat16, device=dev)
        res["x2"] = torch.empty((T, d), dtype=torch.float32, device=dev)
    desc = DecoderDesc(T, d, f, seq_len, n_heads, n_kv, head_dim, rope_base, eps, _ptr(_bits(X)), None,
                       _decoder_block(blk), DecoderBlock(), 0, qparams(), bgd_params())
    o = DecoderFwdOut(*[_ptr(res.get(k)) for k in ("h1", "q", "k", "v", "O", "x2", "y")])
    ctx.check(_lib.realq_decoder_forward(ctx.h, ctypes.byref(desc), ctypes.byref(o)))
    return res
