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
    "realq_hessian_accum", "realq_hessian_accum_noalloc", "realq_chol_inverse",
    "realq_bgd_state_create", "realq_bgd_state_destroy",
    "realq_quantize_block", "realq_quantize_block_rows", "realq_bgd_lock_block",
    "realq_bgd_step", "realq_bgd_loss", "realq_quantize_layer",
    "realq_pullback_metric", "realq_handoff", "realq_mlp_block_sweep",
    "realq_decoder_block_sweep", "realq_decoder_forward", "realq_mfma_peak",
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
                ("form", ctypes.c_int32), ("loss_clip", ctypes.c_float), ("batch", ctypes.c_int64),
                ("resid_increment", ctypes.c_int32)]


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
                ("eps", ctypes.c_float), ("window", ctypes.c_int32), ("q", QParams), ("bgd", BgdParams),
                ("start_module", ctypes.c_int32), ("n_modules", ctypes.c_int32), ("W_fixed", ctypes.c_void_p * 3),
                ("X_fixed", ctypes.c_void_p)]


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
                ("window", ctypes.c_int32), ("q", QParams), ("bgd", BgdParams),
                ("start_module", ctypes.c_int32), ("n_modules", ctypes.c_int32), ("W_fixed", ctypes.c_void_p * 7),
                ("X_fixed", ctypes.c_void_p)]


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
        "realq_hessian_accum_noalloc": (ctypes.c_int, [vp, vp, vp, i64, i64, vp]),
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
        "realq_mfma_peak": (ctypes.c_int, [vp, i64, ctypes.POINTER(ctypes.c_double)]),
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


def _t(t: Optional[torch.Tensor], name: str, dtype, shape, optional: bool = False):
    """Device pointer of ``t`` after checking its dtype and exact shape (the C ABI reads the
    buffer with the layout the shape implies, so a mismatch would read past the allocation)."""
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(int(x) for x in shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return _ptr(t)


def _dims(t: torch.Tensor, name: str, ndim: int):
    if not isinstance(t, torch.Tensor) or t.dim() != ndim:
        raise ValueError(f"{name} must be a {ndim}-d tensor")
    return tuple(t.shape)


F32, F64, BF16, U8 = torch.float32, torch.float64, torch.bfloat16, torch.uint8


def qparams(bits=4, group=128, block=128, grid=80, damp=0.01, sym=False) -> QParams:
    """group = 0: one group per row; sym: symmetric range with the zero fixed at 2^(bits-1)."""
    return QParams(bits, group, block, grid, damp, int(bool(sym)))


def bgd_params(steps=0, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, tok_chunk=0, form=BGD_TOKENS, loss_clip=0.0,
               batch=0, resid_increment=1) -> BgdParams:
    return BgdParams(steps, lr, beta1, beta2, eps, tok_chunk, form, loss_clip, batch, resid_increment)


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

def mfma_peak(ctx: Context, iters: int = 1 << 16) -> float:
    """TFLOP/s of the register-resident bf16 MFMA loop (the achievable MFMA ceiling of this GPU)."""
    v = ctypes.c_double()
    ctx.check(_lib.realq_mfma_peak(ctx.h, iters, ctypes.byref(v)))
    return v.value


def row_groups(m: int, n_groups: int):
    """(r0, r1) of the row groups that hold rows: contiguous ranges of ceil(m / n_groups) rows."""
    r = -(-m // n_groups)
    return [(g * r, min(m, (g + 1) * r)) for g in range(n_groups) if g * r < m]


def fisher_accum(ctx: Context, G: torch.Tensor, F_acc: torch.Tensor):
    """F_acc += sum_t g_t g_t^T (float64 [m,m]); G [T,m] bf16 output gradients."""
    T, m = _dims(G, "G", 2)
    ctx.check(_lib.realq_fisher_accum(ctx.h, _t(G, "G", BF16, (T, m)), T, m, _t(F_acc, "F_acc", F64, (m, m))))


def fisher_finish(ctx: Context, F_acc: torch.Tensor, T_total: int, F: torch.Tensor):
    """F = float32(F_acc / T_total)."""
    m = _dims(F_acc, "F_acc", 2)[0]
    ctx.check(_lib.realq_fisher_finish(ctx.h, _t(F_acc, "F_acc", F64, (m, m)), m, T_total, _t(F, "F", F32, (m, m))))


def saliency(ctx: Context, G: torch.Tensor, n_groups: int, clip_q: float = 0.0, out: Optional[torch.Tensor] = None):
    """[n_groups, T] float32 per-token squared gradient norms of each row group, clipped per group
    at the nearest-rank clip_q quantile over tokens (0 = no clip)."""
    T, m = _dims(G, "G", 2)
    if out is None:
        out = torch.empty((n_groups, T), dtype=torch.float32, device=G.device)
    ctx.check(_lib.realq_saliency(ctx.h, _t(G, "G", BF16, (T, m)), T, m, n_groups, clip_q,
                                  _t(out, "out", F32, (n_groups, T))))
    return out


def hessian_accum(ctx: Context, Xhat: torch.Tensor, s: Optional[torch.Tensor], H_acc: torch.Tensor):
    """H_acc += sum_t s_t xhat_t xhat_t^T (float64 [n,n])."""
    T, n = _dims(Xhat, "Xhat", 2)
    ctx.check(_lib.realq_hessian_accum(ctx.h, _t(Xhat, "Xhat", BF16, (T, n)), _t(s, "s", F32, (T,), True), T, n,
                                       _t(H_acc, "H_acc", F64, (n, n))))


def hessian_accum_noalloc(ctx: Context, Xhat: torch.Tensor, s: Optional[torch.Tensor], H_acc: torch.Tensor):
    """hessian_accum with its staging in the library's fixed per-GPU scratch array (no device
    allocation; calls that overlap on one GPU race)."""
    T, n = _dims(Xhat, "Xhat", 2)
    ctx.check(_lib.realq_hessian_accum_noalloc(ctx.h, _t(Xhat, "Xhat", BF16, (T, n)), _t(s, "s", F32, (T,), True),
                                               T, n, _t(H_acc, "H_acc", F64, (n, n))))


def chol_inverse(ctx: Context, H_acc: torch.Tensor, T_total: int, damp: float, U: torch.Tensor,
                 H_out: Optional[torch.Tensor] = None, dead: Optional[torch.Tensor] = None):
    n = _dims(H_acc, "H_acc", 2)[0]
    ctx.check(_lib.realq_chol_inverse(ctx.h, _t(H_acc, "H_acc", F64, (n, n)), n, T_total, damp,
                                      _t(H_out, "H_out", F32, (n, n), True), _t(U, "U", F32, (n, n)),
                                      _t(dead, "dead", U8, (n,), True)))


class BgdState:
    def __init__(self, ctx: Context, W0, X, Xhat, s=None, M=None, P=None, params: Optional[BgdParams] = None):
        self.ctx = ctx
        self._keep = (W0, X, Xhat, s, M, P)
        m, n = _dims(W0, "W0", 2)
        T = _dims(X, "X", 2)[0]
        params = params or bgd_params()
        h = ctypes.c_void_p()
        ctx.check(_lib.realq_bgd_state_create(
            ctx.h, ctypes.byref(h), _t(W0, "W0", F32, (m, n)), _t(X, "X", BF16, (T, n)),
            _t(Xhat, "Xhat", BF16, (T, n)), _t(s, "s", F32, (T,), True), _t(M, "M", F32, (m, m), True),
            _t(P, "P", F32, (m, m), True), m, n, T, ctypes.byref(params)))
        self.h = h
        self.m, self.n, self.T = m, n, T

    def close(self):
        if getattr(self, "h", None):
            _lib.realq_bgd_state_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _block_outputs(W, qp: QParams, U, dead, codes, scales, zeros):
    m, n = _dims(W, "W", 2)
    ng = -(-n // (qp.group or n))
    return (m, n, _t(W, "W (float64 working weights)", F64, (m, n)), _t(U, "U", F32, (n, n)),
            _t(dead, "dead", U8, (n,), True), _t(codes, "codes", U8, (m, n)), _t(scales, "scales", F32, (m, ng)),
            _t(zeros, "zeros", U8, (m, ng)))


def _state_h(state: Optional[BgdState], m: int, n: int):
    if state is None:
        return None
    if (state.m, state.n) != (m, n):
        raise ValueError(f"state is {state.m}x{state.n}, W is {m}x{n}")
    return state.h


def quantize_block(ctx: Context, W, c0: int, bs: int, U, dead, qp: QParams, codes, scales, zeros,
                   state: Optional[BgdState] = None):
    m, n, pW, pU, pd, pc, ps, pz = _block_outputs(W, qp, U, dead, codes, scales, zeros)
    ctx.check(_lib.realq_quantize_block(ctx.h, pW, m, n, c0, bs, pU, pd, ctypes.byref(qp), pc, ps, pz,
                                        _state_h(state, m, n)))


def quantize_block_rows(ctx: Context, W, r0: int, r1: int, c0: int, bs: int, U, dead, qp: QParams, codes, scales,
                        zeros, state: Optional[BgdState] = None):
    m, n, pW, pU, pd, pc, ps, pz = _block_outputs(W, qp, U, dead, codes, scales, zeros)
    ctx.check(_lib.realq_quantize_block_rows(ctx.h, pW, m, n, r0, r1, c0, bs, pU, pd, ctypes.byref(qp), pc, ps, pz,
                                             _state_h(state, m, n)))


def bgd_lock_block(ctx: Context, state: BgdState, c0: int, bs: int):
    ctx.check(_lib.realq_bgd_lock_block(ctx.h, state.h, c0, bs))


def bgd_step(ctx: Context, state: BgdState, W, c1: int, alpha: float = 1.0, loss_out=None):
    pW = _t(W, "W (float64 working weights)", F64, (state.m, state.n))
    ctx.check(_lib.realq_bgd_step(ctx.h, state.h, pW, c1, alpha, _t(loss_out, "loss_out", F64, (1,), True)))


def bgd_loss(ctx: Context, state: BgdState, W, loss_out):
    pW = _t(W, "W (float64 working weights)", F64, (state.m, state.n))
    ctx.check(_lib.realq_bgd_loss(ctx.h, state.h, pW, _t(loss_out, "loss_out", F64, (1,))))


def pullback_metric(ctx: Context, W_next, P, M_next=None, accumulate=False):
    """P (+)= W_next^T M_next W_next."""
    m_next, m = _dims(W_next, "W_next", 2)
    ctx.check(_lib.realq_pullback_metric(ctx.h, _t(W_next, "W_next", F32, (m_next, m)),
                                         _t(M_next, "M_next", F32, (m_next, m_next), True), m_next, m,
                                         int(accumulate), _t(P, "P", F32, (m, m))))


def handoff(ctx: Context, Wa, X, Y, Wb=None):
    """Y = bf16(X Wa^T), or bf16(silu(X Wa^T) * (X Wb^T)) when Wb is given."""
    T, n = _dims(X, "X", 2)
    m = _dims(Wa, "Wa", 2)[0]
    ctx.check(_lib.realq_handoff(ctx.h, _t(Wa, "Wa", F32, (m, n)), _t(Wb, "Wb", F32, (m, n), True),
                                 _t(X, "X", BF16, (T, n)), T, n, m, _t(Y, "Y", BF16, (T, m))))


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
    m, n = _dims(W0, "W0", 2)
    T = _dims(X, "X", 2)[0]
    dev = W0.device
    n_groups = 0 if s_groups is None else _dims(s_groups, "s_groups", 2)[0]
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
    ng = -(-n // (qp.group or n))
    nb = -(-n // qp.block)
    desc = LayerDesc(m, n, T, _t(W0, "W0", F32, (m, n)), _t(X, "X", BF16, (T, n)), _t(Xhat, "Xhat", BF16, (T, n)),
                     _t(s, "s", F32, (T,), True), _t(M, "M", F32, (m, m), True), _t(P, "P", F32, (m, m), True),
                     woff, wtot, qp, bgd, _t(s_groups, "s_groups", F32, (n_groups, T), True), n_groups)
    lo = LayerOut(_t(out.codes, "codes", U8, (m, n)), _t(out.scales, "scales", F32, (m, ng)),
                  _t(out.zeros, "zeros", U8, (m, ng)), _t(out.W_hat, "W_hat", F32, (m, n)),
                  _t(out.H, "H", F32, lead + (n, n), True), _t(out.U, "U", F32, lead + (n, n), True),
                  _t(out.dead, "dead", U8, lead + (n,), True),
                  _t(out.loss_trace, "loss_trace", F64, (max(1, nb * bgd.steps),), True), math.nan, math.nan)
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


def _mlp_block(gamma, Wg, Wu, Wd, F=None, *, d=None, f=None) -> MLPBlock:
    """MLP block weights after shape checks: gamma [d], Wg and Wu [f, d], Wd [d, f], F [d, d] or None."""
    if d is None:
        d = _dims(gamma, "gamma", 1)[0]
    if f is None:
        f = _dims(Wg, "Wg", 2)[0]
    return MLPBlock(_t(gamma, "gamma", F32, (d,)), _t(Wg, "Wg", F32, (f, d)), _t(Wu, "Wu", F32, (f, d)),
                    _t(Wd, "Wd", F32, (d, f)), _t(F, "F", F32, (d, d), True))


def _fixed(names, shapes, start, n_modules, fixed):
    """start_module / n_modules / W_fixed of a block sweep: the quantized weights of the modules
    before ``start`` (dict name -> float32 tensor), shape-checked."""
    if not 0 <= start < len(names) or n_modules < 0 or start + n_modules > len(names):
        raise ValueError(f"need 0 <= start < {len(names)}, n_modules >= 0, start + n_modules <= {len(names)}")
    fixed = fixed or {}
    ptrs = []
    for k, name in enumerate(names):
        if k < start:
            if name not in fixed:
                raise ValueError(f"fixed weights of {name} are required (it comes before start)")
            ptrs.append(_t(fixed[name], f"fixed[{name}]", F32, shapes[k]))
        else:
            ptrs.append(None)
    return (ctypes.c_void_p * len(names))(*ptrs)


def mlp_block_sweep(ctx: Context, X, Xhat, gamma, Wg, Wu, Wd, F=None, nxt=None, *, eps=1e-6, window=False,
                    qp: Optional[QParams] = None, bgd: Optional[BgdParams] = None, want_trace=True,
                    start=0, n_modules=0, fixed=None, x_fixed=None) -> BlockResult:
    """Quantize gate, up and down of one pre-norm SwiGLU MLP block with Block-GD on the block-output
    surrogate.  X, Xhat [T, d] bf16; gamma [d]; Wg, Wu [f, d]; Wd [d, f]; F [d, d] or None;
    nxt = (gamma, Wg, Wu, Wd, F) of the next block or None.  ``start`` / ``n_modules``: sweep only
    modules start .. start + n_modules - 1 (0: through the last), the earlier ones taken as already
    quantized with weights ``fixed[name]``; ``x_fixed`` [T, cols] bf16: the start module's input
    (u for gate and up, z for down) taken as given."""
    qp = qp or qparams()
    bgd = bgd or bgd_params()
    T, d = _dims(X, "X", 2)
    f = _dims(Wg, "Wg", 2)[0]
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
    nx = _mlp_block(*nxt, d=d) if nxt is not None else MLPBlock()
    fx = _fixed(MLP_MODULES, ((f, d), (f, d), (d, f)), start, n_modules, fixed)
    desc = MLPDesc(T, d, f, _t(X, "X", BF16, (T, d)), _t(Xhat, "Xhat", BF16, (T, d)),
                   _mlp_block(gamma, Wg, Wu, Wd, F, d=d, f=f), nx, eps, int(bool(window)), qp, bgd,
                   start, n_modules, fx, _t(x_fixed, "x_fixed", BF16, (T, (d, d, f)[start]), True))
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


def _decoder_block(w: dict, d: int, Hq: int, Hk: int) -> DecoderBlock:
    """Decoder block weights after shape checks (Hq = n_heads head_dim, Hk = n_kv head_dim)."""
    return DecoderBlock(_t(w["gamma1"], "gamma1", F32, (d,)), _t(w["Wq"], "Wq", F32, (Hq, d)),
                        _t(w["Wk"], "Wk", F32, (Hk, d)), _t(w["Wv"], "Wv", F32, (Hk, d)),
                        _t(w["Wo"], "Wo", F32, (d, Hq)),
                        _mlp_block(w["gamma2"], w["Wg"], w["Wu"], w["Wd"], w.get("F"), d=d))


def decoder_block_sweep(ctx: Context, X, Xhat, blk: dict, nxt: Optional[dict] = None, *, n_heads, n_kv, head_dim,
                        seq_len, rope_base=10000.0, eps=1e-6, window=False, qp: Optional[QParams] = None,
                        bgd: Optional[BgdParams] = None, want_trace=True, start=0, n_modules=0,
                        fixed=None, x_fixed=None) -> BlockResult:
    """Quantize q, k, v, o, gate, up and down of one pre-norm decoder block (rotary causal
    attention with grouped key/value heads, then a SwiGLU MLP) with Block-GD on the block-output
    surrogate.  X, Xhat [T, d] bf16; blk and nxt are dicts of float32 device tensors with keys
    gamma1 [d], Wq [H hd, d], Wk and Wv [Hkv hd, d], Wo [d, H hd], gamma2 [d], Wg and Wu [f, d],
    Wd [d, f] and optionally F [d, d]; nxt is the next block (window partner) or None.
    ``start`` / ``n_modules`` / ``fixed`` / ``x_fixed`` as for mlp_block_sweep (module order q, k, v,
    o, gate, up, down; x_fixed is h1 [T, d] for q, k, v, O [T, H hd] for o, u [T, d] for gate and
    up, z [T, f] for down)."""
    qp = qp or qparams()
    bgd = bgd or bgd_params()
    T, d = _dims(X, "X", 2)
    f = _dims(blk["Wg"], "Wg", 2)[0]
    dev = X.device
    Hq, Hk = n_heads * head_dim, n_kv * head_dim
    shapes = [(Hq, d), (Hk, d), (Hk, d), (d, Hq), (f, d), (f, d), (d, f)]
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
    nx = _decoder_block(nxt, d, Hq, Hk) if nxt is not None else DecoderBlock()
    fx = _fixed(DECODER_MODULES, shapes, start, n_modules, fixed)
    desc = DecoderDesc(T, d, f, seq_len, n_heads, n_kv, head_dim, rope_base, eps, _t(X, "X", BF16, (T, d)),
                       _t(Xhat, "Xhat", BF16, (T, d)), _decoder_block(blk, d, Hq, Hk), nx, int(bool(window)), qp, bgd,
                       start, n_modules, fx, _t(x_fixed, "x_fixed", BF16, (T, (d, d, d, Hq, d, d, f)[start]), True))
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
    T, d = _dims(X, "X", 2)
    f = _dims(blk["Wg"], "Wg", 2)[0]
    dev = X.device
    Hq, Hk = n_heads * head_dim, n_kv * head_dim
    res = {"y": torch.empty((T, d), dtype=torch.float32, device=dev)}
    if intermediates:
        for name, w in (("h1", d), ("q", Hq), ("k", Hk), ("v", Hk), ("O", Hq)):
            res[name] = torch.empty((T, w), dtype=torch.bfloat16, device=dev)
        res["x2"] = torch.empty((T, d), dtype=torch.float32, device=dev)
    desc = DecoderDesc(T, d, f, seq_len, n_heads, n_kv, head_dim, rope_base, eps, _t(X, "X", BF16, (T, d)), None,
                       _decoder_block(blk, d, Hq, Hk), DecoderBlock(), 0, qparams(), bgd_params())
    o = DecoderFwdOut(*[_ptr(res.get(k)) for k in ("h1", "q", "k", "v", "O", "x2", "y")])
    ctx.check(_lib.realq_decoder_forward(ctx.h, ctypes.byref(desc), ctypes.byref(o)))
    return res
