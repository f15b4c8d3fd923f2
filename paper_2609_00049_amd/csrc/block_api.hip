// realq_mlp_block_sweep: the Block-GD surrogate at the output of a pre-norm SwiGLU MLP block
// (Sec. 4.2-4.4), its launch sequence on the context's stream.  GPTQ per column block reuses
// realq_quantize_block; the block's forward and backward run on the bf16 MFMA GEMM (float32
// operands as hi/lo pairs, three passes when both operands are float32) and the kernels of
// block.hip.
#include <cmath>
#include <string>

#include "common.h"
#include "ctx.h"
#include "kernels.h"
#include "../../include/realq.h"

using realq::get_ws;
using realq::set_error;
using realq::Timed;

namespace {

struct Split {  // a float32 matrix as bf16 hi + lo (+ lo2 for all 24 bits: forward weight operands)
    uint16_t* hi = nullptr;
    uint16_t* lo = nullptr;
    uint16_t* lo2 = nullptr;
    bool lo_zero = false;  // lo (and lo2) are all zero: a bf16-exact matrix needs only the hi pass
    const uint16_t* lo_or_null() const { return lo_zero ? nullptr : lo; }
    const uint16_t* lo2_or_null() const { return lo_zero ? nullptr : lo2; }
};

int ws_split(realq_ctx* ctx, const std::string& name, int64_t count, Split& s) {
    void *h, *l;
    int rc;
    if ((rc = get_ws(ctx, (name + "_hi").c_str(), (size_t)count * 2, &h))) return rc;
    if ((rc = get_ws(ctx, (name + "_lo").c_str(), (size_t)count * 2, &l))) return rc;
    s.hi = (uint16_t*)h;
    s.lo = (uint16_t*)l;
    return REALQ_OK;
}

int ws_split3(realq_ctx* ctx, const std::string& name, int64_t count, Split& s) {
    int rc;
    if ((rc = ws_split(ctx, name, count, s))) return rc;
    void* l2;
    if ((rc = get_ws(ctx, (name + "_lo2").c_str(), (size_t)count * 2, &l2))) return rc;
    s.lo2 = (uint16_t*)l2;
    return REALQ_OK;
}

template <class T>
int ws(realq_ctx* ctx, const char* name, int64_t count, T*& p) {
    void* v;
    int rc = get_ws(ctx, name, (size_t)count * sizeof(T), &v);
    p = (T*)v;
    return rc;
}

// out[t][i] = sum_k act[t][k] W[i][k] (W as hi/lo[/lo2], act bf16 [T][K]), token-major float32
// [T][rows].  With lo2 the lo2 product is stored first and the hi/lo pass adds it, so a float32
// weight (a quantized or Block-GD-updated one) enters with all of its 24 bits.
int lin_f32(realq_ctx* ctx, const Split& W, int64_t rows, int64_t K, const uint16_t* act, int64_t T, float* out) {
    realq::GemmArgs g{W.hi, W.lo_or_null(), K, act, K, rows, T, K, 1};
    if (W.lo2_or_null()) {
        realq::GemmArgs g2{W.lo2, nullptr, K, act, K, rows, T, K, 1};
        RQ_HIP(ctx, realq::gemm_store_f32_t(g2, out, rows, ctx->stream));
        RQ_HIP(ctx, realq::gemm_store_f32_t(g, out, rows, ctx->stream, out));
    } else {
        RQ_HIP(ctx, realq::gemm_store_f32_t(g, out, rows, ctx->stream));
    }
    return REALQ_OK;
}
// same, rounded to bf16 (the lo2 product goes through the float32 slot "lin_tmp")
int lin_bf16(realq_ctx* ctx, const Split& W, int64_t rows, int64_t K, const uint16_t* act, int64_t T, uint16_t* out) {
    realq::GemmArgs g{W.hi, W.lo_or_null(), K, act, K, rows, T, K, 1};
    if (W.lo2_or_null()) {
        void* tmp;
        int rc;
        if ((rc = get_ws(ctx, "lin_tmp", (size_t)T * rows * 4, &tmp))) return rc;
        realq::GemmArgs g2{W.lo2, nullptr, K, act, K, rows, T, K, 1};
        RQ_HIP(ctx, realq::gemm_store_f32_t(g2, (float*)tmp, rows, ctx->stream));
        RQ_HIP(ctx, realq::gemm_store_bf16_t(g, out, rows, ctx->stream, (const float*)tmp));
    } else {
        RQ_HIP(ctx, realq::gemm_store_bf16_t(g, out, rows, ctx->stream));
    }
    return REALQ_OK;
}
// C[r][c] = alpha sum_k X[r][k] Y[c][k] with both operands float32 as hi/lo pairs:
// (Xhi + Xlo) Yhi + Xhi Ylo, float32 [rows][cols]
int prod3(realq_ctx* ctx, const Split& X, int64_t rows, int64_t K, const Split& Y, int64_t cols, float alpha,
          float* C) {
    realq::GemmArgs g{X.hi, X.lo_or_null(), K, Y.hi, K, rows, cols, K, 1};
    RQ_HIP(ctx, realq::gemm_store_f32(g, C, cols, 0, alpha, ctx->stream));
    if (Y.lo_or_null()) {
        realq::GemmArgs g2{X.hi, nullptr, K, Y.lo, K, rows, cols, K, 1};
        RQ_HIP(ctx, realq::gemm_acc_f32(g2, C, cols, alpha, ctx->stream));
    }
    return REALQ_OK;
}

// Sets w.lo_zero when the lower terms of a split are all zero (a bf16-exact matrix, such as a
// weight of a bf16 checkpoint): its products then skip the passes of those terms, which would add
// exact zeros.  One stream synchronisation; for the fixed operands set up once per call.
int mark_exact(realq_ctx* ctx, Split& w, int64_t count) {
    int* flag;
    int rc;
    if ((rc = ws(ctx, "nz_flag", 1, flag))) return rc;
    RQ_HIP(ctx, realq::fill_f32(reinterpret_cast<float*>(flag), 0.f, 1, ctx->stream));
    RQ_HIP(ctx, realq::any_nonzero_u16(w.lo, count, flag, ctx->stream));
    if (w.lo2) RQ_HIP(ctx, realq::any_nonzero_u16(w.lo2, count, flag, ctx->stream));
    int host = 1;
    RQ_HIP(ctx, hipMemcpyAsync(&host, flag, sizeof(int), hipMemcpyDeviceToHost, ctx->stream));
    RQ_HIP(ctx, hipStreamSynchronize(ctx->stream));
    w.lo_zero = host == 0;
    return REALQ_OK;
}

// Precomputed splits of one block's weights.
struct BlockW {
    const float* gamma = nullptr;
    Split g, u, d;        // Wg [f][d], Wu [f][d], Wd [d][f]
    Split dT, gT, uT;     // Wd^T [f][d], Wg^T [d][f], Wu^T [d][f] (backward operands)
    Split F;              // [d][d] or empty (identity)
};

int split_block(realq_ctx* ctx, const char* tag, const realq_mlp_block& b, int64_t d, int64_t f, bool backward,
                BlockW& w) {
    hipStream_t s = ctx->stream;
    const std::string t(tag);
    int rc;
    w.gamma = b.gamma;
    if ((rc = ws_split3(ctx, t + "g", f * d, w.g)) || (rc = ws_split3(ctx, t + "u", f * d, w.u)) ||
        (rc = ws_split3(ctx, t + "d", d * f, w.d)) || (rc = ws_split(ctx, t + "dT", f * d, w.dT)))
        return rc;
    RQ_HIP(ctx, realq::split3_f32(b.Wg, d, w.g.hi, w.g.lo, w.g.lo2, d, f, d, s));
    RQ_HIP(ctx, realq::split3_f32(b.Wu, d, w.u.hi, w.u.lo, w.u.lo2, d, f, d, s));
    RQ_HIP(ctx, realq::split3_f32(b.Wd, f, w.d.hi, w.d.lo, w.d.lo2, f, d, f, s));
    RQ_HIP(ctx, realq::transpose_split_f32(b.Wd, f, w.dT.hi, w.dT.lo, d, d, f, s));
    if (backward) {
        if ((rc = ws_split(ctx, t + "gT", d * f, w.gT)) || (rc = ws_split(ctx, t + "uT", d * f, w.uT))) return rc;
        RQ_HIP(ctx, realq::transpose_split_f32(b.Wg, d, w.gT.hi, w.gT.lo, f, f, d, s));
        RQ_HIP(ctx, realq::transpose_split_f32(b.Wu, d, w.uT.hi, w.uT.lo, f, f, d, s));
    }
    if (b.F) {
        if ((rc = ws_split(ctx, t + "F", d * d, w.F))) return rc;
        RQ_HIP(ctx, realq::split_diff_f32(b.F, d, nullptr, 0, w.F.hi, w.F.lo, d, d, d, s));
        if ((rc = mark_exact(ctx, w.F, d * d))) return rc;
    }
    if ((rc = mark_exact(ctx, w.g, f * d)) || (rc = mark_exact(ctx, w.u, f * d)) || (rc = mark_exact(ctx, w.d, d * f)) ||
        (rc = mark_exact(ctx, w.dT, f * d)))
        return rc;
    if (backward && ((rc = mark_exact(ctx, w.gT, d * f)) || (rc = mark_exact(ctx, w.uT, d * f)))) return rc;
    return REALQ_OK;
}

struct Fwd {  // one forward of a block: normalised input, pre-activations, SwiGLU, output
    uint16_t* u;
    float *a, *b;
    uint16_t *z, *out;
    float* y;
};

int alloc_fwd(realq_ctx* ctx, const char* tag, int64_t T, int64_t d, int64_t f, Fwd& F) {
    const std::string t(tag);
    int rc;
    if ((rc = ws(ctx, (t + "u").c_str(), T * d, F.u)) || (rc = ws(ctx, (t + "a").c_str(), T * f, F.a)) ||
        (rc = ws(ctx, (t + "b").c_str(), T * f, F.b)) || (rc = ws(ctx, (t + "z").c_str(), T * f, F.z)) ||
        (rc = ws(ctx, (t + "o").c_str(), T * d, F.out)) || (rc = ws(ctx, (t + "y").c_str(), T * d, F.y)))
        return rc;
    return REALQ_OK;
}

// tokens [t0, ...) of a forward: every buffer is token-major, so a row offset is a pointer offset
Fwd rows_of(const Fwd& F, int64_t t0, int64_t d, int64_t f) {
    return Fwd{F.u + t0 * d, F.a + t0 * f, F.b + t0 * f, F.z + t0 * f, F.out + t0 * d, F.y + t0 * d};
}

// The tokens of Block-GD step t (1-based, counted over a module): consecutive batches of
// `batch` tokens (the last one shorter when batch does not divide T), cycled in order; batch 0
// or >= T means all tokens.
struct TokenBatch {
    int64_t t0, n;
};
TokenBatch step_tokens(int64_t t, int64_t T, int64_t batch) {
    if (batch <= 0 || batch >= T) return {0, T};
    const int64_t nbatch = (T + batch - 1) / batch, t0 = ((t - 1) % nbatch) * batch;
    return {t0, std::min(T, t0 + batch) - t0};
}

// full forward of a block on h (bf16 or float32 input), y written; dy = y - ystar when dy != NULL
int forward(realq_ctx* ctx, const BlockW& w, const uint16_t* hb, const float* hf, int64_t T, int64_t d, int64_t f,
            double eps, Fwd& F, const float* ystar, float* dy) {
    hipStream_t s = ctx->stream;
    if (hb) RQ_HIP(ctx, realq::rmsnorm_bf16(hb, T, d, w.gamma, eps, F.u, s));
    else RQ_HIP(ctx, realq::rmsnorm_f32(hf, T, d, w.gamma, eps, F.u, s));
    int rc;
    if ((rc = lin_f32(ctx, w.g, f, d, F.u, T, F.a)) || (rc = lin_f32(ctx, w.u, f, d, F.u, T, F.b))) return rc;
    RQ_HIP(ctx, realq::swiglu_fwd(F.a, F.b, F.z, T * f, s));
    if ((rc = lin_bf16(ctx, w.d, d, f, F.z, T, F.out))) return rc;
    if (hb) RQ_HIP(ctx, realq::residual_out_bf16(hb, F.out, ystar, F.y, dy, T * d, s));
    else RQ_HIP(ctx, realq::residual_out_f32(hf, F.out, ystar, F.y, dy, T * d, s));
    return REALQ_OK;
}

}  // namespace

extern "C" int realq_mlp_block_sweep(realq_ctx* ctx, const realq_mlp_desc* D, realq_mlp_out* out) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (!D || !out) return set_error(ctx, REALQ_ERR_INVALID_ARG, "mlp_block_sweep: NULL desc or out");
    int rc;
    if ((rc = realq::validate_q(ctx, &D->q)) || (rc = realq::validate_bgd(ctx, &D->bgd))) return rc;
    const int64_t T = D->T, d = D->d, f = D->f;
    if (T < 1 || d < 1 || f < 1 || d % 8 || f % 8)
        return set_error(ctx, REALQ_ERR_SHAPE, "mlp_block_sweep: need T, d, f >= 1 and d, f multiples of 8");
    if (D->bgd.form != REALQ_BGD_TOKENS || D->bgd.loss_clip != 0.f)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "mlp_block_sweep: form and loss_clip must be 0");
    const realq_mlp_block& B0 = D->blk;
    if (!D->X || !D->Xhat || !B0.gamma || !B0.Wg || !B0.Wu || !B0.Wd)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "mlp_block_sweep: NULL input or weight");
    const bool has_next = D->next.Wg != nullptr;
    if (has_next && (!D->next.gamma || !D->next.Wu || !D->next.Wd))
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "mlp_block_sweep: incomplete next block");
    if (!(D->eps > 0.f) || !std::isfinite(D->eps))
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "mlp_block_sweep: eps must be finite and > 0");
    const int start = D->start_module;
    if (start < 0 || start > 2 || D->n_modules < 0 || start + D->n_modules > 3)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "mlp_block_sweep: need 0 <= start_module <= 2, n_modules >= 0 "
                                                     "and start_module + n_modules <= 3");
    const int stop = D->n_modules == 0 ? 3 : start + D->n_modules;
    for (int k = 0; k < start; ++k)
        if (!D->W_fixed[k]) return set_error(ctx, REALQ_ERR_INVALID_ARG, "mlp_block_sweep: NULL W_fixed before start_module");
    for (int k = 0; k < stop; ++k)
        if (!out->W_hat[k] || (k >= start && (!out->codes[k] || !out->scales[k] || !out->zeros[k])))
            return set_error(ctx, REALQ_ERR_INVALID_ARG, "mlp_block_sweep: NULL output array");
    const bool window = D->window != 0 && has_next;
    const double eps = (double)D->eps;
    hipStream_t s = ctx->stream;
    realq::EventPair ev;
    RQ_HIP(ctx, ev.create());
    RQ_HIP(ctx, hipEventRecord(ev.a, s));

    // module shapes: rows x cols (cols = input channels), its original weights
    const int64_t rows[3] = {f, f, d}, cols[3] = {d, d, f};
    const float* W0[3] = {B0.Wg, B0.Wu, B0.Wd};
    const int64_t blk = D->q.block;
    int64_t nb[3], off[3], B_total = 0;
    for (int k = 0; k < 3; ++k) {
        nb[k] = (cols[k] + blk - 1) / blk;
        off[k] = B_total;
        B_total += nb[k];
    }
    const int steps = D->bgd.steps;
    if (out->loss_trace && steps > 0) RQ_HIP(ctx, realq::fill_f64(out->loss_trace, NAN, B_total * steps, s));

    // ---- fixed operands: weight splits, normalised inputs, full-precision outputs
    BlockW w0, w2;
    if ((rc = split_block(ctx, "m0", B0, d, f, false, w0))) return rc;
    if (window && (rc = split_block(ctx, "m2", D->next, d, f, true, w2))) return rc;
    Fwd fs, fq, fn;  // full-precision path, quantized path, next block
    if ((rc = alloc_fwd(ctx, "mfs", T, d, f, fs)) || (rc = alloc_fwd(ctx, "mfq", T, d, f, fq))) return rc;
    if (window && (rc = alloc_fwd(ctx, "mfn", T, d, f, fn))) return rc;
    float *ystar, *y2star = nullptr, *dy, *g, *dz, *G, *mA, *vA, *dy2 = nullptr, *g2 = nullptr, *dz2 = nullptr,
                  *du2 = nullptr;
    uint16_t *uT, *zT;
    double *W, *Hacc, *parts, *lossd;
    float* Uf;
    uint8_t* dead;
    const int64_t npart = realq::dot_f32_partials();
    const int64_t maxRC = f * d, maxN = f > d ? f : d;
    if ((rc = ws(ctx, "m_ystar", T * d, ystar)) || (rc = ws(ctx, "m_dy", T * d, dy)) || (rc = ws(ctx, "m_g", T * d, g)) ||
        (rc = ws(ctx, "m_dz", T * f, dz)) || (rc = ws(ctx, "m_G", maxRC, G)) || (rc = ws(ctx, "m_mA", maxRC, mA)) ||
        (rc = ws(ctx, "m_vA", maxRC, vA)) || (rc = ws(ctx, "m_uT", d * T, uT)) || (rc = ws(ctx, "m_zT", f * T, zT)) ||
        (rc = ws(ctx, "m_W", maxRC, W)) || (rc = ws(ctx, "m_H", maxN * maxN, Hacc)) ||
        (rc = ws(ctx, "m_U", maxN * maxN, Uf)) || (rc = ws(ctx, "m_dead", maxN, dead)) ||
        (rc = ws(ctx, "m_parts", 2 * npart, parts)) || (rc = ws(ctx, "m_loss", 1, lossd)))
        return rc;
    Split sdy, sg, sgT, svT, sW, sdy2, sg2, sda2, sdb2;
    if ((rc = ws_split(ctx, "m_sdy", T * d, sdy)) || (rc = ws_split(ctx, "m_sg", T * d, sg)) ||
        (rc = ws_split(ctx, "m_sgT", d * T, sgT)) || (rc = ws_split(ctx, "m_svT", f * T, svT)) ||
        (rc = ws_split3(ctx, "m_sW", maxRC, sW)))
        return rc;
    if (window) {
        if ((rc = ws(ctx, "m_y2star", T * d, y2star)) || (rc = ws(ctx, "m_dy2", T * d, dy2)) ||
            (rc = ws(ctx, "m_g2", T * d, g2)) || (rc = ws(ctx, "m_dz2", T * f, dz2)) ||
            (rc = ws(ctx, "m_du2", T * d, du2)) || (rc = ws_split(ctx, "m_sdy2", T * d, sdy2)) ||
            (rc = ws_split(ctx, "m_sg2", T * d, sg2)) || (rc = ws_split(ctx, "m_sda2", T * f, sda2)) ||
            (rc = ws_split(ctx, "m_sdb2", T * f, sdb2)))
            return rc;
    }
    void* lin_tmp;  // sized once for every lin_bf16 of the sweep
    if ((rc = get_ws(ctx, "lin_tmp", (size_t)T * d * 4, &lin_tmp))) return rc;
    {
        Timed tm(ctx, "block_init");
        if ((rc = forward(ctx, w0, D->X, nullptr, T, d, f, eps, fs, nullptr, nullptr))) return rc;
        RQ_HIP(ctx, hipMemcpyAsync(ystar, fs.y, (size_t)T * d * 4, hipMemcpyDeviceToDevice, s));
        if (window) {
            if ((rc = forward(ctx, w2, nullptr, ystar, T, d, f, eps, fn, nullptr, nullptr))) return rc;
            RQ_HIP(ctx, hipMemcpyAsync(y2star, fn.y, (size_t)T * d * 4, hipMemcpyDeviceToDevice, s));
        }
        // quantized path with the original weights: u (gate and up input), a and b
        if ((rc = forward(ctx, w0, D->Xhat, nullptr, T, d, f, eps, fq, nullptr, nullptr))) return rc;
        if (D->X_fixed && start <= 1) {
            // the gate and up input taken as given: the quantized path from u on
            RQ_HIP(ctx, hipMemcpyAsync(fq.u, D->X_fixed, (size_t)T * d * 2, hipMemcpyDeviceToDevice, s));
            if ((rc = lin_f32(ctx, w0.g, f, d, fq.u, T, fq.a)) || (rc = lin_f32(ctx, w0.u, f, d, fq.u, T, fq.b)))
                return rc;
            RQ_HIP(ctx, realq::swiglu_fwd(fq.a, fq.b, fq.z, T * f, s));
            if ((rc = lin_bf16(ctx, w0.d, d, f, fq.z, T, fq.out))) return rc;
        }
        RQ_HIP(ctx, realq::transpose_u16(fq.u, d, uT, T, T, d, s));
    }

    // L (and L_next) at the quantized path's current forward fq over tokens [t0, t0 + Tb);
    // g = dL_slide/dy of those tokens (rows 0..Tb-1).  Returns the loss on the device in *lossd
    // (scaled partial sums reduced in a fixed order).
    auto surrogate = [&](double alpha, int64_t t0, int64_t Tb) -> int {
        const Fwd q = rows_of(fq, t0, d, f);
        const uint16_t* xh = D->Xhat + t0 * d;
        RQ_HIP(ctx, realq::residual_out_bf16(xh, q.out, ystar + t0 * d, nullptr, dy, Tb * d, s));
        if (B0.F) {
            RQ_HIP(ctx, realq::scale_split(dy, 1.f, nullptr, sdy.hi, sdy.lo, Tb * d, s));
            if ((rc = prod3(ctx, sdy, Tb, d, w0.F, d, (float)(1.0 / (double)Tb), g))) return rc;
        } else {
            RQ_HIP(ctx, realq::scale_split(dy, (float)(1.0 / (double)Tb), g, nullptr, nullptr, Tb * d, s));
        }
        RQ_HIP(ctx, realq::dot_f32(dy, g, Tb * d, 0.5 * alpha, parts, s));
        if (window && alpha < 1.0) {
            // next block on y = Xhat + out, its loss, and its input gradient blended into g
            RQ_HIP(ctx, realq::residual_out_bf16(xh, q.out, nullptr, q.y, nullptr, Tb * d, s));
            if ((rc = forward(ctx, w2, nullptr, q.y, Tb, d, f, eps, fn, y2star + t0 * d, dy2))) return rc;
            if (D->next.F) {
                RQ_HIP(ctx, realq::scale_split(dy2, 1.f, nullptr, sdy2.hi, sdy2.lo, Tb * d, s));
                if ((rc = prod3(ctx, sdy2, Tb, d, w2.F, d, (float)(1.0 / (double)Tb), g2))) return rc;
            } else {
                RQ_HIP(ctx, realq::scale_split(dy2, (float)(1.0 / (double)Tb), g2, nullptr, nullptr, Tb * d, s));
            }
            RQ_HIP(ctx, realq::dot_f32(dy2, g2, Tb * d, 0.5 * (1.0 - alpha), parts + npart, s));
            RQ_HIP(ctx, realq::scale_split(g2, 1.f, nullptr, sg2.hi, sg2.lo, Tb * d, s));
            if ((rc = prod3(ctx, sg2, Tb, d, w2.dT, f, 1.f, dz2))) return rc;  // dz2 = g2 Wd2
            RQ_HIP(ctx, realq::swiglu_bwd_pair(dz2, fn.a, fn.b, Tb, f, sda2.hi, sda2.lo, sdb2.hi, sdb2.lo, f, s));
            if ((rc = prod3(ctx, sda2, Tb, f, w2.gT, d, 1.f, du2))) return rc;  // du2 = da2 Wg2 + db2 Wu2
            realq::GemmArgs a1{sdb2.hi, sdb2.lo, f, w2.uT.hi, f, Tb, d, f, 1};
            RQ_HIP(ctx, realq::gemm_acc_f32(a1, du2, d, 1.f, s));
            if (w2.uT.lo_or_null()) {
                realq::GemmArgs a2{sdb2.hi, nullptr, f, w2.uT.lo, f, Tb, d, f, 1};
                RQ_HIP(ctx, realq::gemm_acc_f32(a2, du2, d, 1.f, s));
            }
            RQ_HIP(ctx, realq::rmsnorm_bwd_blend(q.y, g2, du2, D->next.gamma, eps, alpha, Tb, d, g, s));
            RQ_HIP(ctx, realq::reduce_partials(parts, 2 * npart, 1.0, lossd, s));
        } else {
            RQ_HIP(ctx, realq::reduce_partials(parts, npart, 1.0, lossd, s));
        }
        return REALQ_OK;
    };

    const float* Wq[3] = {nullptr, nullptr, nullptr};  // quantized weights of finished modules
    for (int mod = 0; mod < stop; ++mod) {
        const int64_t m = rows[mod], n = cols[mod];
        if (mod < start) {  // taken as already quantized
            RQ_HIP(ctx, hipMemcpyAsync(out->W_hat[mod], D->W_fixed[mod], (size_t)m * n * 4, hipMemcpyDeviceToDevice, s));
        } else {
            if (D->X_fixed && mod == 2 && start == 2) {  // the down input taken as given
                RQ_HIP(ctx, hipMemcpyAsync(fq.z, D->X_fixed, (size_t)T * f * 2, hipMemcpyDeviceToDevice, s));
                if ((rc = lin_bf16(ctx, w0.d, d, f, fq.z, T, fq.out))) return rc;
            }
            const uint16_t* inp = mod < 2 ? fq.u : fq.z;
            // GPTQ operands from this module's input in the quantized path
            RQ_HIP(ctx, realq::fill_f64(Hacc, 0.0, n * n, s));
            if ((rc = realq_hessian_accum(ctx, inp, nullptr, T, n, Hacc))) return rc;
            if ((rc = realq_chol_inverse(ctx, Hacc, n, T, D->q.damp, nullptr, Uf, dead))) return rc;
            if (mod == 2) RQ_HIP(ctx, realq::transpose_u16(fq.z, f, zT, T, T, f, s));
            RQ_HIP(ctx, realq::widen_f32(W0[mod], W, m * n, s));
            RQ_HIP(ctx, realq::fill_f32(mA, 0.f, m * n, s));
            RQ_HIP(ctx, realq::fill_f32(vA, 0.f, m * n, s));
            int64_t t_adam = 0;
            for (int64_t b = 0; b < nb[mod]; ++b) {
                const int64_t c0 = b * blk, bs = std::min<int64_t>(blk, n - c0), c1 = c0 + bs;
                if ((rc = realq_quantize_block(ctx, W, m, n, c0, bs, Uf, dead, &D->q, out->codes[mod], out->scales[mod],
                                               out->zeros[mod], nullptr)))
                    return rc;
                if (steps == 0 || c1 >= n) continue;
                double alpha = 1.0;
                if (window && B_total > 1) {
                    const double bg = (double)(off[mod] + b + 1);
                    alpha = std::min(1.0, std::max(0.0, 1.0 - (bg - 1.0) / (double)(B_total - 1)));
                }
                const int64_t nJ = n - c1;
                for (int k = 0; k < steps; ++k) {
                    Timed tm(ctx, "block_step");
                    const TokenBatch tb = step_tokens(t_adam + 1, T, D->bgd.batch);
                    const int64_t Tb = tb.n;
                    const Fwd q = rows_of(fq, tb.t0, d, f);
                    // forward of the partially quantized block with this module's current weights
                    RQ_HIP(ctx, realq::split3_f64(W, sW.hi, sW.lo, sW.lo2, m * n, s));
                    if (mod == 0) {
                        if ((rc = lin_f32(ctx, sW, f, d, q.u, Tb, q.a))) return rc;
                    } else if (mod == 1) {
                        if ((rc = lin_f32(ctx, sW, f, d, q.u, Tb, q.b))) return rc;
                    }
                    if (mod < 2) RQ_HIP(ctx, realq::swiglu_fwd(q.a, q.b, q.z, Tb * f, s));
                    if ((rc = lin_bf16(ctx, mod == 2 ? sW : w0.d, d, f, q.z, Tb, q.out))) return rc;
                    if ((rc = surrogate(alpha, tb.t0, Tb))) return rc;
                    if (out->loss_trace)
                        RQ_HIP(ctx, hipMemcpyAsync(out->loss_trace + (off[mod] + b) * steps + k, lossd, 8,
                                                   hipMemcpyDeviceToDevice, s));
                    // gradient of this module's trailing columns over the step's tokens (the
                    // transposed inputs keep their stride T, the transposed output gradient has Tb)
                    if (mod < 2) {
                        RQ_HIP(ctx, realq::scale_split(g, 1.f, nullptr, sg.hi, sg.lo, Tb * d, s));
                        if ((rc = prod3(ctx, sg, Tb, d, w0.dT, f, 1.f, dz))) return rc;  // dz = g Wd
                        RQ_HIP(ctx, realq::swiglu_bwd(dz, q.a, q.b, mod, Tb, f, 1, svT.hi, svT.lo, Tb, s));
                        realq::GemmArgs gg{svT.hi, svT.lo, Tb, uT + c1 * T + tb.t0, T, f, nJ, Tb, 1};
                        RQ_HIP(ctx, realq::gemm_store_f32(gg, G, nJ, 0, 1.f, s));
                    } else {
                        RQ_HIP(ctx, realq::transpose_split_f32(g, d, sgT.hi, sgT.lo, Tb, Tb, d, s));
                        realq::GemmArgs gg{sgT.hi, sgT.lo, Tb, zT + c1 * T + tb.t0, T, d, nJ, Tb, 1};
                        RQ_HIP(ctx, realq::gemm_store_f32(gg, G, nJ, 0, 1.f, s));
                    }
                    ++t_adam;
                    realq::AdamArgs a{};
                    a.W = W;
                    a.mA = mA;
                    a.vA = vA;
                    a.m = m;
                    a.n = n;
                    a.c1 = c1;
                    a.lr = D->bgd.lr;
                    a.beta1 = D->bgd.beta1;
                    a.beta2 = D->bgd.beta2;
                    a.eps = D->bgd.eps;
                    a.bc1 = (float)(1.0 / (1.0 - std::pow((double)D->bgd.beta1, (double)t_adam)));
                    a.bc2 = (float)(1.0 / (1.0 - std::pow((double)D->bgd.beta2, (double)t_adam)));
                    a.gscale = 1.f;
                    RQ_HIP(ctx, realq::adam_update_dense(a, G, s));
                }
            }
            RQ_HIP(ctx, realq::narrow_f64(W, out->W_hat[mod], m * n, s));
        }
        Wq[mod] = out->W_hat[mod];
        // the quantized path with this module's final weights
        Split q;
        if ((rc = ws_split3(ctx, "m_sq", m * n, q))) return rc;
        RQ_HIP(ctx, realq::split3_f32(Wq[mod], n, q.hi, q.lo, q.lo2, n, m, n, s));
        if (mod == 0 && (rc = lin_f32(ctx, q, f, d, fq.u, T, fq.a))) return rc;
        if (mod == 1 && (rc = lin_f32(ctx, q, f, d, fq.u, T, fq.b))) return rc;
        if (mod < 2) RQ_HIP(ctx, realq::swiglu_fwd(fq.a, fq.b, fq.z, T * f, s));
        if ((rc = lin_bf16(ctx, mod == 2 ? q : w0.d, d, f, fq.z, T, fq.out))) return rc;
    }
    // own-block loss at the quantized weights over all tokens (fq holds the final forward)
    if ((rc = surrogate(1.0, 0, T))) return rc;
    RQ_HIP(ctx, hipEventRecord(ev.b, s));
    RQ_HIP(ctx, hipMemcpyAsync(&out->loss_final, lossd, 8, hipMemcpyDeviceToHost, s));
    RQ_HIP(ctx, hipStreamSynchronize(s));
    float ms = 0.f;
    RQ_HIP(ctx, hipEventElapsedTime(&ms, ev.a, ev.b));
    out->ms_total = ms;
    return realq::harvest(ctx);
}

// ============================================================================ full decoder block

namespace {

struct DecW {  // one decoder block's weights as the GEMMs consume them
    const float* gamma1 = nullptr;
    Split q, k, v, o;   // forward operands: Wq [Hq][d], Wk [Hk][d], Wv [Hk][d], Wo [d][Hq]
    Split oT;           // Wo^T [Hq][d]              (dO = dx2 Wo)
    Split qT, kT, vT;   // Wq^T [d][Hq], Wk^T, Wv^T  (dh1 = dq Wq + dk Wk + dv Wv; next block only)
    BlockW mlp;         // the MLP half, with its backward operands
};

int split_dec(realq_ctx* ctx, const char* tag, const realq_decoder_block& b, int64_t d, int64_t f, int64_t Hq,
              int64_t Hk, bool input_grad, DecW& w) {
    hipStream_t s = ctx->stream;
    const std::string t(tag);
    int rc;
    w.gamma1 = b.gamma1;
    if ((rc = ws_split3(ctx, t + "q", Hq * d, w.q)) || (rc = ws_split3(ctx, t + "k", Hk * d, w.k)) ||
        (rc = ws_split3(ctx, t + "v", Hk * d, w.v)) || (rc = ws_split3(ctx, t + "o", d * Hq, w.o)) ||
        (rc = ws_split(ctx, t + "oT", Hq * d, w.oT)))
        return rc;
    RQ_HIP(ctx, realq::split3_f32(b.Wq, d, w.q.hi, w.q.lo, w.q.lo2, d, Hq, d, s));
    RQ_HIP(ctx, realq::split3_f32(b.Wk, d, w.k.hi, w.k.lo, w.k.lo2, d, Hk, d, s));
    RQ_HIP(ctx, realq::split3_f32(b.Wv, d, w.v.hi, w.v.lo, w.v.lo2, d, Hk, d, s));
    RQ_HIP(ctx, realq::split3_f32(b.Wo, Hq, w.o.hi, w.o.lo, w.o.lo2, Hq, d, Hq, s));
    RQ_HIP(ctx, realq::transpose_split_f32(b.Wo, Hq, w.oT.hi, w.oT.lo, d, d, Hq, s));
    if (input_grad) {
        if ((rc = ws_split(ctx, t + "qT", d * Hq, w.qT)) || (rc = ws_split(ctx, t + "kT", d * Hk, w.kT)) ||
            (rc = ws_split(ctx, t + "vT", d * Hk, w.vT)))
            return rc;
        RQ_HIP(ctx, realq::transpose_split_f32(b.Wq, d, w.qT.hi, w.qT.lo, Hq, Hq, d, s));
        RQ_HIP(ctx, realq::transpose_split_f32(b.Wk, d, w.kT.hi, w.kT.lo, Hk, Hk, d, s));
        RQ_HIP(ctx, realq::transpose_split_f32(b.Wv, d, w.vT.hi, w.vT.lo, Hk, Hk, d, s));
        if ((rc = mark_exact(ctx, w.qT, d * Hq)) || (rc = mark_exact(ctx, w.kT, d * Hk)) ||
            (rc = mark_exact(ctx, w.vT, d * Hk)))
            return rc;
    }
    if ((rc = mark_exact(ctx, w.q, Hq * d)) || (rc = mark_exact(ctx, w.k, Hk * d)) || (rc = mark_exact(ctx, w.v, Hk * d)) ||
        (rc = mark_exact(ctx, w.o, d * Hq)) || (rc = mark_exact(ctx, w.oT, Hq * d)))
        return rc;
    return split_block(ctx, (t + "m").c_str(), b.mlp, d, f, true, w.mlp);
}

struct DecDims {
    int64_t T, d, f, L, H, Hkv, hd, Hq, Hk;
    double base, eps;
    double* rope = nullptr;  // device [L][hd/2][2]: the rotary cos/sin table of (L, hd, base)
};

struct DecF {  // buffers of one forward of the decoder block
    uint16_t *h1, *q, *k, *v, *qr, *kr, *O, *o, *vt;
    float *O32, *x2;
    double* lse;  // [T][H] row log-sum-exp of the attention (the backward recomputes P from it)
    Fwd mlp;
};

// tokens [t0, ...) of a decoder forward (t0 a multiple of the sequence length).  vt is the
// attention's own transposed copy of v, written and read with the stride of the token count it
// is given, so it is shared rather than offset.
DecF rows_of(const DecF& F, const DecDims& D, int64_t t0) {
    DecF v = F;
    v.h1 += t0 * D.d;
    v.q += t0 * D.Hq;
    v.k += t0 * D.Hk;
    v.v += t0 * D.Hk;
    v.qr += t0 * D.Hq;
    v.kr += t0 * D.Hk;
    v.O += t0 * D.Hq;
    v.o += t0 * D.d;
    v.O32 += t0 * D.Hq;
    v.x2 += t0 * D.d;
    v.lse += t0 * D.H;
    v.mlp = rows_of(F.mlp, t0, D.d, D.f);
    return v;
}

int alloc_decf(realq_ctx* ctx, const char* tag, const DecDims& D, DecF& F) {
    const std::string t(tag);
    int rc;
    const int64_t T = D.T;
    if ((rc = ws(ctx, (t + "h1").c_str(), T * D.d, F.h1)) || (rc = ws(ctx, (t + "q").c_str(), T * D.Hq, F.q)) ||
        (rc = ws(ctx, (t + "k").c_str(), T * D.Hk, F.k)) || (rc = ws(ctx, (t + "v").c_str(), T * D.Hk, F.v)) ||
        (rc = ws(ctx, (t + "qr").c_str(), T * D.Hq, F.qr)) || (rc = ws(ctx, (t + "kr").c_str(), T * D.Hk, F.kr)) ||
        (rc = ws(ctx, (t + "O").c_str(), T * D.Hq, F.O)) || (rc = ws(ctx, (t + "oo").c_str(), T * D.d, F.o)) ||
        (rc = ws(ctx, (t + "lse").c_str(), T * D.H, F.lse)) || (rc = ws(ctx, (t + "x2").c_str(), T * D.d, F.x2)) ||
        (rc = ws(ctx, (t + "O32").c_str(), T * D.Hq, F.O32)) || (rc = ws(ctx, (t + "vt").c_str(), T * D.Hk, F.vt)))
        return rc;
    return alloc_fwd(ctx, (t + "m").c_str(), T, D.d, D.f, F.mlp);
}

// stage A: h1 = rmsnorm(x); the projections selected by mask (1 q, 2 k, 4 v) and their rotary
// embeddings; attention (P, O)
int dec_attn(realq_ctx* ctx, const DecW& w, const uint16_t* xb, const float* xf, const DecDims& D, DecF& F,
             int mask, bool norm) {
    hipStream_t s = ctx->stream;
    int rc;
    if (norm) {
        if (xb) RQ_HIP(ctx, realq::rmsnorm_bf16(xb, D.T, D.d, w.gamma1, D.eps, F.h1, s));
        else RQ_HIP(ctx, realq::rmsnorm_f32(xf, D.T, D.d, w.gamma1, D.eps, F.h1, s));
    }
    if ((mask & 1) && (rc = lin_bf16(ctx, w.q, D.Hq, D.d, F.h1, D.T, F.q))) return rc;
    if ((mask & 2) && (rc = lin_bf16(ctx, w.k, D.Hk, D.d, F.h1, D.T, F.k))) return rc;
    if ((mask & 4) && (rc = lin_bf16(ctx, w.v, D.Hk, D.d, F.h1, D.T, F.v))) return rc;
    Timed tm(ctx, "attention");
    if (mask & 1) RQ_HIP(ctx, realq::rope_fwd(F.q, F.qr, D.rope, D.T, D.H, D.hd, D.L, s));
    if (mask & 2) RQ_HIP(ctx, realq::rope_fwd(F.k, F.kr, D.rope, D.T, D.Hkv, D.hd, D.L, s));
    RQ_HIP(ctx, realq::attn_fwd(F.qr, F.kr, F.v, D.T, D.H, D.Hkv, D.hd, D.L, F.lse, F.O32, F.O, F.vt, s));
    return REALQ_OK;
}

// stage B: x2 = x + bf16(O Wo^T)
int dec_o(realq_ctx* ctx, const DecW& w, const uint16_t* xb, const float* xf, const DecDims& D, DecF& F) {
    int rc;
    if ((rc = lin_bf16(ctx, w.o, D.d, D.Hq, F.O, D.T, F.o))) return rc;
    if (xb) RQ_HIP(ctx, realq::residual_out_bf16(xb, F.o, nullptr, F.x2, nullptr, D.T * D.d, ctx->stream));
    else RQ_HIP(ctx, realq::residual_out_f32(xf, F.o, nullptr, F.x2, nullptr, D.T * D.d, ctx->stream));
    return REALQ_OK;
}

int dec_forward(realq_ctx* ctx, const DecW& w, const uint16_t* xb, const float* xf, const DecDims& D, DecF& F) {
    int rc;
    if ((rc = dec_attn(ctx, w, xb, xf, D, F, 7, true)) || (rc = dec_o(ctx, w, xb, xf, D, F))) return rc;
    return forward(ctx, w.mlp, nullptr, F.x2, D.T, D.d, D.f, D.eps, F.mlp, nullptr, nullptr);
}

struct DecWork {  // backward work buffers (sized for the widest use)
    float *dz, *du, *dx2, *dO, *dq, *dk, *dv, *dqr, *dkr, *dh1;
    realq::AttnScratch at;  // shared by every DecWork of a context (used one call at a time)
    Split sg, sda, sdb, sdx2, sdO, sdq, sdk, sdv;
};

int alloc_work(realq_ctx* ctx, const char* tag, const DecDims& D, DecWork& Wk) {
    const std::string t(tag);
    const int64_t T = D.T;
    int rc;
    if ((rc = ws(ctx, (t + "dz").c_str(), T * D.f, Wk.dz)) || (rc = ws(ctx, (t + "du").c_str(), T * D.d, Wk.du)) ||
        (rc = ws(ctx, (t + "dx2").c_str(), T * D.d, Wk.dx2)) || (rc = ws(ctx, (t + "dO").c_str(), T * D.Hq, Wk.dO)) ||
        (rc = ws(ctx, (t + "dq").c_str(), T * D.Hq, Wk.dq)) || (rc = ws(ctx, (t + "dk").c_str(), T * D.Hk, Wk.dk)) ||
        (rc = ws(ctx, (t + "dv").c_str(), T * D.Hk, Wk.dv)) || (rc = ws(ctx, (t + "dqr").c_str(), T * D.Hq, Wk.dqr)) ||
        (rc = ws(ctx, (t + "dkr").c_str(), T * D.Hk, Wk.dkr)) ||
        (rc = ws(ctx, (t + "dh1").c_str(), T * D.d, Wk.dh1)) || (rc = ws_split(ctx, t + "sg", T * D.d, Wk.sg)) ||
        (rc = ws_split(ctx, t + "sda", T * D.f, Wk.sda)) || (rc = ws_split(ctx, t + "sdb", T * D.f, Wk.sdb)) ||
        (rc = ws_split(ctx, t + "sdx2", T * D.d, Wk.sdx2)) || (rc = ws_split(ctx, t + "sdO", T * D.Hq, Wk.sdO)) ||
        (rc = ws_split(ctx, t + "sdq", T * D.Hq, Wk.sdq)) || (rc = ws_split(ctx, t + "sdk", T * D.Hk, Wk.sdk)) ||
        (rc = ws_split(ctx, t + "sdv", T * D.Hk, Wk.sdv)))
        return rc;
    realq::AttnScratch& a = Wk.at;
    const int64_t TL = T * D.H * D.L;
    if ((rc = ws(ctx, "att_D", T * D.H, a.D)) || (rc = ws(ctx, "att_dSh", TL, a.dSh)) ||
        (rc = ws(ctx, "att_dSl", TL, a.dSl)) || (rc = ws(ctx, "att_dSth", TL, a.dSth)) ||
        (rc = ws(ctx, "att_dStl", TL, a.dStl)) || (rc = ws(ctx, "att_Pth", TL, a.Pth)) ||
        (rc = ws(ctx, "att_Ptl", TL, a.Ptl)) || (rc = ws(ctx, "att_kt", T * D.Hk, a.kt)) ||
        (rc = ws(ctx, "att_qt", T * D.Hq, a.qt)) || (rc = ws(ctx, "att_dOth", T * D.Hq, a.dOth)) ||
        (rc = ws(ctx, "att_dOtl", T * D.Hq, a.dOtl)) ||
        (rc = ws(ctx, "att_part", realq::attn_dkv_chunks(D.L) * 2 * T * D.Hk, a.part)))
        return rc;
    return REALQ_OK;
}

int prod3_acc(realq_ctx* ctx, const Split& X, int64_t rows, int64_t K, const Split& Y, int64_t cols, float* C) {
    realq::GemmArgs g{X.hi, X.lo_or_null(), K, Y.hi, K, rows, cols, K, 1};
    RQ_HIP(ctx, realq::gemm_acc_f32(g, C, cols, 1.f, ctx->stream));
    if (Y.lo_or_null()) {
        realq::GemmArgs g2{X.hi, nullptr, K, Y.lo, K, rows, cols, K, 1};
        RQ_HIP(ctx, realq::gemm_acc_f32(g2, C, cols, 1.f, ctx->stream));
    }
    return REALQ_OK;
}

// From g = dL/dy: dx2 = g + RMSNorm backward of (da Wg + db Wu) at x2 (casts as the identity).
int back_to_x2(realq_ctx* ctx, const DecW& w, const DecDims& D, const DecF& F, const float* g, DecWork& Wk) {
    hipStream_t s = ctx->stream;
    int rc;
    const int64_t T = D.T, d = D.d, f = D.f;
    RQ_HIP(ctx, realq::scale_split(g, 1.f, nullptr, Wk.sg.hi, Wk.sg.lo, T * d, s));
    if ((rc = prod3(ctx, Wk.sg, T, d, w.mlp.dT, f, 1.f, Wk.dz))) return rc;
    RQ_HIP(ctx, realq::swiglu_bwd_pair(Wk.dz, F.mlp.a, F.mlp.b, T, f, Wk.sda.hi, Wk.sda.lo, Wk.sdb.hi, Wk.sdb.lo, f, s));
    if ((rc = prod3(ctx, Wk.sda, T, f, w.mlp.gT, d, 1.f, Wk.du)) || (rc = prod3_acc(ctx, Wk.sdb, T, f, w.mlp.uT, d, Wk.du)))
        return rc;
    RQ_HIP(ctx, realq::rmsnorm_bwd_blend(F.x2, g, Wk.du, w.mlp.gamma, D.eps, 0.0, T, d, Wk.dx2, s));
    return REALQ_OK;
}

// From dx2: dO = dx2 Wo, the attention backward, and dq, dk (before the rotary embedding), dv.
int back_to_qkv(realq_ctx* ctx, const DecW& w, const DecDims& D, const DecF& F, DecWork& Wk) {
    hipStream_t s = ctx->stream;
    int rc;
    const int64_t T = D.T;
    RQ_HIP(ctx, realq::scale_split(Wk.dx2, 1.f, nullptr, Wk.sdx2.hi, Wk.sdx2.lo, T * D.d, s));
    if ((rc = prod3(ctx, Wk.sdx2, T, D.d, w.oT, D.Hq, 1.f, Wk.dO))) return rc;
    Timed tm(ctx, "attention");
    RQ_HIP(ctx, realq::attn_bwd(F.lse, F.O32, Wk.dO, F.qr, F.kr, F.v, T, D.H, D.Hkv, D.hd, D.L, Wk.at, Wk.dqr, Wk.dkr,
                                Wk.dv, s));
    RQ_HIP(ctx, realq::rope_inv(Wk.dqr, Wk.dq, D.rope, T, D.H, D.hd, D.L, s));
    RQ_HIP(ctx, realq::rope_inv(Wk.dkr, Wk.dk, D.rope, T, D.Hkv, D.hd, D.L, s));
    return REALQ_OK;
}


// Shape, pointer and scalar checks shared by the decoder entry points.
int check_decoder(realq_ctx* ctx, const realq_decoder_desc* Dd, const char* who, DecDims& D) {
    D.T = Dd->T;
    D.d = Dd->d;
    D.f = Dd->f;
    D.L = Dd->seq_len;
    D.H = Dd->n_heads;
    D.Hkv = Dd->n_kv;
    D.hd = Dd->head_dim;
    D.Hq = D.H * D.hd;
    D.Hk = D.Hkv * D.hd;
    D.base = (double)Dd->rope_base;
    D.eps = (double)Dd->eps;
    if (D.T < 1 || D.d < 1 || D.f < 1 || D.L < 32 || D.L > 4096 || D.L % 32 || D.T % D.L || D.H < 1 || D.Hkv < 1 ||
        D.H % D.Hkv || D.hd < 32 || D.hd % 32 || D.hd > 256 || D.d % 8 || D.f % 8)
        return set_error(ctx, REALQ_ERR_SHAPE, std::string(who) + ": unsupported shape (see realq.h)");
    const realq_decoder_block& B0 = Dd->blk;
    if (!Dd->X || !B0.gamma1 || !B0.Wq || !B0.Wk || !B0.Wv || !B0.Wo || !B0.mlp.gamma || !B0.mlp.Wg || !B0.mlp.Wu ||
        !B0.mlp.Wd)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, std::string(who) + ": NULL input or weight");
    if (!(Dd->eps > 0.f) || !std::isfinite(Dd->eps) || !(Dd->rope_base > 0.f) || !std::isfinite(Dd->rope_base))
        return set_error(ctx, REALQ_ERR_INVALID_ARG, std::string(who) + ": eps and rope_base must be finite and > 0");
    return REALQ_OK;
}

// The rotary cos/sin table of the decoder's (seq_len, head_dim, rope_base), filled on the stream.
int rope_init(realq_ctx* ctx, DecDims& D) {
    int rc;
    if ((rc = ws(ctx, "d_rope", D.L * D.hd, D.rope))) return rc;
    RQ_HIP(ctx, realq::rope_table(D.rope, D.L, D.hd, D.base, ctx->stream));
    return REALQ_OK;
}

}  // namespace

extern "C" int realq_decoder_forward(realq_ctx* ctx, const realq_decoder_desc* Dd, realq_decoder_fwd_out* out) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (!Dd || !out || !out->y) return set_error(ctx, REALQ_ERR_INVALID_ARG, "decoder_forward: NULL desc or y");
    int rc;
    DecDims D;
    if ((rc = check_decoder(ctx, Dd, "decoder_forward", D)) || (rc = rope_init(ctx, D))) return rc;
    hipStream_t s = ctx->stream;
    DecW w;
    DecF F;
    if ((rc = split_dec(ctx, "df", Dd->blk, D.d, D.f, D.Hq, D.Hk, false, w)) || (rc = alloc_decf(ctx, "dff", D, F)) ||
        (rc = dec_forward(ctx, w, Dd->X, nullptr, D, F)))
        return rc;
    const int64_t T = D.T;
    auto cp = [&](void* dst, const void* src, int64_t bytes) -> int {
        if (dst) RQ_HIP(ctx, hipMemcpyAsync(dst, src, (size_t)bytes, hipMemcpyDeviceToDevice, s));
        return REALQ_OK;
    };
    if ((rc = cp(out->h1, F.h1, T * D.d * 2)) || (rc = cp(out->q, F.q, T * D.Hq * 2)) ||
        (rc = cp(out->k, F.k, T * D.Hk * 2)) || (rc = cp(out->v, F.v, T * D.Hk * 2)) ||
        (rc = cp(out->O, F.O, T * D.Hq * 2)) || (rc = cp(out->x2, F.x2, T * D.d * 4)) ||
        (rc = cp(out->y, F.mlp.y, T * D.d * 4)))
        return rc;
    RQ_HIP(ctx, hipStreamSynchronize(s));
    return realq::harvest(ctx);
}

extern "C" int realq_decoder_block_sweep(realq_ctx* ctx, const realq_decoder_desc* Dd, realq_decoder_out* out) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (!Dd || !out) return set_error(ctx, REALQ_ERR_INVALID_ARG, "decoder_block_sweep: NULL desc or out");
    int rc;
    if ((rc = realq::validate_q(ctx, &Dd->q)) || (rc = realq::validate_bgd(ctx, &Dd->bgd))) return rc;
    if (Dd->bgd.form != REALQ_BGD_TOKENS || Dd->bgd.loss_clip != 0.f)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "decoder_block_sweep: form and loss_clip must be 0");
    DecDims D;
    if ((rc = check_decoder(ctx, Dd, "decoder_block_sweep", D)) || (rc = rope_init(ctx, D))) return rc;
    if (Dd->bgd.batch % D.L)
        return set_error(ctx, REALQ_ERR_SHAPE, "decoder_block_sweep: batch must be a multiple of seq_len");
    if (!Dd->Xhat) return set_error(ctx, REALQ_ERR_INVALID_ARG, "decoder_block_sweep: NULL Xhat");
    const realq_decoder_block& B0 = Dd->blk;
    const realq_decoder_block& N0 = Dd->next;
    const bool has_next = N0.Wq != nullptr;
    if (has_next && (!N0.gamma1 || !N0.Wk || !N0.Wv || !N0.Wo || !N0.mlp.gamma || !N0.mlp.Wg || !N0.mlp.Wu ||
                     !N0.mlp.Wd))
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "decoder_block_sweep: incomplete next block");
    const int start = Dd->start_module;
    if (start < 0 || start > 6 || Dd->n_modules < 0 || start + Dd->n_modules > 7)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "decoder_block_sweep: need 0 <= start_module <= 6, n_modules >= 0 "
                                                     "and start_module + n_modules <= 7");
    const int stop = Dd->n_modules == 0 ? 7 : start + Dd->n_modules;
    for (int k = 0; k < start; ++k)
        if (!Dd->W_fixed[k])
            return set_error(ctx, REALQ_ERR_INVALID_ARG, "decoder_block_sweep: NULL W_fixed before start_module");
    for (int k = 0; k < stop; ++k)
        if (!out->W_hat[k] || (k >= start && (!out->codes[k] || !out->scales[k] || !out->zeros[k])))
            return set_error(ctx, REALQ_ERR_INVALID_ARG, "decoder_block_sweep: NULL output array");
    const bool window = Dd->window != 0 && has_next;
    const int64_t T = D.T, d = D.d, f = D.f;
    hipStream_t s = ctx->stream;
    realq::EventPair ev;
    RQ_HIP(ctx, ev.create());
    RQ_HIP(ctx, hipEventRecord(ev.a, s));

    // modules q, k, v, o, gate, up, down: rows x cols and original weights
    const int64_t rows[7] = {D.Hq, D.Hk, D.Hk, d, f, f, d}, cols[7] = {d, d, d, D.Hq, d, d, f};
    const float* W0[7] = {B0.Wq, B0.Wk, B0.Wv, B0.Wo, B0.mlp.Wg, B0.mlp.Wu, B0.mlp.Wd};
    const int64_t blk = Dd->q.block;
    int64_t nb[7], off[7], B_total = 0;
    for (int k = 0; k < 7; ++k) {
        nb[k] = (cols[k] + blk - 1) / blk;
        off[k] = B_total;
        B_total += nb[k];
    }
    const int steps = Dd->bgd.steps;
    if (out->loss_trace && steps > 0) RQ_HIP(ctx, realq::fill_f64(out->loss_trace, NAN, B_total * steps, s));

    DecW wq, wn;  // the quantized path's current weights; the next block's
    if ((rc = split_dec(ctx, "d0", B0, d, f, D.Hq, D.Hk, false, wq))) return rc;
    if (window && (rc = split_dec(ctx, "d2", N0, d, f, D.Hq, D.Hk, true, wn))) return rc;
    DecF Fs, Fq, Fn;
    if ((rc = alloc_decf(ctx, "dfs", D, Fs)) || (rc = alloc_decf(ctx, "dfq", D, Fq))) return rc;
    if (window && (rc = alloc_decf(ctx, "dfn", D, Fn))) return rc;
    DecWork Wk, Wn;
    if ((rc = alloc_work(ctx, "dwq", D, Wk))) return rc;
    if (window && (rc = alloc_work(ctx, "dwn", D, Wn))) return rc;
    const int64_t maxRC = std::max({D.Hq * d, d * f, D.Hq * d}), maxN = std::max({d, f, D.Hq});
    float *ystar, *y2star = nullptr, *dy, *g, *G, *mA, *vA, *dy2 = nullptr, *g2 = nullptr, *Uf;
    uint16_t *h1T, *OT, *uT, *zT;
    double *W, *Hacc, *parts, *lossd;
    uint8_t* dead;
    const int64_t npart = realq::dot_f32_partials();
    if ((rc = ws(ctx, "d_ystar", T * d, ystar)) || (rc = ws(ctx, "d_dy", T * d, dy)) || (rc = ws(ctx, "d_g", T * d, g)) ||
        (rc = ws(ctx, "d_G", maxRC, G)) || (rc = ws(ctx, "d_mA", maxRC, mA)) || (rc = ws(ctx, "d_vA", maxRC, vA)) ||
        (rc = ws(ctx, "d_h1T", d * T, h1T)) || (rc = ws(ctx, "d_OT", D.Hq * T, OT)) || (rc = ws(ctx, "d_uT", d * T, uT)) ||
        (rc = ws(ctx, "d_zT", f * T, zT)) || (rc = ws(ctx, "d_W", maxRC, W)) || (rc = ws(ctx, "d_H", maxN * maxN, Hacc)) ||
        (rc = ws(ctx, "d_U", maxN * maxN, Uf)) || (rc = ws(ctx, "d_dead", maxN, dead)) ||
        (rc = ws(ctx, "d_parts", 2 * npart, parts)) || (rc = ws(ctx, "d_loss", 1, lossd)))
        return rc;
    Split sdy, sdy2, sgT, svT;
    if ((rc = ws_split(ctx, "d_sdy", T * d, sdy)) || (rc = ws_split(ctx, "d_sgT", maxN * T, sgT)) ||
        (rc = ws_split(ctx, "d_svT", maxN * T, svT)))
        return rc;
    if (window && ((rc = ws(ctx, "d_y2star", T * d, y2star)) || (rc = ws(ctx, "d_dy2", T * d, dy2)) ||
                   (rc = ws(ctx, "d_g2", T * d, g2)) || (rc = ws_split(ctx, "d_sdy2", T * d, sdy2))))
        return rc;
    void* lin_tmp;  // sized once for every lin_bf16 of the sweep
    if ((rc = get_ws(ctx, "lin_tmp", (size_t)T * std::max(d, D.Hq) * 4, &lin_tmp))) return rc;
    {
        Timed tm(ctx, "block_init");
        if ((rc = dec_forward(ctx, wq, Dd->X, nullptr, D, Fs))) return rc;
        RQ_HIP(ctx, hipMemcpyAsync(ystar, Fs.mlp.y, (size_t)T * d * 4, hipMemcpyDeviceToDevice, s));
        if (window) {
            if ((rc = dec_forward(ctx, wn, nullptr, ystar, D, Fn))) return rc;
            RQ_HIP(ctx, hipMemcpyAsync(y2star, Fn.mlp.y, (size_t)T * d * 4, hipMemcpyDeviceToDevice, s));
        }
        if ((rc = dec_forward(ctx, wq, Dd->Xhat, nullptr, D, Fq))) return rc;
        RQ_HIP(ctx, realq::transpose_u16(Fq.h1, d, h1T, T, T, d, s));
    }

    // L_slide and g = dL_slide/dy at the quantized path's current forward Fq over the whole
    // sequences of tokens [t0, t0 + Tb); g holds those tokens' rows from row 0
    auto surrogate = [&](double alpha, int64_t t0, int64_t Tb) -> int {
        const DecF q = rows_of(Fq, D, t0);
        DecDims Db = D;
        Db.T = Tb;
        RQ_HIP(ctx, realq::residual_out_f32(q.x2, q.mlp.out, ystar + t0 * d, nullptr, dy, Tb * d, s));
        if (B0.mlp.F) {
            RQ_HIP(ctx, realq::scale_split(dy, 1.f, nullptr, sdy.hi, sdy.lo, Tb * d, s));
            if ((rc = prod3(ctx, sdy, Tb, d, wq.mlp.F, d, (float)(1.0 / (double)Tb), g))) return rc;
        } else {
            RQ_HIP(ctx, realq::scale_split(dy, (float)(1.0 / (double)Tb), g, nullptr, nullptr, Tb * d, s));
        }
        RQ_HIP(ctx, realq::dot_f32(dy, g, Tb * d, 0.5 * alpha, parts, s));
        if (window && alpha < 1.0) {
            RQ_HIP(ctx, realq::residual_out_f32(q.x2, q.mlp.out, nullptr, q.mlp.y, nullptr, Tb * d, s));
            if ((rc = dec_forward(ctx, wn, nullptr, q.mlp.y, Db, Fn))) return rc;
            RQ_HIP(ctx, realq::residual_out_f32(Fn.x2, Fn.mlp.out, y2star + t0 * d, nullptr, dy2, Tb * d, s));
            if (N0.mlp.F) {
                RQ_HIP(ctx, realq::scale_split(dy2, 1.f, nullptr, sdy2.hi, sdy2.lo, Tb * d, s));
                if ((rc = prod3(ctx, sdy2, Tb, d, wn.mlp.F, d, (float)(1.0 / (double)Tb), g2))) return rc;
            } else {
                RQ_HIP(ctx, realq::scale_split(dy2, (float)(1.0 / (double)Tb), g2, nullptr, nullptr, Tb * d, s));
            }
            RQ_HIP(ctx, realq::dot_f32(dy2, g2, Tb * d, 0.5 * (1.0 - alpha), parts + npart, s));
            // the next block's input gradient: through its MLP half, attention and first norm
            if ((rc = back_to_x2(ctx, wn, Db, Fn, g2, Wn)) || (rc = back_to_qkv(ctx, wn, Db, Fn, Wn))) return rc;
            RQ_HIP(ctx, realq::scale_split(Wn.dq, 1.f, nullptr, Wn.sdq.hi, Wn.sdq.lo, Tb * D.Hq, s));
            RQ_HIP(ctx, realq::scale_split(Wn.dk, 1.f, nullptr, Wn.sdk.hi, Wn.sdk.lo, Tb * D.Hk, s));
            RQ_HIP(ctx, realq::scale_split(Wn.dv, 1.f, nullptr, Wn.sdv.hi, Wn.sdv.lo, Tb * D.Hk, s));
            if ((rc = prod3(ctx, Wn.sdq, Tb, D.Hq, wn.qT, d, 1.f, Wn.dh1)) ||
                (rc = prod3_acc(ctx, Wn.sdk, Tb, D.Hk, wn.kT, d, Wn.dh1)) ||
                (rc = prod3_acc(ctx, Wn.sdv, Tb, D.Hk, wn.vT, d, Wn.dh1)))
                return rc;
            RQ_HIP(ctx, realq::rmsnorm_bwd_blend(q.mlp.y, Wn.dx2, Wn.dh1, wn.gamma1, D.eps, alpha, Tb, d, g, s));
            RQ_HIP(ctx, realq::reduce_partials(parts, 2 * npart, 1.0, lossd, s));
        } else {
            RQ_HIP(ctx, realq::reduce_partials(parts, npart, 1.0, lossd, s));
        }
        return REALQ_OK;
    };

    Split* fwd_slot[7] = {&wq.q, &wq.k, &wq.v, &wq.o, &wq.mlp.g, &wq.mlp.u, &wq.mlp.d};
    // forward of the quantized path over tokens [t0, t0 + Tb) from module mod's stage (its
    // weights changed); the earlier stages of those tokens are current in Fq
    auto refresh = [&](int mod, int64_t t0, int64_t Tb) -> int {
        DecF q = rows_of(Fq, D, t0);
        DecDims Db = D;
        Db.T = Tb;
        const uint16_t* xh = Dd->Xhat + t0 * d;
        if (mod <= 2) {
            if ((rc = dec_attn(ctx, wq, xh, nullptr, Db, q, 1 << mod, false))) return rc;
        }
        if (mod <= 3 && (rc = dec_o(ctx, wq, xh, nullptr, Db, q))) return rc;
        if (mod <= 3) return forward(ctx, wq.mlp, nullptr, q.x2, Tb, d, f, D.eps, q.mlp, nullptr, nullptr);
        if (mod == 4 && (rc = lin_f32(ctx, wq.mlp.g, f, d, q.mlp.u, Tb, q.mlp.a))) return rc;
        if (mod == 5 && (rc = lin_f32(ctx, wq.mlp.u, f, d, q.mlp.u, Tb, q.mlp.b))) return rc;
        if (mod <= 5) RQ_HIP(ctx, realq::swiglu_fwd(q.mlp.a, q.mlp.b, q.mlp.z, Tb * f, s));
        return lin_bf16(ctx, wq.mlp.d, d, f, q.mlp.z, Tb, q.mlp.out);
    };

    for (int mod = 0; mod < stop; ++mod) {
        const int64_t m = rows[mod], n = cols[mod];
        if (mod < start) {  // taken as already quantized
            RQ_HIP(ctx, hipMemcpyAsync(out->W_hat[mod], Dd->W_fixed[mod], (size_t)m * n * 4, hipMemcpyDeviceToDevice,
                                       s));
        } else {
            if (Dd->X_fixed && mod == start) {
                // this module's input taken as given; the quantized path recomputed from it on
                if (mod <= 2) {
                    RQ_HIP(ctx, hipMemcpyAsync(Fq.h1, Dd->X_fixed, (size_t)T * d * 2, hipMemcpyDeviceToDevice, s));
                    RQ_HIP(ctx, realq::transpose_u16(Fq.h1, d, h1T, T, T, d, s));
                    if ((rc = dec_attn(ctx, wq, Dd->Xhat, nullptr, D, Fq, 7, false))) return rc;
                    if ((rc = refresh(3, 0, T))) return rc;
                } else if (mod == 3) {
                    RQ_HIP(ctx, hipMemcpyAsync(Fq.O, Dd->X_fixed, (size_t)T * D.Hq * 2, hipMemcpyDeviceToDevice, s));
                    if ((rc = refresh(3, 0, T))) return rc;
                } else if (mod <= 5) {
                    RQ_HIP(ctx, hipMemcpyAsync(Fq.mlp.u, Dd->X_fixed, (size_t)T * d * 2, hipMemcpyDeviceToDevice, s));
                    if ((rc = lin_f32(ctx, wq.mlp.u, f, d, Fq.mlp.u, T, Fq.mlp.b))) return rc;
                    if ((rc = refresh(4, 0, T))) return rc;
                } else {
                    RQ_HIP(ctx, hipMemcpyAsync(Fq.mlp.z, Dd->X_fixed, (size_t)T * f * 2, hipMemcpyDeviceToDevice, s));
                    if ((rc = refresh(6, 0, T))) return rc;
                }
            }
            const uint16_t* inp = mod <= 2 ? Fq.h1 : (mod == 3 ? Fq.O : (mod <= 5 ? Fq.mlp.u : Fq.mlp.z));
            RQ_HIP(ctx, realq::fill_f64(Hacc, 0.0, n * n, s));
            if ((rc = realq_hessian_accum(ctx, inp, nullptr, T, n, Hacc))) return rc;
            if ((rc = realq_chol_inverse(ctx, Hacc, n, T, Dd->q.damp, nullptr, Uf, dead))) return rc;
            const uint16_t* inT = h1T;
            if (mod == 3) {
                RQ_HIP(ctx, realq::transpose_u16(Fq.O, D.Hq, OT, T, T, D.Hq, s));
                inT = OT;
            } else if (mod == 4 || mod == 5) {
                if (mod == 4 || start == 5) RQ_HIP(ctx, realq::transpose_u16(Fq.mlp.u, d, uT, T, T, d, s));
                inT = uT;
            } else if (mod == 6) {
                RQ_HIP(ctx, realq::transpose_u16(Fq.mlp.z, f, zT, T, T, f, s));
                inT = zT;
            }
            RQ_HIP(ctx, realq::widen_f32(W0[mod], W, m * n, s));
            RQ_HIP(ctx, realq::fill_f32(mA, 0.f, m * n, s));
            RQ_HIP(ctx, realq::fill_f32(vA, 0.f, m * n, s));
            int64_t t_adam = 0;
            for (int64_t b = 0; b < nb[mod]; ++b) {
                const int64_t c0 = b * blk, bs = std::min<int64_t>(blk, n - c0), c1 = c0 + bs;
                if ((rc = realq_quantize_block(ctx, W, m, n, c0, bs, Uf, dead, &Dd->q, out->codes[mod], out->scales[mod],
                                               out->zeros[mod], nullptr)))
                    return rc;
                if (steps == 0 || c1 >= n) continue;
                double alpha = 1.0;
                if (window && B_total > 1) {
                    const double bg = (double)(off[mod] + b + 1);
                    alpha = std::min(1.0, std::max(0.0, 1.0 - (bg - 1.0) / (double)(B_total - 1)));
                }
                const int64_t nJ = n - c1;
                for (int k = 0; k < steps; ++k) {
                    Timed tm(ctx, "block_step");
                    const TokenBatch tb = step_tokens(t_adam + 1, T, Dd->bgd.batch);
                    const int64_t Tb = tb.n;
                    const DecF q = rows_of(Fq, D, tb.t0);
                    DecDims Db = D;
                    Db.T = Tb;
                    fwd_slot[mod]->lo_zero = false;
                    RQ_HIP(ctx, realq::split3_f64(W, fwd_slot[mod]->hi, fwd_slot[mod]->lo, fwd_slot[mod]->lo2, m * n, s));
                    if ((rc = refresh(mod, tb.t0, Tb)) || (rc = surrogate(alpha, tb.t0, Tb))) return rc;
                    if (out->loss_trace)
                        RQ_HIP(ctx, hipMemcpyAsync(out->loss_trace + (off[mod] + b) * steps + k, lossd, 8,
                                                   hipMemcpyDeviceToDevice, s));
                    // gradient of this module's trailing columns over the step's tokens:
                    // (dL/d output)^T input[:, J] (the transposed input keeps its stride T)
                    const float* gout = nullptr;
                    int64_t gw = 0;
                    if (mod == 6) {
                        gout = g;
                        gw = d;
                    } else if (mod >= 4) {
                        RQ_HIP(ctx, realq::scale_split(g, 1.f, nullptr, Wk.sg.hi, Wk.sg.lo, Tb * d, s));
                        if ((rc = prod3(ctx, Wk.sg, Tb, d, wq.mlp.dT, f, 1.f, Wk.dz))) return rc;
                        RQ_HIP(ctx, realq::swiglu_bwd(Wk.dz, q.mlp.a, q.mlp.b, mod - 4, Tb, f, 1, svT.hi, svT.lo, Tb, s));
                    } else {
                        if ((rc = back_to_x2(ctx, wq, Db, q, g, Wk))) return rc;
                        if (mod == 3) {
                            gout = Wk.dx2;
                            gw = d;
                        } else {
                            if ((rc = back_to_qkv(ctx, wq, Db, q, Wk))) return rc;
                            gout = mod == 0 ? Wk.dq : (mod == 1 ? Wk.dk : Wk.dv);
                            gw = mod == 0 ? D.Hq : D.Hk;
                        }
                    }
                    const Split* A = &svT;
                    if (gout) {
                        RQ_HIP(ctx, realq::transpose_split_f32(gout, gw, sgT.hi, sgT.lo, Tb, Tb, gw, s));
                        A = &sgT;
                    }
                    realq::GemmArgs gg{A->hi, A->lo, Tb, inT + c1 * T + tb.t0, T, m, nJ, Tb, 1};
                    RQ_HIP(ctx, realq::gemm_store_f32(gg, G, nJ, 0, 1.f, s));
                    ++t_adam;
                    realq::AdamArgs a{};
                    a.W = W;
                    a.mA = mA;
                    a.vA = vA;
                    a.m = m;
                    a.n = n;
                    a.c1 = c1;
                    a.lr = Dd->bgd.lr;
                    a.beta1 = Dd->bgd.beta1;
                    a.beta2 = Dd->bgd.beta2;
                    a.eps = Dd->bgd.eps;
                    a.bc1 = (float)(1.0 / (1.0 - std::pow((double)Dd->bgd.beta1, (double)t_adam)));
                    a.bc2 = (float)(1.0 / (1.0 - std::pow((double)Dd->bgd.beta2, (double)t_adam)));
                    a.gscale = 1.f;
                    RQ_HIP(ctx, realq::adam_update_dense(a, G, s));
                }
            }
            RQ_HIP(ctx, realq::narrow_f64(W, out->W_hat[mod], m * n, s));
        }
        fwd_slot[mod]->lo_zero = false;
        RQ_HIP(ctx, realq::split3_f32(out->W_hat[mod], n, fwd_slot[mod]->hi, fwd_slot[mod]->lo, fwd_slot[mod]->lo2, n,
                                      m, n, s));
        if ((rc = refresh(mod, 0, T))) return rc;
    }
    if ((rc = surrogate(1.0, 0, T))) return rc;
    RQ_HIP(ctx, hipEventRecord(ev.b, s));
    RQ_HIP(ctx, hipMemcpyAsync(&out->loss_final, lossd, 8, hipMemcpyDeviceToHost, s));
    RQ_HIP(ctx, hipStreamSynchronize(s));
    float ms = 0.f;
    RQ_HIP(ctx, hipEventElapsedTime(&ms, ev.a, ev.b));
    out->ms_total = ms;
    return realq::harvest(ctx);
}
