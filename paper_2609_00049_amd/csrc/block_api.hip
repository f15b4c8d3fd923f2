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

struct Split {  // a float32 matrix as a bf16 hi/lo pair
    uint16_t* hi = nullptr;
    uint16_t* lo = nullptr;
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

template <class T>
int ws(realq_ctx* ctx, const char* name, int64_t count, T*& p) {
    void* v;
    int rc = get_ws(ctx, name, (size_t)count * sizeof(T), &v);
    p = (T*)v;
    return rc;
}

// out[t][i] = sum_k act[t][k] W[i][k] (W as hi/lo, act bf16 [T][K]), token-major float32 [T][rows]
int lin_f32(realq_ctx* ctx, const Split& W, int64_t rows, int64_t K, const uint16_t* act, int64_t T, float* out) {
    realq::GemmArgs g{W.hi, W.lo, K, act, K, rows, T, K, 1};
    RQ_HIP(ctx, realq::gemm_store_f32_t(g, out, rows, ctx->stream));
    return REALQ_OK;
}
// same, rounded to bf16
int lin_bf16(realq_ctx* ctx, const Split& W, int64_t rows, int64_t K, const uint16_t* act, int64_t T, uint16_t* out) {
    realq::GemmArgs g{W.hi, W.lo, K, act, K, rows, T, K, 1};
    RQ_HIP(ctx, realq::gemm_store_bf16_t(g, out, rows, ctx->stream));
    return REALQ_OK;
}
// C[r][c] = alpha sum_k X[r][k] Y[c][k] with both operands float32 as hi/lo pairs:
// (Xhi + Xlo) Yhi + Xhi Ylo, float32 [rows][cols]
int prod3(realq_ctx* ctx, const Split& X, int64_t rows, int64_t K, const Split& Y, int64_t cols, float alpha,
          float* C) {
    realq::GemmArgs g{X.hi, X.lo, K, Y.hi, K, rows, cols, K, 1};
    RQ_HIP(ctx, realq::gemm_store_f32(g, C, cols, 0, alpha, ctx->stream));
    realq::GemmArgs g2{X.hi, nullptr, K, Y.lo, K, rows, cols, K, 1};
    RQ_HIP(ctx, realq::gemm_acc_f32(g2, C, cols, alpha, ctx->stream));
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
    if ((rc = ws_split(ctx, t + "g", f * d, w.g)) || (rc = ws_split(ctx, t + "u", f * d, w.u)) ||
        (rc = ws_split(ctx, t + "d", d * f, w.d)) || (rc = ws_split(ctx, t + "dT", f * d, w.dT)))
        return rc;
    RQ_HIP(ctx, realq::split_diff_f32(b.Wg, d, nullptr, 0, w.g.hi, w.g.lo, d, f, d, s));
    RQ_HIP(ctx, realq::split_diff_f32(b.Wu, d, nullptr, 0, w.u.hi, w.u.lo, d, f, d, s));
    RQ_HIP(ctx, realq::split_diff_f32(b.Wd, f, nullptr, 0, w.d.hi, w.d.lo, f, d, f, s));
    RQ_HIP(ctx, realq::transpose_split_f32(b.Wd, f, w.dT.hi, w.dT.lo, d, d, f, s));
    if (backward) {
        if ((rc = ws_split(ctx, t + "gT", d * f, w.gT)) || (rc = ws_split(ctx, t + "uT", d * f, w.uT))) return rc;
        RQ_HIP(ctx, realq::transpose_split_f32(b.Wg, d, w.gT.hi, w.gT.lo, f, f, d, s));
        RQ_HIP(ctx, realq::transpose_split_f32(b.Wu, d, w.uT.hi, w.uT.lo, f, f, d, s));
    }
    if (b.F) {
        if ((rc = ws_split(ctx, t + "F", d * d, w.F))) return rc;
        RQ_HIP(ctx, realq::split_diff_f32(b.F, d, nullptr, 0, w.F.hi, w.F.lo, d, d, d, s));
    }
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
    if (D->bgd.form != REALQ_BGD_TOKENS || D->bgd.loss_clip != 0.f || D->bgd.batch != 0)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "mlp_block_sweep: form, loss_clip and batch must be 0");
    const realq_mlp_block& B0 = D->blk;
    if (!D->X || !D->Xhat || !B0.gamma || !B0.Wg || !B0.Wu || !B0.Wd)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "mlp_block_sweep: NULL input or weight");
    const bool has_next = D->next.Wg != nullptr;
    if (has_next && (!D->next.gamma || !D->next.Wu || !D->next.Wd))
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "mlp_block_sweep: incomplete next block");
    if (!(D->eps > 0.f) || !std::isfinite(D->eps))
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "mlp_block_sweep: eps must be finite and > 0");
    for (int k = 0; k < 3; ++k)
        if (!out->codes[k] || !out->scales[k] || !out->zeros[k] || !out->W_hat[k])
            return set_error(ctx, REALQ_ERR_INVALID_ARG, "mlp_block_sweep: NULL output array");
    const bool window = D->window != 0 && has_next;
    const double eps = (double)D->eps;
    hipStream_t s = ctx->stream;
    hipEvent_t ev0, ev1;
    RQ_HIP(ctx, hipEventCreate(&ev0));
    RQ_HIP(ctx, hipEventCreate(&ev1));
    RQ_HIP(ctx, hipEventRecord(ev0, s));

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
        (rc = ws_split(ctx, "m_sW", maxRC, sW)))
        return rc;
    if (window) {
        if ((rc = ws(ctx, "m_y2star", T * d, y2star)) || (rc = ws(ctx, "m_dy2", T * d, dy2)) ||
            (rc = ws(ctx, "m_g2", T * d, g2)) || (rc = ws(ctx, "m_dz2", T * f, dz2)) ||
            (rc = ws(ctx, "m_du2", T * d, du2)) || (rc = ws_split(ctx, "m_sdy2", T * d, sdy2)) ||
            (rc = ws_split(ctx, "m_sg2", T * d, sg2)) || (rc = ws_split(ctx, "m_sda2", T * f, sda2)) ||
            (rc = ws_split(ctx, "m_sdb2", T * f, sdb2)))
            return rc;
    }
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
        RQ_HIP(ctx, realq::transpose_u16(fq.u, d, uT, T, T, d, s));
    }

    // L (and L_next) at the quantized path's current forward fq; g = dL_slide/dy.  Returns
    // the loss on the device in *lossd (scaled partial sums reduced in a fixed order).
    auto surrogate = [&](double alpha) -> int {
        RQ_HIP(ctx, realq::residual_out_bf16(D->Xhat, fq.out, ystar, nullptr, dy, T * d, s));
        if (B0.F) {
            RQ_HIP(ctx, realq::scale_split(dy, 1.f, nullptr, sdy.hi, sdy.lo, T * d, s));
            if ((rc = prod3(ctx, sdy, T, d, w0.F, d, (float)(1.0 / (double)T), g))) return rc;
        } else {
            RQ_HIP(ctx, realq::scale_split(dy, (float)(1.0 / (double)T), g, nullptr, nullptr, T * d, s));
        }
        RQ_HIP(ctx, realq::dot_f32(dy, g, T * d, 0.5 * alpha, parts, s));
        if (window && alpha < 1.0) {
            // next block on y = Xhat + out, its loss, and its input gradient blended into g
            RQ_HIP(ctx, realq::residual_out_bf16(D->Xhat, fq.out, nullptr, fq.y, nullptr, T * d, s));
            if ((rc = forward(ctx, w2, nullptr, fq.y, T, d, f, eps, fn, y2star, dy2))) return rc;
            if (D->next.F) {
                RQ_HIP(ctx, realq::scale_split(dy2, 1.f, nullptr, sdy2.hi, sdy2.lo, T * d, s));
                if ((rc = prod3(ctx, sdy2, T, d, w2.F, d, (float)(1.0 / (double)T), g2))) return rc;
            } else {
                RQ_HIP(ctx, realq::scale_split(dy2, (float)(1.0 / (double)T), g2, nullptr, nullptr, T * d, s));
            }
            RQ_HIP(ctx, realq::dot_f32(dy2, g2, T * d, 0.5 * (1.0 - alpha), parts + npart, s));
            RQ_HIP(ctx, realq::scale_split(g2, 1.f, nullptr, sg2.hi, sg2.lo, T * d, s));
            if ((rc = prod3(ctx, sg2, T, d, w2.dT, f, 1.f, dz2))) return rc;  // dz2 = g2 Wd2
            RQ_HIP(ctx, realq::swiglu_bwd(dz2, fn.a, fn.b, 0, T, f, 0, sda2.hi, sda2.lo, f, s));
            RQ_HIP(ctx, realq::swiglu_bwd(dz2, fn.a, fn.b, 1, T, f, 0, sdb2.hi, sdb2.lo, f, s));
            if ((rc = prod3(ctx, sda2, T, f, w2.gT, d, 1.f, du2))) return rc;  // du2 = da2 Wg2 + db2 Wu2
            realq::GemmArgs a1{sdb2.hi, sdb2.lo, f, w2.uT.hi, f, T, d, f, 1};
            RQ_HIP(ctx, realq::gemm_acc_f32(a1, du2, d, 1.f, s));
            realq::GemmArgs a2{sdb2.hi, nullptr, f, w2.uT.lo, f, T, d, f, 1};
            RQ_HIP(ctx, realq::gemm_acc_f32(a2, du2, d, 1.f, s));
            RQ_HIP(ctx, realq::rmsnorm_bwd_blend(fq.y, g2, du2, D->next.gamma, eps, alpha, T, d, g, s));
            RQ_HIP(ctx, realq::reduce_partials(parts, 2 * npart, 1.0, lossd, s));
        } else {
            RQ_HIP(ctx, realq::reduce_partials(parts, npart, 1.0, lossd, s));
        }
        return REALQ_OK;
    };

    const float* Wq[3] = {nullptr, nullptr, nullptr};  // quantized weights of finished modules
    for (int mod = 0; mod < 3; ++mod) {
        const int64_t m = rows[mod], n = cols[mod];
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
                // forward of the partially quantized block with this module's current weights
                RQ_HIP(ctx, realq::split_f64(W, sW.hi, sW.lo, m * n, s));
                if (mod == 0) {
                    if ((rc = lin_f32(ctx, sW, f, d, fq.u, T, fq.a))) return rc;
                } else if (mod == 1) {
                    if ((rc = lin_f32(ctx, sW, f, d, fq.u, T, fq.b))) return rc;
                }
                if (mod < 2) RQ_HIP(ctx, realq::swiglu_fwd(fq.a, fq.b, fq.z, T * f, s));
                if ((rc = lin_bf16(ctx, mod == 2 ? sW : w0.d, d, f, fq.z, T, fq.out))) return rc;
                if ((rc = surrogate(alpha))) return rc;
                if (out->loss_trace)
                    RQ_HIP(ctx, hipMemcpyAsync(out->loss_trace + (off[mod] + b) * steps + k, lossd, 8,
                                               hipMemcpyDeviceToDevice, s));
                // gradient of this module's trailing columns
                if (mod < 2) {
                    RQ_HIP(ctx, realq::scale_split(g, 1.f, nullptr, sg.hi, sg.lo, T * d, s));
                    if ((rc = prod3(ctx, sg, T, d, w0.dT, f, 1.f, dz))) return rc;  // dz = g Wd
                    RQ_HIP(ctx, realq::swiglu_bwd(dz, fq.a, fq.b, mod, T, f, 1, svT.hi, svT.lo, T, s));
                    realq::GemmArgs gg{svT.hi, svT.lo, T, uT + c1 * T, T, f, nJ, T, 1};
                    RQ_HIP(ctx, realq::gemm_store_f32(gg, G, nJ, 0, 1.f, s));
                } else {
                    RQ_HIP(ctx, realq::transpose_split_f32(g, d, sgT.hi, sgT.lo, T, T, d, s));
                    realq::GemmArgs gg{sgT.hi, sgT.lo, T, zT + c1 * T, T, d, nJ, T, 1};
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
        Wq[mod] = out->W_hat[mod];
        // the quantized path with this module's final weights
        Split q;
        if ((rc = ws_split(ctx, "m_sq", m * n, q))) return rc;
        RQ_HIP(ctx, realq::split_diff_f32(Wq[mod], n, nullptr, 0, q.hi, q.lo, n, m, n, s));
        if (mod == 0 && (rc = lin_f32(ctx, q, f, d, fq.u, T, fq.a))) return rc;
        if (mod == 1 && (rc = lin_f32(ctx, q, f, d, fq.u, T, fq.b))) return rc;
        if (mod < 2) RQ_HIP(ctx, realq::swiglu_fwd(fq.a, fq.b, fq.z, T * f, s));
        if ((rc = lin_bf16(ctx, mod == 2 ? q : w0.d, d, f, fq.z, T, fq.out))) return rc;
    }
    // own-block loss at the quantized weights (fq holds the final forward)
    if ((rc = surrogate(1.0))) return rc;
    RQ_HIP(ctx, hipEventRecord(ev1, s));
    RQ_HIP(ctx, hipMemcpyAsync(&out->loss_final, lossd, 8, hipMemcpyDeviceToHost, s));
    RQ_HIP(ctx, hipStreamSynchronize(s));
    float ms = 0.f;
    RQ_HIP(ctx, hipEventElapsedTime(&ms, ev0, ev1));
    out->ms_total = ms;
    (void)hipEventDestroy(ev0);
    (void)hipEventDestroy(ev1);
    return realq::harvest(ctx);
}
