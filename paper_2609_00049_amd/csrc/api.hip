// C ABI of the REAL-Q layer sweep (declared in include/realq.h): argument checks,
// workspace management, and the launch sequences of the five public calls.
// Everything runs on the context's stream; the only host synchronisations are the
// positive-definiteness check of realq_chol_inverse and the end of
// realq_quantize_layer.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "common.h"
#include "ctx.h"
#include "kernels.h"
#include "plan.h"
#include "../../include/realq.h"

namespace realq {

int set_error(realq_ctx* ctx, int code, const std::string& msg) {
    if (ctx) ctx->err = msg;
    return code;
}

int get_ws(realq_ctx* ctx, const char* slot, size_t bytes, void** out) {
    auto& b = ctx->ws[slot];
    if (bytes == 0) bytes = 16;
    if (b.bytes < bytes) {
        if (b.p) {
            hipError_t e = hipStreamSynchronize(ctx->stream);
            if (e != hipSuccess) return set_error(ctx, REALQ_ERR_HIP, std::string("sync: ") + hipGetErrorString(e));
            (void)hipFree(b.p);
            b.p = nullptr;
            b.bytes = 0;
        }
        void* p = nullptr;
        if (hipMalloc(&p, bytes) != hipSuccess || !p) {
            (void)hipGetLastError();
            return set_error(ctx, REALQ_ERR_OOM,
                             std::string("device allocation of ") + std::to_string(bytes) + " bytes for " + slot);
        }
        b.p = p;
        b.bytes = bytes;
    }
    *out = b.p;
    return REALQ_OK;
}

int harvest(realq_ctx* ctx) {
    if (ctx->pending.empty()) return REALQ_OK;
    RQ_HIP(ctx, hipEventSynchronize(ctx->pending.back().b));
    for (auto& p : ctx->pending) {
        float ms = 0.f;
        RQ_HIP(ctx, hipEventElapsedTime(&ms, p.a, p.b));
        auto& s = ctx->stats[p.name];
        s.launches += 1;
        s.ms += ms;
        ctx->free_events.push_back({p.a, p.b});
    }
    ctx->pending.clear();
    return REALQ_OK;
}

}  // namespace realq

using realq::get_ws;
using realq::validate_bgd;
using realq::validate_q;
using realq::set_error;
using realq::Timed;

// ============================================================================ BGD state

struct realq_bgd_state {
    realq_ctx* ctx = nullptr;
    int64_t m = 0, n = 0, T = 0, Tc = 0;
    const float* W0 = nullptr;
    const uint16_t* X = nullptr;
    const uint16_t* Xhat = nullptr;
    const float* s = nullptr;
    const float* M = nullptr;
    const float* P = nullptr;
    realq_bgd_params prm{};
    int64_t t = 0;  // Adam step counter (one per module)
    int64_t locked = 0;  // columns [0, locked) are folded into the residual base
    bool owns = true;
    float* B = nullptr;  // [m,T] residual base
    float* mA = nullptr;
    float* vA = nullptr;  // [m,n]
    uint16_t* Dhi = nullptr;
    uint16_t* Dlo = nullptr;  // [m,n] split(W - W0)
    uint16_t* XhT = nullptr;  // [n,T]
    uint16_t* Rhi = nullptr;  // split(R o s): blocked layout [m, r_ld(Tc)], or with the clip
    uint16_t* Rlo = nullptr;  // two arrays Rhi/Rlo [m, Tc]
    int64_t Tb = 0, nbatch = 1;  // tokens per step and number of batches (mini-batch BGD)
    float* Rf = nullptr;         // [m,Tc] residual kept whole for the clip
    float* tau = nullptr;        // [Tc] per-token clip thresholds
    // increments within a column block: L0 the loss of the block's first step (device scalar),
    // G0 its gradient ([m, n - c1], unscaled sum over tokens), Dacc [m,n] the weight change since
    // then and Dinc = bf16(Dacc); inc_c1 names the block they belong to (-1: none) and inc_ready
    // says Dinc holds the change of the current weights
    bool inc = false;
    double* L0 = nullptr;
    float* G0 = nullptr;
    float* Dacc = nullptr;
    uint16_t* Dinc = nullptr;
    int64_t inc_c1 = -1;
    bool inc_ready = false;
    int64_t inc_taken = 0;  // later steps taken since the block's first (at most steps - 1)
    // Gram form
    bool gram = false;
    uint16_t* Ghi = nullptr;
    uint16_t* Glo = nullptr;  // [n,n] split(Xhat^T S Xhat)
    float* C0 = nullptr;      // [m,n] W0 Delta^T S Xhat
    float* Pm = nullptr;      // [m,n] D Xhat^T S Xhat (per step)
    double* cconst = nullptr; // <W0 Delta^T S Delta, W0> (device scalar)
    // blended metric alpha M + (1 - alpha) P as a bf16 pair [m,m], formed once per alpha
    uint16_t* Mah = nullptr;
    uint16_t* Mal = nullptr;
    float Ma_alpha = -1.f;
    std::vector<void*> allocations;
};

extern "C" {

void realq_qparams_default(realq_qparams* q) {
    if (!q) return;
    q->bits = 4;
    q->group = 128;
    q->block = 128;
    q->grid = 80;
    q->damp = 0.01f;
}

void realq_bgd_params_default(realq_bgd_params* b) {
    if (!b) return;
    b->steps = 0;
    b->lr = 1e-3f;
    b->beta1 = 0.9f;
    b->beta2 = 0.999f;
    b->eps = 1e-8f;
    b->tok_chunk = 0;
    b->form = REALQ_BGD_TOKENS;
    b->loss_clip = 0.f;
    b->batch = 0;
    b->resid_increment = 1;
}

int realq_ctx_create(realq_ctx** out, void* hip_stream) {
    if (!out) return REALQ_ERR_INVALID_ARG;
    *out = nullptr;
    realq_ctx* c = new (std::nothrow) realq_ctx();
    if (!c) return REALQ_ERR_OOM;
    c->stream = (hipStream_t)hip_stream;
    if (hipGetDevice(&c->device) != hipSuccess ||
        hipDeviceGetAttribute(&c->cus, hipDeviceAttributeMultiprocessorCount, c->device) != hipSuccess) {
        (void)hipGetLastError();
        delete c;
        return REALQ_ERR_HIP;
    }
    if (c->cus < 1) c->cus = 1;
    *out = c;
    return REALQ_OK;
}

void realq_ctx_destroy(realq_ctx* ctx) {
    if (!ctx) return;
    (void)hipStreamSynchronize(ctx->stream);
    for (auto& kv : ctx->ws)
        if (kv.second.p) (void)hipFree(kv.second.p);
    for (auto& p : ctx->pending) {
        (void)hipEventDestroy(p.a);
        (void)hipEventDestroy(p.b);
    }
    for (auto& p : ctx->free_events) {
        (void)hipEventDestroy(p.first);
        (void)hipEventDestroy(p.second);
    }
    delete ctx;
}

const char* realq_last_error(const realq_ctx* ctx) { return ctx ? ctx->err.c_str() : "null context"; }

int realq_ctx_set_timing(realq_ctx* ctx, int enable) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    ctx->timing = enable != 0;
    return REALQ_OK;
}

static const char* kTimedNames[] = {"hessian",    "chol",      "quantize",   "obs",        "lock",
                                    "resid",      "grad",      "resid_inc",  "grad_inc",   "adam",
                                    "init",       "gram",      "gram_step",  "dense_loss", "saliency",
                                    "block_init", "block_step", "attention", "metric"};

int realq_ctx_kernel_time(realq_ctx* ctx, const char* name, int64_t* launches, double* total_ms) {
    if (!ctx || !name) return REALQ_ERR_INVALID_ARG;
    bool known = false;
    for (const char* k : kTimedNames) known |= std::strcmp(k, name) == 0;
    if (!known) return set_error(ctx, REALQ_ERR_INVALID_ARG, std::string("unknown kernel name ") + name);
    int rc = realq::harvest(ctx);
    if (rc) return rc;
    auto it = ctx->stats.find(name);
    if (launches) *launches = it == ctx->stats.end() ? 0 : it->second.launches;
    if (total_ms) *total_ms = it == ctx->stats.end() ? 0.0 : it->second.ms;
    return REALQ_OK;
}

int realq_ctx_reset_timing(realq_ctx* ctx) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    int rc = realq::harvest(ctx);
    ctx->stats.clear();
    return rc;
}

// ============================================================================ a1: Hessian

}  // extern "C"

// Token chunks of tc tokens staged in caller-provided bf16 buffers of n * tc elements each (xt, and
// hi, lo, lo2 when s is given): the chunk transposed (and, with weights, s_t xhat_t split into three
// bf16 terms), then H_acc += chunk^T chunk on MFMA with a float64 epilogue.  timed = false skips the
// timing events (the allocation-free entry point creates none).
int realq::hessian_accum_chunks(realq_ctx* ctx, const uint16_t* Xhat, const float* s, int64_t T, int64_t n,
                                double* H_acc, int64_t tc, uint16_t* xt, uint16_t* hi, uint16_t* lo, uint16_t* lo2,
                                bool timed) {
    Timed tm(ctx, timed ? "hessian" : nullptr);
    for (int64_t t0 = 0; t0 < T; t0 += tc) {
        const int64_t cur = std::min(tc, T - t0);
        RQ_HIP(ctx, realq::transpose_u16(Xhat + t0 * n, n, xt, tc, cur, n, ctx->stream));
        realq::GemmArgs g{};
        g.B = xt;
        g.ldb = tc;
        g.M = n;
        g.N = n;
        g.K = cur;
        g.lda = tc;
        g.splits = 1;
        if (s) {
            // s_t xhat_t in three bf16 terms: with a heavy-tailed s a few tokens carry H, and the
            // 2^-17 remainder of a hi/lo pair would not average out over the tokens
            RQ_HIP(ctx, realq::transpose_scale_split(Xhat + t0 * n, n, s + t0, hi, lo, lo2, tc, cur, n, ctx->stream));
            g.Ahi = hi;
            g.Alo = lo;
        } else {
            g.Ahi = xt;
            g.Alo = nullptr;
        }
        RQ_HIP(ctx, realq::gemm_acc_f64(g, H_acc, n, ctx->stream));
        if (s) {
            g.Ahi = lo2;
            g.Alo = nullptr;
            RQ_HIP(ctx, realq::gemm_acc_f64(g, H_acc, n, ctx->stream));
        }
    }
    return REALQ_OK;
}

extern "C" {

int realq_hessian_accum(realq_ctx* ctx, const uint16_t* Xhat, const float* s, int64_t T, int64_t n, double* H_acc) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (T < 0 || n <= 0) return set_error(ctx, REALQ_ERR_SHAPE, "hessian_accum: need T >= 0, n > 0");
    if (T == 0) return REALQ_OK;
    if (!Xhat || !H_acc) return set_error(ctx, REALQ_ERR_INVALID_ARG, "hessian_accum: NULL Xhat or H_acc");
    // token chunk bounded so the transposed workspace stays near 256 MiB per operand
    int64_t tc = (int64_t)(128ll << 20) / n;
    tc = tc < 256 ? 256 : (tc / 256) * 256;
    if (tc > T) tc = ((T + 7) / 8) * 8;
    void *xt = nullptr, *hi = nullptr, *lo = nullptr, *lo2 = nullptr;
    int rc = get_ws(ctx, "h_xt", (size_t)n * tc * 2, &xt);
    if (rc) return rc;
    if (s) {
        if ((rc = get_ws(ctx, "h_hi", (size_t)n * tc * 2, &hi))) return rc;
        if ((rc = get_ws(ctx, "h_lo", (size_t)n * tc * 2, &lo))) return rc;
        if ((rc = get_ws(ctx, "h_lo2", (size_t)n * tc * 2, &lo2))) return rc;
    }
    return realq::hessian_accum_chunks(ctx, Xhat, s, T, n, H_acc, tc, (uint16_t*)xt, (uint16_t*)hi, (uint16_t*)lo,
                                       (uint16_t*)lo2, true);
}

// ============================================================================ a0: Stage-0 accumulators

int realq_fisher_accum(realq_ctx* ctx, const uint16_t* G, int64_t T, int64_t m, double* F_acc) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (T < 0 || m <= 0) return set_error(ctx, REALQ_ERR_SHAPE, "fisher_accum: need T >= 0, m > 0");
    if (T == 0) return REALQ_OK;
    if (!G || !F_acc) return set_error(ctx, REALQ_ERR_INVALID_ARG, "fisher_accum: NULL G or F_acc");
    // sum_t g_t g_t^T is the unweighted Hessian contraction with the gradients in place of the inputs
    return realq_hessian_accum(ctx, G, nullptr, T, m, F_acc);
}

int realq_fisher_finish(realq_ctx* ctx, const double* F_acc, int64_t m, int64_t T_total, float* F) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (m <= 0 || T_total <= 0) return set_error(ctx, REALQ_ERR_SHAPE, "fisher_finish: need m > 0, T_total > 0");
    if (!F_acc || !F) return set_error(ctx, REALQ_ERR_INVALID_ARG, "fisher_finish: NULL F_acc or F");
    RQ_HIP(ctx, realq::div_narrow(F_acc, (double)T_total, F, m * m, ctx->stream));
    return REALQ_OK;
}

int realq_saliency(realq_ctx* ctx, const uint16_t* G, int64_t T, int64_t m, int32_t n_groups, float clip_q,
                   float* s_out) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (T < 0 || m <= 0) return set_error(ctx, REALQ_ERR_SHAPE, "saliency: need T >= 0, m > 0");
    if (n_groups < 1 || n_groups > m) return set_error(ctx, REALQ_ERR_INVALID_ARG, "saliency: need 1 <= n_groups <= m");
    if (!std::isfinite(clip_q) || clip_q < 0.f || clip_q > 1.f)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "saliency: clip_q must lie in [0, 1] (0 = off)");
    if (T == 0) return REALQ_OK;
    if (!G || !s_out) return set_error(ctx, REALQ_ERR_INVALID_ARG, "saliency: NULL G or s_out");
    const int64_t k = clip_q > 0.f ? std::max<int64_t>(1, (int64_t)std::ceil((double)clip_q * (double)T)) : 0;
    void *s64, *tau, *sel;
    int rc;
    if ((rc = get_ws(ctx, "sal_s", (size_t)n_groups * T * 8, &s64))) return rc;
    if ((rc = get_ws(ctx, "sal_tau", (size_t)n_groups * 8, &tau))) return rc;
    if ((rc = get_ws(ctx, "sal_sel", (size_t)realq::saliency_select_bytes(n_groups), &sel))) return rc;
    Timed tm(ctx, "saliency");
    RQ_HIP(ctx, realq::saliency(G, T, m, n_groups, k, (double*)s64, (double*)tau, sel, s_out, ctx->stream));
    return REALQ_OK;
}

// ============================================================================ a2: inverse factor

int realq_chol_inverse(realq_ctx* ctx, const double* H_acc, int64_t n, int64_t T_total, float damp, float* H_out,
                       float* U, uint8_t* dead) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (n <= 0 || T_total <= 0) return set_error(ctx, REALQ_ERR_SHAPE, "chol_inverse: need n > 0 and T_total > 0");
    if (!H_acc || !U) return set_error(ctx, REALQ_ERR_INVALID_ARG, "chol_inverse: NULL H_acc or U");
    if (!(damp > 0.f) || !std::isfinite(damp))
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "chol_inverse: damp must be finite and > 0");
    const int64_t np = ((n + 63) / 64) * 64;
    void *A, *L, *D, *F, *S;
    int rc;
    if ((rc = get_ws(ctx, "c_A", (size_t)np * np * 8, &A))) return rc;
    if ((rc = get_ws(ctx, "c_L", (size_t)np * np * 8, &L))) return rc;
    if ((rc = get_ws(ctx, "c_D", (size_t)np * 64 * 8, &D))) return rc;
    if ((rc = get_ws(ctx, "c_F", 64, &F))) return rc;
    if ((rc = get_ws(ctx, "c_S", 64, &S))) return rc;
    // two flag words (not positive definite; non-finite accumulator) cleared by one double fill
    RQ_HIP(ctx, realq::fill_f64((double*)F, 0.0, 1, ctx->stream));
    realq::CholArgs c{};
    c.Hacc = H_acc;
    c.n = n;
    c.np = np;
    c.scale = 2.0 / (double)T_total;
    c.damp = damp;
    c.Hout = H_out;
    c.dead = dead;
    c.A = (double*)A;
    c.Linv = (double*)L;
    c.diaginv = (double*)D;
    c.flag = (int*)F;
    c.scratch = (double*)S;
    c.U = U;
    {
        Timed tm(ctx, "chol");
        RQ_HIP(ctx, realq::chol_inverse(c, ctx->stream));
    }
    int flag[2] = {0, 0};
    RQ_HIP(ctx, hipMemcpyAsync(flag, F, sizeof(flag), hipMemcpyDeviceToHost, ctx->stream));
    RQ_HIP(ctx, hipStreamSynchronize(ctx->stream));
    if (flag[1])
        return set_error(ctx, REALQ_ERR_NONFINITE,
                         "chol_inverse: the Hessian accumulator holds NaN or Inf (non-finite Xhat or s)");
    if (flag[0]) return set_error(ctx, REALQ_ERR_NOT_SPD, "chol_inverse: damped Hessian is not positive definite");
    return REALQ_OK;
}

// ============================================================================ BGD state

// Row stride (bf16 values) of split(R o s) in the blocked layout for `cur` tokens: hi and lo of
// every 32 tokens, rounded up to whole blocks.
static int64_t r_ld(int64_t cur) { return 2 * ((cur + 31) / 32) * 32; }
// row stride of bf16(acc o s) on a later step of a column block (row-major, in the same buffer)
static int64_t q_ld(int64_t cur) { return ((cur + 31) / 32) * 32; }

static int state_alloc(realq_bgd_state* st, void** p, size_t bytes, const char* slot) {
    realq_ctx* ctx = st->ctx;
    if (!st->owns) return get_ws(ctx, slot, bytes, p);
    *p = nullptr;
    if (hipMalloc(p, bytes ? bytes : 16) != hipSuccess || !*p) {
        (void)hipGetLastError();
        return set_error(ctx, REALQ_ERR_OOM, std::string("device allocation of ") + std::to_string(bytes) + " bytes");
    }
    st->allocations.push_back(*p);
    return REALQ_OK;
}

static void state_free(realq_bgd_state* st) {
    if (!st) return;
    if (st->ctx) (void)hipStreamSynchronize(st->ctx->stream);
    for (void* p : st->allocations) (void)hipFree(p);
    st->allocations.clear();
}

// Calibration Gram matrices of the input perturbation Delta = Xhat - X, accumulated over token
// chunks in float64: Gdh = Delta^T S Xhat and Gdd = Delta^T S Delta (S = diag(s) or I).  The
// float32 operand s o Delta is carried as a hi/lo bf16 pair against Xhat (bf16) and against
// both halves of Delta.
static int gram_accum(realq_ctx* ctx, const uint16_t* Xhat, const uint16_t* X, const float* sw, int64_t T, int64_t n,
                      double* Gdh, double* Gdd) {
    hipStream_t s = ctx->stream;
    int rc;
    void *sdh, *sdl, *dh, *dl, *xt;
    int64_t tc = (int64_t)(128ll << 20) / n;
    tc = tc < 256 ? 256 : (tc / 256) * 256;
    if (tc > T) tc = ((T + 7) / 8) * 8;
    if ((rc = get_ws(ctx, "g_sdh", (size_t)n * tc * 2, &sdh))) return rc;
    if ((rc = get_ws(ctx, "g_sdl", (size_t)n * tc * 2, &sdl))) return rc;
    if ((rc = get_ws(ctx, "g_dh16", (size_t)n * tc * 2, &dh))) return rc;
    if ((rc = get_ws(ctx, "g_dl16", (size_t)n * tc * 2, &dl))) return rc;
    if ((rc = get_ws(ctx, "g_xt", (size_t)n * tc * 2, &xt))) return rc;
    Timed tm(ctx, "gram");
    RQ_HIP(ctx, realq::fill_f64(Gdh, 0.0, n * n, s));
    RQ_HIP(ctx, realq::fill_f64(Gdd, 0.0, n * n, s));
    for (int64_t t0 = 0; t0 < T; t0 += tc) {
        const int64_t cur = std::min(tc, T - t0);
        RQ_HIP(ctx, realq::transpose_delta_split(Xhat + t0 * n, X + t0 * n, n, sw ? sw + t0 : nullptr, (uint16_t*)sdh,
                                                 (uint16_t*)sdl, (uint16_t*)dh, (uint16_t*)dl, tc, cur, n, s));
        RQ_HIP(ctx, realq::transpose_u16(Xhat + t0 * n, n, (uint16_t*)xt, tc, cur, n, s));
        realq::GemmArgs g{(const uint16_t*)sdh, (const uint16_t*)sdl, tc, (const uint16_t*)xt, tc, n, n, cur, 1};
        RQ_HIP(ctx, realq::gemm_acc_f64(g, Gdh, n, s));
        g.B = (const uint16_t*)dh;
        RQ_HIP(ctx, realq::gemm_acc_f64(g, Gdd, n, s));
        g.B = (const uint16_t*)dl;
        RQ_HIP(ctx, realq::gemm_acc_f64(g, Gdd, n, s));
    }
    return REALQ_OK;
}

extern "C++" {
int realq::validate_bgd(realq_ctx* ctx, const realq_bgd_params* p) {
    if (!p) return set_error(ctx, REALQ_ERR_INVALID_ARG, "NULL bgd params");
    if (p->steps < 0) return set_error(ctx, REALQ_ERR_INVALID_ARG, "bgd steps must be >= 0");
    if (!std::isfinite(p->lr) || p->lr < 0.f) return set_error(ctx, REALQ_ERR_INVALID_ARG, "lr must be finite, >= 0");
    if (!(p->beta1 >= 0.f && p->beta1 < 1.f) || !(p->beta2 >= 0.f && p->beta2 < 1.f))
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "Adam betas must lie in [0, 1)");
    if (!(p->eps > 0.f)) return set_error(ctx, REALQ_ERR_INVALID_ARG, "Adam eps must be > 0");
    if (p->tok_chunk < 0) return set_error(ctx, REALQ_ERR_INVALID_ARG, "tok_chunk must be >= 0");
    if (p->form != REALQ_BGD_TOKENS && p->form != REALQ_BGD_GRAM)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "form must be REALQ_BGD_TOKENS or REALQ_BGD_GRAM");
    if (!std::isfinite(p->loss_clip) || p->loss_clip < 0.f || p->loss_clip > 1.f)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "loss_clip must lie in [0, 1] (0 = off)");
    if (p->batch < 0) return set_error(ctx, REALQ_ERR_INVALID_ARG, "batch must be >= 0");
    if (p->resid_increment != 0 && p->resid_increment != 1)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "resid_increment must be 0 or 1");
    return REALQ_OK;
}
}  // extern "C++"

static int state_init_gram(realq_bgd_state* st);

// Whether steps after a block's first may take residual and gradient as increments
// (resid_increment in realq.h).  Adam's step is at most lr (1 - b1) / sqrt((1 - b2)(1 - b1^2/b2))
// for any gradient history (Cauchy-Schwarz on the two moment sums, bias corrections included), so
// the weight change over the steps - 1 later steps of a block is at most that times steps - 1;
// the increments are taken when this bound is within rms(W0) / 32, the module has at most
// kIncMaxColumns input columns (64 column blocks) and at least kIncTokensPerColumn tokens per
// input column.
static constexpr int64_t kIncMaxColumns = 8192;
static constexpr int64_t kIncTokensPerColumn = 16;
static int inc_init(realq_bgd_state* st) {
    realq_ctx* ctx = st->ctx;
    const realq_bgd_params& p = st->prm;
    st->inc = false;
    st->inc_c1 = -1;
    st->inc_ready = false;
    const double b1 = p.beta1, b2 = p.beta2;
    const int64_t m = st->m, n = st->n, T = st->T;
    if (!p.resid_increment || p.steps < 2 || p.loss_clip > 0.f || st->Tb != T || !(b1 * b1 < b2) ||
        n > kIncMaxColumns || T < kIncTokensPerColumn * n)
        return REALQ_OK;
    const double step_max = (1.0 - b1) / std::sqrt((1.0 - b2) * (1.0 - b1 * b1 / b2));
    const double disp = (double)(p.steps - 1) * step_max * (double)p.lr;
    void *parts, *ms;
    int rc;
    if ((rc = get_ws(ctx, "i_parts", (size_t)realq::dot_f32_partials() * 8, &parts))) return rc;
    if ((rc = get_ws(ctx, "i_ms", 8, &ms))) return rc;
    RQ_HIP(ctx, realq::dot_f32(st->W0, st->W0, m * n, 1.0, (double*)parts, ctx->stream));
    RQ_HIP(ctx, realq::reduce_partials((const double*)parts, realq::dot_f32_partials(), 1.0 / ((double)m * (double)n),
                                       (double*)ms, ctx->stream));
    double msq = 0.0;
    RQ_HIP(ctx, hipMemcpyAsync(&msq, ms, 8, hipMemcpyDeviceToHost, ctx->stream));
    RQ_HIP(ctx, hipStreamSynchronize(ctx->stream));
    if (!(disp <= std::sqrt(msq) / 32.0)) return REALQ_OK;
    void* q;
    if ((rc = state_alloc(st, &q, 8, "s_L0"))) return rc;
    st->L0 = (double*)q;
    if ((rc = state_alloc(st, &q, (size_t)m * n * 4, "s_Dacc"))) return rc;
    st->Dacc = (float*)q;
    if ((rc = state_alloc(st, &q, (size_t)m * n * 2, "s_Dinc"))) return rc;
    st->Dinc = (uint16_t*)q;
    if ((rc = state_alloc(st, &q, (size_t)m * n * 4, "s_G0"))) return rc;
    st->G0 = (float*)q;
    st->inc = true;
    return REALQ_OK;
}

static int state_init(realq_bgd_state* st) {
    if (st->prm.form == REALQ_BGD_GRAM) return state_init_gram(st);
    realq_ctx* ctx = st->ctx;
    const int64_t m = st->m, n = st->n, T = st->T;
    hipStream_t s = ctx->stream;
    st->gram = false;
    st->Tb = (st->prm.batch > 0 && st->prm.batch < T) ? st->prm.batch : T;
    st->nbatch = (T + st->Tb - 1) / st->Tb;
    int64_t Tc = st->prm.tok_chunk > 0 ? std::min<int64_t>(st->prm.tok_chunk, st->Tb) : st->Tb;
    st->Tc = Tc;
    int rc;
    void* p;
    if ((rc = state_alloc(st, &p, (size_t)m * T * 4, "s_B"))) return rc;
    st->B = (float*)p;
    if ((rc = state_alloc(st, &p, (size_t)m * n * 4, "s_m"))) return rc;
    st->mA = (float*)p;
    if ((rc = state_alloc(st, &p, (size_t)m * n * 4, "s_v"))) return rc;
    st->vA = (float*)p;
    if ((rc = state_alloc(st, &p, (size_t)m * n * 2, "s_Dh"))) return rc;
    st->Dhi = (uint16_t*)p;
    if ((rc = state_alloc(st, &p, (size_t)m * n * 2, "s_Dl"))) return rc;
    st->Dlo = (uint16_t*)p;
    if ((rc = state_alloc(st, &p, (size_t)n * T * 2, "s_XT"))) return rc;
    st->XhT = (uint16_t*)p;
    if (st->prm.loss_clip > 0.f) {
        // the clip writes split(R o s) as two arrays
        if ((rc = state_alloc(st, &p, (size_t)m * Tc * 2, "s_Rh"))) return rc;
        st->Rhi = (uint16_t*)p;
        if ((rc = state_alloc(st, &p, (size_t)m * Tc * 2, "s_Rl"))) return rc;
        st->Rlo = (uint16_t*)p;
    } else {
        // one array of 128-byte lines (32 tokens' hi, then their lo): whole-line stores
        if ((rc = state_alloc(st, &p, (size_t)m * r_ld(Tc) * 2, "s_Rh"))) return rc;
        st->Rhi = (uint16_t*)p;
        st->Rlo = nullptr;
    }
    if (st->prm.loss_clip > 0.f) {
        if ((rc = state_alloc(st, &p, (size_t)m * Tc * 4, "s_Rf"))) return rc;
        st->Rf = (float*)p;
        if ((rc = state_alloc(st, &p, (size_t)Tc * 4, "s_tau"))) return rc;
        st->tau = (float*)p;
    }

    Timed tm(ctx, "init");
    RQ_HIP(ctx, realq::fill_f32(st->mA, 0.f, m * n, s));
    RQ_HIP(ctx, realq::fill_f32(st->vA, 0.f, m * n, s));
    RQ_HIP(ctx, realq::transpose_u16(st->Xhat, n, st->XhT, T, T, n, s));
    // Residual base before any block is locked: B = W0 (Xhat - X)^T.
    if (st->X == st->Xhat) {
        RQ_HIP(ctx, realq::fill_f32(st->B, 0.f, m * T, s));
    } else {
        // W0 = W0hi + W0lo (in the D buffers for now), Xhat - X = Dxh + Dxl (bf16 pairs, exact
        // difference in float32 first): B = W0 Dxh^T (both halves of W0) + W0hi Dxl^T.
        RQ_HIP(ctx, realq::split_diff_f32(st->W0, n, nullptr, 0, st->Dhi, st->Dlo, n, m, n, s));
        const int64_t tcx = std::max<int64_t>(8, std::min<int64_t>(T, ((int64_t)(256ll << 20) / (2 * n) / 8) * 8));
        void *xh, *xl;
        if ((rc = get_ws(ctx, "i_xh", (size_t)tcx * n * 2, &xh))) return rc;
        if ((rc = get_ws(ctx, "i_xl", (size_t)tcx * n * 2, &xl))) return rc;
        for (int64_t t0 = 0; t0 < T; t0 += tcx) {
            const int64_t cur = std::min(tcx, T - t0);
            RQ_HIP(ctx, realq::split_diff_bf16(st->Xhat + t0 * n, st->X + t0 * n, (uint16_t*)xh, (uint16_t*)xl,
                                               cur * n, s));
            realq::GemmArgs g{st->Dhi, st->Dlo, n, (const uint16_t*)xh, n, m, cur, n, 1};
            RQ_HIP(ctx, realq::gemm_store_f32(g, st->B + t0, T, 0, 1.f, s));
            realq::GemmArgs g2{st->Dhi, nullptr, n, (const uint16_t*)xl, n, m, cur, n, 1};
            RQ_HIP(ctx, realq::gemm_acc_f32(g2, st->B + t0, T, 1.f, s));
        }
    }
    RQ_HIP(ctx, realq::fill_u16(st->Dhi, 0, m * n, s));
    RQ_HIP(ctx, realq::fill_u16(st->Dlo, 0, m * n, s));
    st->t = 0;
    st->locked = 0;
    return inc_init(st);
}

// Gram form: the three calibration Gram matrices once, then C0 = W0 G_dh and the constant
// c = <W0 G_dd, W0>; no residual base and no transposed activations are kept.
static int state_init_gram(realq_bgd_state* st) {
    realq_ctx* ctx = st->ctx;
    const int64_t m = st->m, n = st->n, T = st->T;
    hipStream_t s = ctx->stream;
    st->gram = true;
    st->Tc = T;
    st->Tb = T;
    st->nbatch = 1;
    int rc;
    void* p;
    if ((rc = state_alloc(st, &p, (size_t)m * n * 4, "s_m"))) return rc;
    st->mA = (float*)p;
    if ((rc = state_alloc(st, &p, (size_t)m * n * 4, "s_v"))) return rc;
    st->vA = (float*)p;
    if ((rc = state_alloc(st, &p, (size_t)m * n * 2, "s_Dh"))) return rc;
    st->Dhi = (uint16_t*)p;
    if ((rc = state_alloc(st, &p, (size_t)m * n * 2, "s_Dl"))) return rc;
    st->Dlo = (uint16_t*)p;
    if ((rc = state_alloc(st, &p, (size_t)n * n * 2, "s_Gh"))) return rc;
    st->Ghi = (uint16_t*)p;
    if ((rc = state_alloc(st, &p, (size_t)n * n * 2, "s_Gl"))) return rc;
    st->Glo = (uint16_t*)p;
    if ((rc = state_alloc(st, &p, (size_t)m * n * 4, "s_C0"))) return rc;
    st->C0 = (float*)p;
    if ((rc = state_alloc(st, &p, (size_t)m * n * 4, "s_P"))) return rc;
    st->Pm = (float*)p;
    if ((rc = state_alloc(st, &p, 8, "s_c"))) return rc;
    st->cconst = (double*)p;
    void *ghh, *gdh, *gdd, *A, *E, *parts;
    const int64_t np = realq::dot_f64_partials();
    if ((rc = get_ws(ctx, "i_Ghh", (size_t)n * n * 8, &ghh))) return rc;
    if ((rc = get_ws(ctx, "i_Gdh", (size_t)n * n * 8, &gdh))) return rc;
    if ((rc = get_ws(ctx, "i_Gdd", (size_t)n * n * 8, &gdd))) return rc;
    if ((rc = get_ws(ctx, "i_A", (size_t)m * n * 8, &A))) return rc;
    if ((rc = get_ws(ctx, "i_E", (size_t)m * n * 8, &E))) return rc;
    if ((rc = get_ws(ctx, "i_parts", (size_t)np * 8, &parts))) return rc;
    RQ_HIP(ctx, realq::fill_f64((double*)ghh, 0.0, n * n, s));
    if ((rc = realq_hessian_accum(ctx, st->Xhat, st->s, T, n, (double*)ghh))) return rc;
    if ((rc = gram_accum(ctx, st->Xhat, st->X, st->s, T, n, (double*)gdh, (double*)gdd))) return rc;
    Timed tm(ctx, "init");
    RQ_HIP(ctx, realq::fill_f32(st->mA, 0.f, m * n, s));
    RQ_HIP(ctx, realq::fill_f32(st->vA, 0.f, m * n, s));
    RQ_HIP(ctx, realq::fill_u16(st->Dhi, 0, m * n, s));
    RQ_HIP(ctx, realq::fill_u16(st->Dlo, 0, m * n, s));
    RQ_HIP(ctx, realq::split_f64((const double*)ghh, st->Ghi, st->Glo, n * n, s));
    double* Ad = (double*)A;
    double* Ed = (double*)E;
    RQ_HIP(ctx, realq::widen_f32(st->W0, Ad, m * n, s));
    RQ_HIP(ctx, realq::dgemm(Ad, n, (const double*)gdh, n, Ed, n, m, n, n, false, s));
    RQ_HIP(ctx, realq::narrow_f64(Ed, st->C0, m * n, s));
    RQ_HIP(ctx, realq::dgemm(Ad, n, (const double*)gdd, n, Ed, n, m, n, n, false, s));
    RQ_HIP(ctx, realq::dot_f64(Ed, Ad, m * n, (double*)parts, s));
    RQ_HIP(ctx, realq::reduce_partials((const double*)parts, np, 1.0, st->cconst, s));
    st->t = 0;
    st->locked = 0;
    return REALQ_OK;
}

// P = D G_hh on columns [p0, n) (three MFMA passes: D_hi G_hi + D_lo G_hi + D_hi G_lo).
static int gram_product(realq_ctx* ctx, realq_bgd_state* st, int64_t p0) {
    const int64_t m = st->m, n = st->n, pw = n - p0;
    if (pw <= 0) return REALQ_OK;
    Timed tm(ctx, "gram_step");
    realq::GemmArgs g{st->Dhi, st->Dlo, n, st->Ghi + p0 * n, n, m, pw, n, 1};
    RQ_HIP(ctx, realq::gemm_store_f32(g, st->Pm + p0, n, 0, 1.f, ctx->stream));
    realq::GemmArgs g2{st->Dhi, nullptr, n, st->Glo + p0 * n, n, m, pw, n, 1};
    RQ_HIP(ctx, realq::gemm_acc_f32(g2, st->Pm + p0, n, 1.f, ctx->stream));
    return REALQ_OK;
}

// L = (c + sum (2 C0 + P) (W - W0)) / 2T with P over all columns.
static int gram_loss(realq_ctx* ctx, realq_bgd_state* st, const double* W, double* loss_out) {
    const int64_t np = realq::dot_f64_partials();
    void* parts;
    int rc;
    if ((rc = get_ws(ctx, "b_gparts", (size_t)(np + 1) * 8, &parts))) return rc;
    RQ_HIP(ctx, realq::dot_gram(st->C0, st->Pm, W, st->W0, st->m * st->n, (double*)parts, ctx->stream));
    RQ_HIP(ctx, hipMemcpyAsync((double*)parts + np, st->cconst, 8, hipMemcpyDeviceToDevice, ctx->stream));
    RQ_HIP(ctx, realq::reduce_partials((const double*)parts, np + 1, 0.5 / (double)st->T, loss_out, ctx->stream));
    return REALQ_OK;
}

static int check_state_args(realq_ctx* ctx, const float* W0, const uint16_t* X, const uint16_t* Xhat, int64_t m,
                            int64_t n, int64_t T, const realq_bgd_params* params, const float* M, const float* P) {
    if (m <= 0 || n <= 0 || T <= 0) return set_error(ctx, REALQ_ERR_SHAPE, "bgd state: need m, n, T > 0");
    if (!W0 || !X || !Xhat) return set_error(ctx, REALQ_ERR_INVALID_ARG, "bgd state: NULL W0, X or Xhat");
    int rc = validate_bgd(ctx, params);
    if (rc) return rc;
    const bool clip = params->loss_clip > 0.f, minib = params->batch > 0 && params->batch < T;
    if (params->form == REALQ_BGD_GRAM && (clip || minib))
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "the Gram form takes neither loss_clip nor a batch smaller than T");
    if (clip && (M || P))
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "loss_clip needs the identity metric (no M, no window partner P)");
    return REALQ_OK;
}

int realq_bgd_state_create(realq_ctx* ctx, realq_bgd_state** out, const float* W0, const uint16_t* X,
                           const uint16_t* Xhat, const float* s, const float* M, const float* P, int64_t m, int64_t n,
                           int64_t T, const realq_bgd_params* params) {
    if (!ctx || !out) return REALQ_ERR_INVALID_ARG;
    *out = nullptr;
    int rc = check_state_args(ctx, W0, X, Xhat, m, n, T, params, M, P);
    if (rc) return rc;
    realq_bgd_state* st = new (std::nothrow) realq_bgd_state();
    if (!st) return set_error(ctx, REALQ_ERR_OOM, "host allocation");
    st->ctx = ctx;
    st->m = m;
    st->n = n;
    st->T = T;
    st->W0 = W0;
    st->X = X;
    st->Xhat = Xhat;
    st->s = s;
    st->M = M;
    st->P = P;
    st->prm = *params;
    st->owns = true;
    rc = state_init(st);
    if (rc) {
        state_free(st);
        delete st;
        return rc;
    }
    *out = st;
    return REALQ_OK;
}

void realq_bgd_state_destroy(realq_bgd_state* st) {
    if (!st) return;
    state_free(st);
    delete st;
}

// ============================================================================ a3-a6: one column block

extern "C++" {
int realq::validate_q(realq_ctx* ctx, const realq_qparams* qp) {
    if (!qp) return set_error(ctx, REALQ_ERR_INVALID_ARG, "NULL qparams");
    if (qp->bits < 2 || qp->bits > 4) return set_error(ctx, REALQ_ERR_INVALID_ARG, "bits must be 2, 3 or 4");
    if (qp->group < 0) return set_error(ctx, REALQ_ERR_INVALID_ARG, "group must be >= 1, or 0 for one group per row");
    if (qp->block < 1 || qp->block > 128) return set_error(ctx, REALQ_ERR_INVALID_ARG, "block must be in 1..128");
    if (qp->grid < 1 || qp->grid > 100) return set_error(ctx, REALQ_ERR_INVALID_ARG, "grid must be in 1..100");
    if (qp->group > 0 && qp->block % qp->group != 0 && qp->group % qp->block != 0)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "block and group must divide one another");
    if (qp->sym != 0 && qp->sym != 1) return set_error(ctx, REALQ_ERR_INVALID_ARG, "sym must be 0 or 1");
    if (!(qp->damp > 0.f) || !std::isfinite(qp->damp))
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "damp must be finite and > 0");
    return REALQ_OK;
}
}  // extern "C++"

// Rows [r0, r1) of one column block: search, quantize and compensate inside the block, then the
// trailing update; with a state, its copy of W - W0 follows on those rows.
static int quantize_rows(realq_ctx* ctx, double* W, int64_t m, int64_t n, int64_t r0, int64_t r1, int64_t c0,
                         int64_t bs, const float* U, const uint8_t* dead, const realq_qparams* qp, uint8_t* codes,
                         float* scales, uint8_t* zeros, realq_bgd_state* st) {
    int rc = validate_q(ctx, qp);
    if (rc) return rc;
    if (m <= 0 || n <= 0) return set_error(ctx, REALQ_ERR_SHAPE, "quantize_block: need m, n > 0");
    if (r0 < 0 || r1 <= r0 || r1 > m) return set_error(ctx, REALQ_ERR_SHAPE, "quantize_block: need 0 <= r0 < r1 <= m");
    if (c0 < 0 || bs < 1 || bs > 128 || c0 + bs > n)
        return set_error(ctx, REALQ_ERR_SHAPE, "quantize_block: need 0 <= c0, 1 <= bs <= 128, c0 + bs <= n");
    if (c0 % qp->block != 0 || (bs != qp->block && c0 + bs != n))
        return set_error(ctx, REALQ_ERR_SHAPE, "quantize_block: the block must be a whole column block of the sweep");
    if (!W || !U || !codes || !scales || !zeros)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "quantize_block: NULL W, U, codes, scales or zeros");
    if (st && (st->m != m || st->n != n))
        return set_error(ctx, REALQ_ERR_SHAPE, "quantize_block: state shape differs from W");
    if (st && st->locked != c0)
        return set_error(ctx, REALQ_ERR_SHAPE, "quantize_block: blocks must be quantized in column order");
    if (st) {  // the trailing update changes D: the next step starts a block
        st->inc_c1 = -1;
        st->inc_ready = false;
    }
    const int64_t mr = r1 - r0;
    const int64_t group = qp->group > 0 ? qp->group : n;  // 0: one group per row
    const int64_t ngroups = (n + group - 1) / group;
    void* E;
    if ((rc = get_ws(ctx, "q_E", (size_t)mr * bs * 8, &E))) return rc;
    hipStream_t s = ctx->stream;
    realq::QuantArgs q{};
    q.W = W + r0 * n;
    q.m = mr;
    q.n = n;
    q.c0 = c0;
    q.bs = bs;
    q.U = U;
    q.dead = dead;
    q.bits = qp->bits;
    q.group = (int)group;
    q.grid = qp->grid;
    q.sym = qp->sym;
    q.codes = codes + r0 * n;
    q.scales = scales + r0 * ngroups;
    q.zeros = zeros + r0 * ngroups;
    q.ngroups = ngroups;
    q.E = (double*)E;
    q.W0 = st ? st->W0 + r0 * n : nullptr;
    q.Dhi = st ? st->Dhi + r0 * n : nullptr;
    q.Dlo = st ? st->Dlo + r0 * n : nullptr;
    {
        Timed tm(ctx, "quantize");
        RQ_HIP(ctx, realq::quantize_block(q, s));
    }
    const int64_t c1 = c0 + bs;
    if (c1 < n) {
        realq::ObsArgs a{};
        a.E = (const double*)E;
        a.lde = bs;
        a.U = U + c0 * n + c1;
        a.ldu = n;
        a.W = W + r0 * n + c1;
        a.ldw = n;
        a.M = mr;
        a.N = n - c1;
        a.K = bs;
        if (st) {
            a.W0 = st->W0 + r0 * n + c1;
            a.ldw0 = n;
            a.Dhi = st->Dhi + r0 * n + c1;
            a.Dlo = st->Dlo + r0 * n + c1;
            a.ldd = n;
        }
        Timed tm(ctx, "obs");
        RQ_HIP(ctx, realq::obs_update(a, s));
    }
    return REALQ_OK;
}

// The block's quantized weights stay locked (Sec. 4.3): B += (W_hat - W0)[:, block] Xhat[:, block]^T
// (the Gram form keeps no residual base and only moves the boundary).
static int lock_block(realq_ctx* ctx, realq_bgd_state* st, int64_t c0, int64_t bs) {
    const int64_t n = st->n;
    if (c0 != st->locked || bs < 1 || c0 + bs > n)
        return set_error(ctx, REALQ_ERR_SHAPE, "bgd_lock_block: blocks must be locked in column order");
    st->inc_c1 = -1;  // the residual base moves: the next step starts a block
    st->inc_ready = false;
    if (!st->gram) {
        realq::GemmArgs g{st->Dhi + c0, st->Dlo + c0, n, st->Xhat + c0, n, st->m, st->T, bs, 1};
        Timed tm(ctx, "lock");
        RQ_HIP(ctx, realq::gemm_acc_f32(g, st->B, st->T, 1.f, ctx->stream));
    }
    st->locked = c0 + bs;
    return REALQ_OK;
}

int realq_quantize_block(realq_ctx* ctx, double* W, int64_t m, int64_t n, int64_t c0, int64_t bs, const float* U,
                         const uint8_t* dead, const realq_qparams* qp, uint8_t* codes, float* scales, uint8_t* zeros,
                         realq_bgd_state* st) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    int rc = quantize_rows(ctx, W, m, n, 0, m, c0, bs, U, dead, qp, codes, scales, zeros, st);
    if (rc) return rc;
    return st ? lock_block(ctx, st, c0, bs) : REALQ_OK;
}

int realq_quantize_block_rows(realq_ctx* ctx, double* W, int64_t m, int64_t n, int64_t r0, int64_t r1, int64_t c0,
                              int64_t bs, const float* U, const uint8_t* dead, const realq_qparams* qp,
                              uint8_t* codes, float* scales, uint8_t* zeros, realq_bgd_state* st) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    return quantize_rows(ctx, W, m, n, r0, r1, c0, bs, U, dead, qp, codes, scales, zeros, st);
}

int realq_bgd_lock_block(realq_ctx* ctx, realq_bgd_state* st, int64_t c0, int64_t bs) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (!st) return set_error(ctx, REALQ_ERR_INVALID_ARG, "bgd_lock_block: NULL state");
    return lock_block(ctx, st, c0, bs);
}

// ============================================================================ a7-a9: one BGD step

int realq_bgd_step(realq_ctx* ctx, realq_bgd_state* st, double* W, int64_t c1, float alpha, double* loss_out) {
    if (!ctx || !st) return REALQ_ERR_INVALID_ARG;
    if (!W) return set_error(ctx, REALQ_ERR_INVALID_ARG, "bgd_step: NULL W");
    if (c1 < 0 || c1 > st->n) return set_error(ctx, REALQ_ERR_SHAPE, "bgd_step: need 0 <= c1 <= n");
    if (!std::isfinite(alpha) || alpha < 0.f || alpha > 1.f)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "bgd_step: alpha must lie in [0, 1]");
    const int64_t m = st->m, n = st->n, T = st->T, Tc = st->Tc, nJ = n - c1;
    hipStream_t s = ctx->stream;
    if (nJ == 0) {
        if (loss_out) RQ_HIP(ctx, realq::fill_f64(loss_out, NAN, 1, s));
        return REALQ_OK;
    }
    const bool dense = st->M || (st->P && alpha < 1.f);
    const bool clip = st->prm.loss_clip > 0.f;
    int rc;
    void *Gp = nullptr, *Gacc = nullptr;
    int64_t splits_used = 1;
    // tokens of this step: mini-batch (t mod nbatch) of the module's Adam step t (1-based), cut
    // into chunks; the plan sizes the split-K and loss-partial workspaces for every chunk
    const realq::plan::StepPlan pl = realq::plan::plan_step(m, nJ, T, st->Tb, Tc, st->t, ctx->cus,
                                                            clip ? realq::clip_apply_partials() : 0);
    // increments (token form): a later step of the block takes the change of its residual as
    // Q = bf16(Dacc) Xhat_J^T, its gradient as G0 + bf16(Q o s) Xhat_J and its loss as
    // L0 + <G0, bf16(Dacc)> / T + sum s Q^2 / 2T; the block's first step writes L0 and G0 and
    // restarts Dacc
    // (a caller taking more than `steps` steps at one c1 gets a fresh first step every `steps`
    // steps, so the displacement bound of the gate holds)
    const bool inc_step = st->inc && !st->gram && st->inc_c1 == c1 && st->inc_ready &&
                          st->inc_taken < (int64_t)st->prm.steps - 1;
    const bool inc_first = st->inc && !st->gram && !inc_step;
    const int64_t Tn = pl.Tn;
    const int64_t nchunks = (int64_t)pl.chunks.size();
    if (st->gram) {
        // gradient (1/T) M_a (C0 + D G_hh)[:, J]; the loss needs D G_hh on every column
        const bool want_loss = loss_out && !dense;
        if ((rc = get_ws(ctx, "b_G", (size_t)m * nJ * 4, &Gacc))) return rc;
        if ((rc = gram_product(ctx, st, want_loss ? 0 : c1))) return rc;
        if (loss_out) {
            if (dense) RQ_HIP(ctx, realq::fill_f64(loss_out, NAN, 1, s));
            else if ((rc = gram_loss(ctx, st, W, loss_out))) return rc;
        }
        RQ_HIP(ctx, realq::gram_grad(st->C0, st->Pm, n, c1, m, nJ, (float*)Gacc, s));
    } else {
        void* parts;
        if ((rc = get_ws(ctx, "b_Gp", (size_t)pl.gp_slices * m * nJ * 4, &Gp))) return rc;
        if (nchunks > 1 || dense)
            if ((rc = get_ws(ctx, "b_G", (size_t)m * nJ * 4, &Gacc))) return rc;
        if ((rc = get_ws(ctx, "b_parts", (size_t)pl.parts_total * 8, &parts))) return rc;
        double* const pbase = (double*)parts;
        const bool via_acc = nchunks > 1 || dense;
        // a later step's gradient GEMM gives the change since the block's first: that one is
        // added back (in Adam, or as the start of the accumulated gradient)
        if (inc_step && via_acc)
            RQ_HIP(ctx, hipMemcpyAsync(Gacc, st->G0, (size_t)m * nJ * 4, hipMemcpyDeviceToDevice, s));

        for (int64_t ch = 0; ch < nchunks; ++ch) {
            const int64_t t0 = pl.chunks[ch].t0, cur = pl.chunks[ch].len;
            double* const pch = pbase + pl.chunks[ch].parts_off;
            realq::GemmArgs g{st->Dhi + c1, st->Dlo + c1, n, st->Xhat + t0 * n + c1, n, m, cur, nJ, 1};
            if (inc_step) {
                realq::GemmArgs gi{st->Dinc + c1, nullptr, n, st->Xhat + t0 * n + c1, n, m, cur, nJ, 1};
                Timed tm(ctx, "resid_inc");
                RQ_HIP(ctx, realq::gemm_resid_inc(gi, st->s ? st->s + t0 : nullptr, st->Rhi, q_ld(cur), pch, s));
            } else if (!clip) {
                Timed tm(ctx, "resid");
                RQ_HIP(ctx, realq::gemm_resid(g, st->B + t0, T, st->s ? st->s + t0 : nullptr, st->Rhi, nullptr,
                                              r_ld(cur), pch, s, true));
            } else {
                // residual kept whole, per-token thresholds over the m channels, then the
                // clipped, weighted split for the gradient GEMM and the loss partials
                Timed tm(ctx, "resid");
                RQ_HIP(ctx, realq::gemm_resid_f32(g, st->B + t0, T, st->Rf, cur, s));
                const int64_t k = std::max<int64_t>(1, (int64_t)std::ceil((double)st->prm.loss_clip * (double)m));
                RQ_HIP(ctx, realq::clip_select(st->Rf, cur, m, cur, std::min(k, m), st->tau, s));
                RQ_HIP(ctx, realq::clip_apply(st->Rf, cur, m, cur, st->tau, st->s ? st->s + t0 : nullptr, st->Rhi,
                                              st->Rlo, pch, s));
            }
            {
                realq::GemmArgs g{st->Rhi, clip ? st->Rlo : st->Rhi + 32, clip ? cur : r_ld(cur),
                                  st->XhT + c1 * T + t0, T, m, nJ, cur, pl.splits};
                g.a_blocked = clip ? 0 : 1;
                if (inc_step) {  // bf16(Q o s) alone, row-major
                    g.Alo = nullptr;
                    g.lda = q_ld(cur);
                    g.a_blocked = 0;
                }
                splits_used = realq::gemm_effective_splits(cur, pl.splits);
                Timed tm(ctx, inc_step ? "grad_inc" : "grad");
                RQ_HIP(ctx, realq::gemm_grad(g, (float*)Gp, nJ, m * nJ, s));
            }
            if (via_acc) {
                // Gacc (+)= sum of this chunk's split slices, chunks in order
                RQ_HIP(ctx, realq::reduce_splits((const float*)Gp, splits_used, m, nJ, 1.f, (float*)Gacc,
                                                 ch > 0 || inc_step, s));
            }
        }
        if (inc_first && via_acc)
            RQ_HIP(ctx, hipMemcpyAsync(st->G0, Gacc, (size_t)m * nJ * 4, hipMemcpyDeviceToDevice, s));
        // the identity-metric loss of the block's first step (its partials exist for any metric: a
        // caller may change alpha between the steps of one block)
        if (inc_first) RQ_HIP(ctx, realq::reduce_partials(pbase, pl.parts_total, 0.5 / (double)Tn, st->L0, s));
        if (loss_out) {
            if (dense) {
                RQ_HIP(ctx, realq::fill_f64(loss_out, NAN, 1, s));
            } else if (inc_step) {
                void* dots;
                if ((rc = get_ws(ctx, "b_incdots", (size_t)realq::inc_loss_partials() * 8, &dots))) return rc;
                RQ_HIP(ctx, realq::inc_loss(st->L0, st->G0, st->Dinc + c1, n, m, nJ, pbase, pl.parts_total,
                                            (double)Tn, (double*)dots, loss_out, s));
            } else {
                RQ_HIP(ctx, realq::reduce_partials(pbase, pl.parts_total, 0.5 / (double)Tn, loss_out, s));
            }
        }
    }
    st->t += 1;
    realq::AdamArgs a{};
    a.W = W;
    a.W0 = st->W0;
    a.mA = st->mA;
    a.vA = st->vA;
    a.Dhi = st->Dhi;
    a.Dlo = st->Dlo;
    a.m = m;
    a.n = n;
    a.c1 = c1;
    a.Gp = (const float*)Gp;
    a.splits = splits_used;
    a.gscale = (float)(1.0 / (double)Tn);
    a.lr = st->prm.lr;
    a.beta1 = st->prm.beta1;
    a.beta2 = st->prm.beta2;
    a.eps = st->prm.eps;
    a.bc1 = (float)(1.0 / (1.0 - std::pow((double)st->prm.beta1, (double)st->t)));
    a.bc2 = (float)(1.0 / (1.0 - std::pow((double)st->prm.beta2, (double)st->t)));
    if (st->inc && !st->gram) {
        a.Dacc = st->Dacc;
        a.Dinc = st->Dinc;
        a.inc_reset = inc_first ? 1 : 0;
        a.G0 = st->G0;
        a.g0_mode = (nchunks > 1 || dense) ? 0 : (inc_first ? 1 : 2);
        st->inc_c1 = c1;
        st->inc_ready = true;
        st->inc_taken = inc_first ? 0 : st->inc_taken + 1;
    }
    if (!dense && nchunks == 1 && !st->gram) {
        Timed tm(ctx, "adam");
        RQ_HIP(ctx, realq::adam_update(a, s));
    } else if (!dense) {
        a.Gp = (const float*)Gacc;
        a.splits = 1;
        Timed tm(ctx, "adam");
        RQ_HIP(ctx, realq::adam_update(a, s));
    } else {
        // G = (1/T) M_a Gacc with M_a = alpha M + (1 - alpha) P (M = I when absent; Eq. slide_window),
        // on the matrix cores: M_a as a bf16 pair formed once per alpha (one per column block),
        // Gacc transposed and split; hi*hi + lo*hi in one launch, hi*lo accumulated in a second
        // (the lo*lo term is below float32 rounding of the product).
        if (!st->Mah) {
            void* p;
            if ((rc = state_alloc(st, &p, (size_t)m * m * 2, "s_Mah"))) return rc;
            st->Mah = (uint16_t*)p;
            if ((rc = state_alloc(st, &p, (size_t)m * m * 2, "s_Mal"))) return rc;
            st->Mal = (uint16_t*)p;
            st->Ma_alpha = -1.f;
        }
        if (st->Ma_alpha != alpha) {
            RQ_HIP(ctx, realq::blend_split(st->M, alpha < 1.f ? st->P : nullptr, alpha, m, st->Mah, st->Mal, s));
            st->Ma_alpha = alpha;
        }
        void *Gm, *gth, *gtl;
        if ((rc = get_ws(ctx, "b_Gm", (size_t)m * nJ * 4, &Gm))) return rc;
        if ((rc = get_ws(ctx, "b_GTh", (size_t)m * nJ * 2, &gth))) return rc;
        if ((rc = get_ws(ctx, "b_GTl", (size_t)m * nJ * 2, &gtl))) return rc;
        const float invT = (float)(1.0 / (double)Tn);
        {
            Timed tm(ctx, "metric");
            RQ_HIP(ctx,
                   realq::transpose_split_f32((const float*)Gacc, nJ, (uint16_t*)gth, (uint16_t*)gtl, m, m, nJ, s));
            realq::GemmArgs g1{st->Mah, st->Mal, m, (const uint16_t*)gth, m, m, nJ, m, 1};
            RQ_HIP(ctx, realq::gemm_store_f32(g1, (float*)Gm, nJ, 0, invT, s));
            realq::GemmArgs g2{st->Mah, nullptr, m, (const uint16_t*)gtl, m, m, nJ, m, 1};
            RQ_HIP(ctx, realq::gemm_acc_f32(g2, (float*)Gm, nJ, invT, s));
        }
        Timed tm(ctx, "adam");
        RQ_HIP(ctx, realq::adam_update_dense(a, (const float*)Gm, s));
    }
    return REALQ_OK;
}

int realq_bgd_loss(realq_ctx* ctx, realq_bgd_state* st, const double* W, double* loss_out) {
    if (!ctx || !st) return REALQ_ERR_INVALID_ARG;
    if (!W || !loss_out) return set_error(ctx, REALQ_ERR_INVALID_ARG, "bgd_loss: NULL W or loss_out");
    if (st->M) return set_error(ctx, REALQ_ERR_SHAPE, "bgd_loss: only the identity metric is supported");
    if (st->gram) {
        int rc = gram_product(ctx, st, 0);
        if (rc) return rc;
        return gram_loss(ctx, st, W, loss_out);
    }
    // R = B + (W - W0)[:, J] Xhat[:, J]^T with J the columns not yet folded into B.
    const int64_t m = st->m, T = st->T, Tc = st->Tc, n = st->n, c1 = st->locked, nJ = n - c1;
    int64_t nparts = 0;
    const std::vector<realq::plan::Chunk> chunks = realq::plan::plan_loss(m, T, Tc, &nparts);
    void* parts;
    int rc;
    if ((rc = get_ws(ctx, "b_parts", (size_t)nparts * 8, &parts))) return rc;
    if (nJ > 0) RQ_HIP(ctx, realq::split_diff_f64(W + c1, n, st->W0 + c1, n, st->Dhi + c1, st->Dlo + c1, n, m, nJ,
                                                  ctx->stream));
    for (const auto& c : chunks) {
        realq::GemmArgs g{st->Dhi + c1, st->Dlo + c1, n, st->Xhat + c.t0 * n + c1, n, m, c.len, nJ, 1};
        RQ_HIP(ctx, realq::gemm_loss(g, st->B + c.t0, T, st->s ? st->s + c.t0 : nullptr, (double*)parts + c.parts_off,
                                     ctx->stream));
    }
    RQ_HIP(ctx, realq::reduce_partials((const double*)parts, nparts, 0.5 / (double)T, loss_out, ctx->stream));
    return REALQ_OK;
}

// ============================================================================ a10: window partner and hand-off

int realq_pullback_metric(realq_ctx* ctx, const float* W_next, const float* M_next, int64_t m_next, int64_t m,
                          int accumulate, float* P) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (m_next <= 0 || m <= 0) return set_error(ctx, REALQ_ERR_SHAPE, "pullback_metric: need m_next, m > 0");
    if (!W_next || !P) return set_error(ctx, REALQ_ERR_INVALID_ARG, "pullback_metric: NULL W_next or P");
    hipStream_t s = ctx->stream;
    void *WT, *T1 = nullptr;
    int rc;
    if ((rc = get_ws(ctx, "p_WT", (size_t)m * m_next * 4, &WT))) return rc;
    RQ_HIP(ctx, realq::transpose_f32(W_next, m, (float*)WT, m_next, m_next, m, s));  // WT = W_next^T [m, m_next]
    const float* right = W_next;
    if (M_next) {  // T1 = M_next W_next  [m_next, m]
        if ((rc = get_ws(ctx, "p_T1", (size_t)m_next * m * 4, &T1))) return rc;
        realq::SgemmArgs a{};
        a.A = M_next;
        a.lda = m_next;
        a.B = W_next;
        a.ldb = m;
        a.C = (float*)T1;
        a.ldc = m;
        a.M = m_next;
        a.N = m;
        a.K = m_next;
        a.alpha = 1.f;
        a.beta = 0.f;
        RQ_HIP(ctx, realq::sgemm(a, s));
        right = (const float*)T1;
    }
    realq::SgemmArgs a{};
    a.A = (const float*)WT;
    a.lda = m_next;
    a.B = right;
    a.ldb = m;
    a.C = P;
    a.ldc = m;
    a.M = m;
    a.N = m;
    a.K = m_next;
    a.alpha = 1.f;
    a.beta = accumulate ? 1.f : 0.f;
    RQ_HIP(ctx, realq::sgemm(a, s));
    return REALQ_OK;
}

int realq_handoff(realq_ctx* ctx, const float* Wa, const float* Wb, const uint16_t* X, int64_t T, int64_t n,
                  int64_t m, uint16_t* Y) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (T < 0 || n <= 0 || m <= 0) return set_error(ctx, REALQ_ERR_SHAPE, "handoff: need T >= 0, n, m > 0");
    if (T == 0) return REALQ_OK;
    if (!Wa || !X || !Y) return set_error(ctx, REALQ_ERR_INVALID_ARG, "handoff: NULL Wa, X or Y");
    hipStream_t s = ctx->stream;
    void *hi, *lo;
    int rc;
    if ((rc = get_ws(ctx, "h_wh", (size_t)m * n * 2, &hi))) return rc;
    if ((rc = get_ws(ctx, "h_wl", (size_t)m * n * 2, &lo))) return rc;
    // acc[i][t] = sum_j W[i][j] X[t][j], stored token-major
    realq::GemmArgs g{(const uint16_t*)hi, (const uint16_t*)lo, n, X, n, m, T, n, 1};
    if (!Wb) {
        RQ_HIP(ctx, realq::split_diff_f32(Wa, n, nullptr, 0, (uint16_t*)hi, (uint16_t*)lo, n, m, n, s));
        RQ_HIP(ctx, realq::gemm_store_bf16_t(g, Y, m, s));
        return REALQ_OK;
    }
    void* G;
    if ((rc = get_ws(ctx, "h_gate", (size_t)T * m * 4, &G))) return rc;
    RQ_HIP(ctx, realq::split_diff_f32(Wa, n, nullptr, 0, (uint16_t*)hi, (uint16_t*)lo, n, m, n, s));
    RQ_HIP(ctx, realq::gemm_store_f32_t(g, (float*)G, m, s));  // gate pre-activation, token-major
    RQ_HIP(ctx, realq::split_diff_f32(Wb, n, nullptr, 0, (uint16_t*)hi, (uint16_t*)lo, n, m, n, s));
    RQ_HIP(ctx, realq::gemm_swiglu_t(g, (const float*)G, m, Y, m, s));
    return REALQ_OK;
}

// ============================================================================ a11 with a dense metric
// L = (1/2T) sum_t s_t R_t^T M R_t with R = W0 Delta^T + D Xhat^T (Delta = Xhat - X, D = W - W0)
// expands through the calibration Gram matrices G_dd = Delta^T S Delta, G_dh = Delta^T S Xhat
// and G_hh = Xhat^T S Xhat (the Hessian accumulator) into
//   2T L = <W0 G_dd, M W0> + 2 <W0 G_dh, M D> + <D G_hh, M D>,
// n x n token contractions plus m x n x n and m x m x n float64 products instead of an
// m x m x T contraction.  Every term is built from the small quantities Delta and D.
static int dense_final_loss(realq_ctx* ctx, const realq_layer_desc* d, const double* W, const double* Ghh,
                            double* loss_dev) {
    const int64_t m = d->m, n = d->n, T = d->T;
    hipStream_t s = ctx->stream;
    int rc;
    void *gdh, *gdd, *A, *D, *E, *MX, *M64, *parts;
    if ((rc = get_ws(ctx, "g_dh", (size_t)n * n * 8, &gdh))) return rc;
    if ((rc = get_ws(ctx, "g_dd", (size_t)n * n * 8, &gdd))) return rc;
    if ((rc = gram_accum(ctx, d->Xhat, d->X, d->s, T, n, (double*)gdh, (double*)gdd))) return rc;
    Timed tm(ctx, "dense_loss");
    const int64_t np = realq::dot_f64_partials();
    if ((rc = get_ws(ctx, "g_A", (size_t)m * n * 8, &A))) return rc;
    if ((rc = get_ws(ctx, "g_D", (size_t)m * n * 8, &D))) return rc;
    if ((rc = get_ws(ctx, "g_E", (size_t)m * n * 8, &E))) return rc;
    if ((rc = get_ws(ctx, "g_MX", (size_t)m * n * 8, &MX))) return rc;
    if ((rc = get_ws(ctx, "g_M", (size_t)m * m * 8, &M64))) return rc;
    if ((rc = get_ws(ctx, "g_parts", (size_t)4 * np * 8, &parts))) return rc;
    double* Ad = (double*)A;
    double* Dd = (double*)D;
    double* Ed = (double*)E;
    double* MXd = (double*)MX;
    double* pp = (double*)parts;
    RQ_HIP(ctx, realq::widen_f32(d->W0, Ad, m * n, s));
    RQ_HIP(ctx, realq::sub_f64_f32(W, d->W0, Dd, m * n, s));
    RQ_HIP(ctx, realq::widen_f32(d->M, (double*)M64, m * m, s));
    // <W0 G_dd, M W0>
    RQ_HIP(ctx, realq::dgemm(Ad, n, (const double*)gdd, n, Ed, n, m, n, n, false, s));
    RQ_HIP(ctx, realq::dgemm((const double*)M64, m, Ad, n, MXd, n, m, n, m, false, s));
    RQ_HIP(ctx, realq::dot_f64(Ed, MXd, m * n, pp, s));
    // 2 <W0 G_dh, M D>
    RQ_HIP(ctx, realq::dgemm(Ad, n, (const double*)gdh, n, Ed, n, m, n, n, false, s));
    RQ_HIP(ctx, realq::dgemm((const double*)M64, m, Dd, n, MXd, n, m, n, m, false, s));
    RQ_HIP(ctx, realq::dot_f64(Ed, MXd, m * n, pp + np, s));
    RQ_HIP(ctx, realq::dot_f64(Ed, MXd, m * n, pp + 2 * np, s));
    // <D G_hh, M D>
    RQ_HIP(ctx, realq::dgemm(Dd, n, Ghh, n, Ed, n, m, n, n, false, s));
    RQ_HIP(ctx, realq::dot_f64(Ed, MXd, m * n, pp + 3 * np, s));
    RQ_HIP(ctx, realq::reduce_partials(pp, 4 * np, 0.5 / (double)T, loss_dev, s));
    return REALQ_OK;
}

// ============================================================================ a1-a11: whole module

int realq_quantize_layer(realq_ctx* ctx, const realq_layer_desc* d, realq_layer_out* out) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (!d || !out) return set_error(ctx, REALQ_ERR_INVALID_ARG, "quantize_layer: NULL desc or out");
    int rc = validate_q(ctx, &d->q);
    if (rc) return rc;
    if ((rc = check_state_args(ctx, d->W0, d->X, d->Xhat, d->m, d->n, d->T, &d->bgd, d->M, d->P))) return rc;
    if (!out->codes || !out->scales || !out->zeros || !out->W_hat)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "quantize_layer: NULL codes, scales, zeros or W_hat");
    const int64_t m = d->m, n = d->n, T = d->T;
    const bool grouped = d->s_groups != nullptr;
    if (!grouped && d->n_groups != 0)
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "quantize_layer: n_groups needs s_groups (0 without)");
    if (grouped && (d->n_groups < 1 || d->n_groups > m))
        return set_error(ctx, REALQ_ERR_INVALID_ARG, "quantize_layer: need 1 <= n_groups <= m");
    // row groups of rsz rows (one group of all m rows without s_groups); ngr of them hold rows
    const int64_t rsz = grouped ? (m + d->n_groups - 1) / d->n_groups : m;
    const int64_t ngr = (m + rsz - 1) / rsz;
    hipStream_t s = ctx->stream;
    realq::EventPair ev;
    RQ_HIP(ctx, ev.create());
    RQ_HIP(ctx, hipEventRecord(ev.a, s));

    // a1-a2: Hessian and inverse factor of every row group (each factorisation synchronises once)
    void *Hacc, *Uw = out->U, *deadw = out->dead;
    if ((rc = get_ws(ctx, "l_H", (size_t)n * n * 8, &Hacc))) return rc;
    if (!Uw && (rc = get_ws(ctx, "l_U", (size_t)ngr * n * n * 4, &Uw))) return rc;
    if (!deadw && (rc = get_ws(ctx, "l_dead", (size_t)ngr * n, &deadw))) return rc;
    for (int64_t g = 0; g < ngr; ++g) {
        RQ_HIP(ctx, realq::fill_f64((double*)Hacc, 0.0, n * n, s));
        const float* sg = grouped ? d->s_groups + g * T : d->s;
        if ((rc = realq_hessian_accum(ctx, d->Xhat, sg, T, n, (double*)Hacc))) return rc;
        if ((rc = realq_chol_inverse(ctx, (const double*)Hacc, n, T, d->q.damp, out->H ? out->H + g * n * n : nullptr,
                                     (float*)Uw + g * n * n, (uint8_t*)deadw + g * n)))
            return rc;
    }

    // state on context workspaces (reused across calls of the same size)
    realq_bgd_state st;
    st.ctx = ctx;
    st.m = m;
    st.n = n;
    st.T = T;
    st.W0 = d->W0;
    st.X = d->X;
    st.Xhat = d->Xhat;
    st.s = d->s;
    st.M = d->M;
    st.P = d->P;
    st.prm = d->bgd;
    st.owns = false;
    const bool bgd = d->bgd.steps > 0;
    if (bgd && (rc = state_init(&st))) return rc;

    // float64 working weights; W_hat receives their float32 rounding at the end
    void* Ww;
    if ((rc = get_ws(ctx, "l_W", (size_t)m * n * 8, &Ww))) return rc;
    double* W = (double*)Ww;
    RQ_HIP(ctx, realq::widen_f32(d->W0, W, m * n, s));
    const int64_t nb = (n + d->q.block - 1) / d->q.block;
    if (out->loss_trace && bgd) RQ_HIP(ctx, realq::fill_f64(out->loss_trace, NAN, nb * d->bgd.steps, s));
    for (int64_t b = 0; b < nb; ++b) {
        const int64_t c0 = b * d->q.block, bs = std::min<int64_t>(d->q.block, n - c0), c1 = c0 + bs;
        char rname[48];
        snprintf(rname, sizeof(rname), "block %lld (columns %lld..%lld)", (long long)b, (long long)c0,
                 (long long)(c1 - 1));
        realq::Range block_range(rname);
        for (int64_t g = 0; g < ngr; ++g) {
            if ((rc = quantize_rows(ctx, W, m, n, g * rsz, std::min(m, (g + 1) * rsz), c0, bs,
                                    (const float*)Uw + g * n * n, (const uint8_t*)deadw + g * n, &d->q, out->codes,
                                    out->scales, out->zeros, bgd ? &st : nullptr)))
                return rc;
        }
        if (bgd && (rc = lock_block(ctx, &st, c0, bs))) return rc;
        if (!bgd || c1 >= n) continue;
        float alpha = 1.f;
        if (d->window_total > 1) {
            const double bg = (double)(d->window_offset + b + 1);
            alpha = (float)(1.0 - (bg - 1.0) / (double)(d->window_total - 1));
            alpha = std::min(1.f, std::max(0.f, alpha));
        }
        for (int k = 0; k < d->bgd.steps; ++k) {
            double* lo = out->loss_trace ? out->loss_trace + b * d->bgd.steps + k : nullptr;
            if ((rc = realq_bgd_step(ctx, &st, W, c1, alpha, lo))) return rc;
        }
    }
    // a11: final loss (own metric) at the quantized weights
    out->loss_final = NAN;
    void* lf;
    if ((rc = get_ws(ctx, "l_loss", 8, &lf))) return rc;
    if (!d->M) {
        if (!bgd) {
            // no state yet: build the residual base once for the loss
            st.prm.tok_chunk = d->bgd.tok_chunk;
            if ((rc = state_init(&st))) return rc;
        }
        if ((rc = realq_bgd_loss(ctx, &st, W, (double*)lf))) return rc;
    } else {
        if (grouped) {  // the loss weighs tokens by s, not by a row group's saliency
            RQ_HIP(ctx, realq::fill_f64((double*)Hacc, 0.0, n * n, s));
            if ((rc = realq_hessian_accum(ctx, d->Xhat, d->s, T, n, (double*)Hacc))) return rc;
        }
        if ((rc = dense_final_loss(ctx, d, W, (const double*)Hacc, (double*)lf))) return rc;
    }
    RQ_HIP(ctx, realq::narrow_f64(W, out->W_hat, m * n, s));
    RQ_HIP(ctx, hipEventRecord(ev.b, s));
    RQ_HIP(ctx, hipMemcpyAsync(&out->loss_final, lf, 8, hipMemcpyDeviceToHost, s));
    RQ_HIP(ctx, hipStreamSynchronize(s));
    float ms = 0.f;
    RQ_HIP(ctx, hipEventElapsedTime(&ms, ev.a, ev.b));
    out->ms_total = ms;
    if ((rc = realq::harvest(ctx))) return rc;
    if (!std::isfinite(out->loss_final))
        return set_error(ctx, REALQ_ERR_NONFINITE,
                         "quantize_layer: the final loss is not finite (NaN or Inf in W0, X, s or the metric)");
    return REALQ_OK;
}

}  // extern "C"
