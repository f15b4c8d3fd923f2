// Host-side launch planning of the layer sweep (see plan.h).
#include "plan.h"

#include <algorithm>

namespace realq {
namespace plan {

int64_t tiles(int64_t M, int64_t N, bool large) {
    const int64_t bm = large ? kLargeBM : kSmallBM, bn = large ? kLargeBN : kSmallBN;
    return ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
}

bool pick_large(int64_t M, int64_t N, int tile) {
    return tile == 1 || (tile == 0 && tiles(M, N, true) >= kLargeMinTiles);
}

int64_t num_blocks(int64_t M, int64_t N, int tile) { return tiles(M, N, pick_large(M, N, tile)); }

int64_t k_per_split(int64_t K, int64_t splits) {
    if (splits < 1) splits = 1;
    int64_t kps = (K + splits - 1) / splits;
    kps = ((kps + kBK - 1) / kBK) * kBK;
    return kps <= 0 ? kBK : kps;
}

int64_t effective_splits(int64_t K, int64_t splits) {
    const int64_t kps = k_per_split(K, splits);
    const int64_t s = (K + kps - 1) / kps;
    return s < 1 ? 1 : s;
}

int64_t choose_splits(int64_t M, int64_t N, int64_t K, int cus) {
    if (cus < 1) cus = 1;
    const int64_t blocks = tiles(M, N, true);
    int64_t smax = std::min<int64_t>(16, K / 256);
    if (smax < 1) smax = 1;
    int64_t best = 1;
    double best_fill = -1.0;
    for (int64_t q = 1; q <= smax; ++q) {
        const int64_t bq = blocks * q;
        const int64_t rounds = (bq + cus - 1) / cus;
        const double fill = (double)bq / (double)(rounds * cus);
        if (fill >= 0.97) return q;
        if (fill > best_fill + 1e-9) {
            best_fill = fill;
            best = q;
        }
    }
    return best;
}

StepPlan plan_step(int64_t m, int64_t nJ, int64_t T, int64_t Tb, int64_t Tc, int64_t t, int cus,
                   int64_t clip_parts) {
    StepPlan p;
    if (Tb < 1 || Tb > T) Tb = T;
    if (Tc < 1 || Tc > Tb) Tc = Tb;
    const int64_t nbatch = (T + Tb - 1) / Tb;
    p.bt0 = (t % nbatch) * Tb;
    p.Tn = std::min(Tb, T - p.bt0);
    // The split factor is fixed from the full chunk length; a shorter chunk re-rounds its K
    // range and can come out with more splits for the same factor, so every chunk is given the
    // effective factor of a full chunk instead: effective_splits(len, S_eff) <= S_eff.
    const int64_t S = choose_splits(m, nJ, Tc, cus);
    p.splits = effective_splits(Tc, S);
    p.gp_slices = 1;
    for (int64_t t0 = p.bt0; t0 < p.bt0 + p.Tn; t0 += Tc) {
        Chunk c;
        c.t0 = t0;
        c.len = std::min(Tc, p.bt0 + p.Tn - t0);
        c.parts_off = p.parts_total;
        // the residual launch picks its tile from (m, len), so a short chunk may switch tiles
        c.parts = clip_parts > 0 ? clip_parts : num_blocks(m, c.len, 0);
        p.parts_total += c.parts;
        p.gp_slices = std::max(p.gp_slices, effective_splits(c.len, p.splits));
        p.chunks.push_back(c);
    }
    return p;
}

std::vector<Chunk> plan_loss(int64_t m, int64_t T, int64_t Tc, int64_t* parts_total) {
    std::vector<Chunk> out;
    if (Tc < 1 || Tc > T) Tc = T;
    int64_t total = 0;
    for (int64_t t0 = 0; t0 < T; t0 += Tc) {
        Chunk c;
        c.t0 = t0;
        c.len = std::min(Tc, T - t0);
        c.parts_off = total;
        c.parts = num_blocks(m, c.len, 0);
        total += c.parts;
        out.push_back(c);
    }
    if (parts_total) *parts_total = total;
    return out;
}

}  // namespace plan
}  // namespace realq
