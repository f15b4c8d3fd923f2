// CPU test of the sweep's launch planning (paper_2609_00049_amd/csrc/plan.cpp), built with
// AddressSanitizer and UndefinedBehaviorSanitizer by tests/test_host_plan.py.  It checks that the
// split-K and loss-partial workspaces a Block-GD step allocates hold everything its launches write,
// for every chunk of every step, including a short last mini-batch and a short last token chunk.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "plan.h"

using namespace realq::plan;

static int failures = 0;
#define CHECK(cond)                                                              \
    do {                                                                         \
        if (!(cond)) {                                                           \
            std::fprintf(stderr, "%s:%d: CHECK failed: %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                          \
        }                                                                        \
    } while (0)

// Replays the writes of one planned step into buffers of exactly the planned sizes (the
// sanitizer traps any write past them): each chunk's residual launch writes one partial per block
// of its own tile choice, each gradient launch writes effective_splits(len, splits) slices.
static void replay(const StepPlan& p, int64_t m, int64_t nJ, int64_t clip_parts) {
    std::vector<double> parts((size_t)p.parts_total);
    std::vector<char> written((size_t)p.parts_total, 0);
    const int64_t slice = m * nJ;
    std::vector<float> gp((size_t)(p.gp_slices * slice));
    int64_t covered = 0;
    for (const Chunk& c : p.chunks) {
        CHECK(c.len >= 1);
        CHECK(c.t0 == p.bt0 + covered);
        covered += c.len;
        const int64_t nblk = clip_parts > 0 ? clip_parts : num_blocks(m, c.len, 0);
        CHECK(nblk == c.parts);
        for (int64_t b = 0; b < nblk; ++b) {
            parts.at((size_t)(c.parts_off + b)) = 1.0;  // at() also checks the index
            CHECK(!written[(size_t)(c.parts_off + b)]);
            written[(size_t)(c.parts_off + b)] = 1;
        }
        const int64_t z = effective_splits(c.len, p.splits);
        CHECK(z <= p.gp_slices);
        CHECK(k_per_split(c.len, p.splits) * z >= c.len);
        for (int64_t s = 0; s < z; ++s) gp[(size_t)(s * slice + slice - 1)] = 1.f;
    }
    CHECK(covered == p.Tn);
    for (char w : written) CHECK(w);  // the reduction reads every partial: each one is written
}

int main() {
    // A 512x512 layer with 8192 tokens in batches of 4160: the second batch is 4032 tokens; with
    // the full-batch split factor passed unchanged it would round to one more slice than the
    // workspace holds.
    {
        const int64_t m = 512, nJ = 384, T = 8192, Tb = 4160;
        CHECK(choose_splits(m, nJ, Tb, 256) == 16);
        CHECK(effective_splits(4160, 16) == 15 && effective_splits(4032, 16) == 16);  // the overflow
        for (int64_t t = 0; t < 4; ++t) {
            StepPlan p = plan_step(m, nJ, T, Tb, Tb, t, 256, 0);
            CHECK(p.Tn == (t % 2 == 0 ? 4160 : 4032));
            CHECK(p.splits == 15 && p.gp_slices <= p.splits);
            replay(p, m, nJ, 0);
        }
    }
    // 14336 rows, 3072 tokens in chunks of 2048: the last 1024-token chunk has fewer than 256
    // large tiles and switches to the small tile, which writes four times as many partials.
    {
        StepPlan p = plan_step(14336, 1024, 3072, 3072, 2048, 0, 256, 0);
        CHECK(p.chunks.size() == 2);
        CHECK(p.chunks[0].parts == 56 * 8);
        CHECK(p.chunks[1].parts == 112 * 8);
        CHECK(p.parts_total == 56 * 8 + 112 * 8);
        replay(p, 14336, 1024, 0);
        int64_t tot = 0;
        std::vector<Chunk> l = plan_loss(14336, 3072, 2048, &tot);
        CHECK(l.size() == 2 && tot == 56 * 8 + 112 * 8 && l[1].parts_off == 56 * 8);
    }
    // the clip writes a fixed number of partials per chunk
    {
        StepPlan p = plan_step(300, 200, 5000, 2000, 700, 2, 256, 512);
        CHECK(p.Tn == 1000);
        CHECK(p.parts_total == 2 * 512);
        replay(p, 300, 200, 512);
    }
    // the split factor of a full chunk never grows on a shorter one
    for (int64_t K = 1; K <= 9000; K += 7)
        for (int64_t s = 1; s <= 16; ++s) {
            const int64_t se = effective_splits(K, s);
            for (int64_t k2 = 1; k2 <= K; k2 += 97) CHECK(effective_splits(k2, se) <= se);
        }
    // randomised shapes, batches, chunks and CU counts
    std::mt19937_64 rng(1234);
    auto pick = [&](int64_t lo, int64_t hi) { return lo + (int64_t)(rng() % (uint64_t)(hi - lo + 1)); };
    for (int it = 0; it < 3000; ++it) {
        const int64_t m = pick(1, 3000), nJ = pick(1, 600), T = pick(1, 20000);
        const int64_t Tb = pick(0, 1) ? T : pick(1, T);
        const int64_t Tc = pick(0, 2) == 0 ? Tb : pick(1, Tb);
        const int64_t t = pick(0, 40);
        const int cus = (int)pick(1, 304);
        const int64_t clip = pick(0, 3) == 0 ? 512 : 0;
        StepPlan p = plan_step(m, nJ, T, Tb, Tc, t, cus, clip);
        CHECK(p.Tn >= 1 && p.bt0 + p.Tn <= T);
        CHECK(p.splits >= 1 && p.splits <= 16);
        replay(p, m, nJ, clip);
    }
    if (failures) {
        std::fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    std::printf("plan: all checks passed\n");
    return 0;
}
