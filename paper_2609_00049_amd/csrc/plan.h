// Host-side launch planning of the layer sweep: GEMM tile choice, split-K factors and the
// layout of the per-chunk workspaces of one Block-GD step.  Pure C++ (no HIP types), so the
// CPU test suite compiles this unit on its own with AddressSanitizer and checks the sizing
// arithmetic against the launches it describes.
#pragma once
#include <stdint.h>

#include <vector>

namespace realq {
namespace plan {

// Tile shapes of the bf16 MFMA GEMM (the kernel asserts that its configurations match).
constexpr int64_t kBK = 32;                          // K slice
constexpr int64_t kLargeBM = 256, kLargeBN = 256;    // 8 waves
constexpr int64_t kSmallBM = 128, kSmallBN = 128;    // 4 waves
constexpr int64_t kLargeMinTiles = 256;              // the large tile once a launch has this many

int64_t tiles(int64_t M, int64_t N, bool large);
// tile: 0 = chosen from the shape, 1 = large, 2 = small
bool pick_large(int64_t M, int64_t N, int tile);
int64_t num_blocks(int64_t M, int64_t N, int tile);
// K range per split (a multiple of kBK) and the number of non-empty splits it gives.
int64_t k_per_split(int64_t K, int64_t splits);
int64_t effective_splits(int64_t K, int64_t splits);
// Split-K factor of the gradient GEMM (always the large tile): the smallest factor up to 16
// whose launch fills at least 97% of its last round of `cus` blocks, else the fullest one;
// every split keeps at least 256 tokens.
int64_t choose_splits(int64_t M, int64_t N, int64_t K, int cus);

// One token chunk of a Block-GD step: tokens [t0, t0 + len) of the calibration set, and the
// range [parts_off, parts_off + parts) of the loss-partial workspace its residual launch (or,
// with the clip, its clip launch) writes.
struct Chunk {
    int64_t t0, len, parts_off, parts;
};

struct StepPlan {
    int64_t bt0 = 0, Tn = 0;   // tokens of the step: [bt0, bt0 + Tn)
    int64_t splits = 1;        // split factor passed to every chunk's gradient GEMM
    int64_t gp_slices = 1;     // gradient slices the split-K workspace must hold (max over chunks)
    int64_t parts_total = 0;   // loss partials over all chunks
    std::vector<Chunk> chunks;
};

// Step t (0-based count of earlier Adam steps of the module) of a Block-GD sweep over m rows,
// nJ trailing columns and T tokens, with batches of Tb tokens (Tb = T: full batch) cut into
// chunks of Tc tokens.  clip_parts > 0: each chunk writes that many partials (the clip
// launch) instead of one per residual block.
StepPlan plan_step(int64_t m, int64_t nJ, int64_t T, int64_t Tb, int64_t Tc, int64_t t, int cus,
                   int64_t clip_parts);
// Chunks of a residual-loss pass over all T tokens (one partial per residual block).
std::vector<Chunk> plan_loss(int64_t m, int64_t T, int64_t Tc, int64_t* parts_total);

}  // namespace plan
}  // namespace realq
