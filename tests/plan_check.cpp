// Host-side checks of the launch plans the library sizes its workspace by and that block-size
// invariance rests on.  Built by tests/test_plans_cpu.py with the host compiler against
// libsdsat.so (the plan functions are host code; no device is touched).  Prints one line per
// failed check and exits non-zero if any failed.
//  1. Attention: the split-partial buffer sized at init (attention_partial_floats for max_batch,
//     max_block, the cache capacity) holds the partials of every plan a forward block can make:
//     any batch <= max_batch, block rows <= max_block, cache length + rows <= capacity.
//  2. Attention: the key partition (32-key blocks per split) and the waves per workgroup depend on
//     the batch and the capacity only, never on the block rows or the cache length, for blocks of
//     one 16-row tile (the decode blocks whose rows must match single-token steps bit for bit).
//  3. Residual GEMMs: the partial-tile buffer (gemm_resid_part_bytes) holds every split plan of
//     up to 64 rows.
//  4. Skinny GEMMs: the contraction slices (waves x workgroups per tile) do not depend on the rows
//     M, for M = 1..64, so a row's value is the same in any block.
#include <algorithm>
#include <cstdio>

#include "kernels.h"

using namespace sdsat;

static int failures = 0;
#define CHECK(cond, ...)                      \
    do {                                      \
        if (!(cond)) {                        \
            std::printf("FAIL: " __VA_ARGS__); \
            std::printf("\n");                \
            ++failures;                       \
        }                                     \
    } while (0)

int main() {
    struct Cfg { int maxB, H, Dh, maxQ, max_ctx; };
    const Cfg cfgs[] = {
        {1, 32, 128, 512, 812},    // 7B bench: batch 1, k = 5, prompt 512, 256 new tokens
        {1, 40, 128, 1024, 2614},  // 13B: k = 10, prompt 2048, 512 new tokens
        {4, 32, 128, 1024, 1324},  // 7B batch 4: prompts 4 x 1024
        {8, 32, 128, 11, 16427},   // micro-benchmark: 16384 keys, q 6 and 11
        {1, 2, 128, 64, 370}, {1, 2, 128, 16, 100}, {3, 2, 128, 6, 86}, {2, 4, 64, 17, 2000},
        {1, 4, 64, 64, 1200}, {2, 4, 128, 16, 1800}, {8, 2, 128, 70, 200},
    };
    for (const Cfg& c : cfgs) {
        const int S = (c.max_ctx + 31) / 32 * 32;
        const size_t have = attention_partial_floats(c.maxB, c.H, c.maxQ, c.Dh, S);
        for (int B = 1; B <= c.maxB; ++B) {
            const AttnPlan ref = plan_attention(B, c.H, 1, c.Dh, 0, S);
            for (int q = 1; q <= c.maxQ; q += (q < 20 ? 1 : 37)) {
                for (int len = 0; len + q <= S; len += 1 + len / 5) {
                    const AttnPlan p = plan_attention(B, c.H, q, c.Dh, len, S);
                    CHECK(attention_plan_partial_floats(p, B, c.H, c.Dh) <= have,
                          "attention partials: B %d H %d q %d len %d S %d need %zu have %zu", B, c.H, q, len, S,
                          attention_plan_partial_floats(p, B, c.H, c.Dh), have);
                    CHECK(p.grid == B * c.H * p.row_tiles * p.splits * p.cols && p.splits >= 1 && p.waves >= 1 &&
                              p.per_split >= 1 && (long)p.splits * p.per_split * 32 >= std::min(S, len + q),
                          "attention plan shape: B %d q %d len %d", B, q, len);
                    if (q <= 16) {
                        CHECK(p.per_split == ref.per_split && p.waves == ref.waves,
                              "key partition varies with the block: B %d q %d len %d (%d/%d waves %d/%d)", B, q, len,
                              p.per_split, ref.per_split, p.waves, ref.waves);
                    }
                }
            }
        }
    }
    // residual and skinny GEMM plans at the model shapes (d, F) and small test shapes
    const int shapes[][2] = {{4096, 11008}, {5120, 13824}, {256, 688}, {512, 1376}, {1024, 2752}};
    for (const auto& sh : shapes) {
        const int d = sh[0], F = sh[1];
        const int ks_d = (d + 31) / 32, ks_f = (F + 31) / 32;
        struct G { int n_tiles, k_steps; bool resid; } gs[] = {
            {3 * d / 16, ks_d, false}, {d / 16, ks_d, true}, {(2 * F + 15) / 16, ks_d, false},
            {d / 16, ks_f, true}, {(32016 + 15) / 16, ks_d, false}};
        for (const G& g : gs) {
            const size_t part = g.resid ? gemm_resid_part_bytes(g.n_tiles, g.k_steps, 64) : 0;
            const GemmPlan p1 = g.resid ? plan_gemm_resid(1, g.n_tiles, g.k_steps) : plan_gemm(1, g.n_tiles, g.k_steps);
            for (int M = 1; M <= 64; ++M) {
                const GemmPlan p = g.resid ? plan_gemm_resid(M, g.n_tiles, g.k_steps) : plan_gemm(M, g.n_tiles, g.k_steps);
                CHECK(p.waves * p.ksplit == p1.waves * p1.ksplit,
                      "contraction slices vary with M: d %d tiles %d steps %d M %d (%d x %d vs %d x %d)", d, g.n_tiles,
                      g.k_steps, M, p.waves, p.ksplit, p1.waves, p1.ksplit);
                CHECK(p.mt == (M + 15) / 16 && p.grid * p.ntw >= g.n_tiles * (p.ksplit > 1 ? p.ksplit : 1) / p.ksplit,
                      "GEMM plan shape: tiles %d M %d", g.n_tiles, M);
                if (g.resid && p.ksplit > 1)
                    CHECK((size_t)g.n_tiles * p.waves * p.ksplit * p.mt * 64 * 16 <= part,
                          "residual partials: tiles %d steps %d M %d need %zu have %zu", g.n_tiles, g.k_steps, M,
                          (size_t)g.n_tiles * p.waves * p.ksplit * p.mt * 64 * 16, part);
            }
        }
    }
    std::printf("%s (%d failed)\n", failures ? "FAILED" : "ok", failures);
    return failures ? 1 : 0;
}
