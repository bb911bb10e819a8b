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
//  5. The prefill launches refuse, before any device call, arguments their kernels do not handle:
//     fused epilogues with a split contraction, heads other than 64 / 128 columns, segments that are
//     not whole heads, rows not whole sequences, caches not in 32-key blocks, missing buffers; the
//     prefill attention with a tree mask or a head width it has no instance for.  Only invalid
//     argument sets are passed (a valid one would launch).
#include <algorithm>
#include <cstdio>
#include <vector>

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
                    if (q <= kAttnSplitRows) {
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
    // 5. launch-argument checks (each set below is invalid in exactly the way its label says)
    {
        int dummy[64];
        void* ptr = dummy;
        auto qkv = [&]() {
            PrefillGemmArgs p{};
            p.M = 140; p.N = 3 * 256; p.K = 256; p.A = ptr; p.lda = 256; p.W0 = p.W1 = p.W2 = ptr; p.n_per = 256;
            p.ksplit = 1; p.ep = PG_QKV; p.q = 70; p.H = 2; p.Dh = 128; p.S_max = 512;
            p.cache_len = dummy; p.rope = reinterpret_cast<const float*>(ptr); p.qbuf = reinterpret_cast<float*>(ptr);
            p.kc = p.vc = ptr; p.err = dummy;
            return p;
        };
        auto swiglu = [&]() {
            PrefillGemmArgs p{};
            p.M = 140; p.N = 2 * 688; p.K = 256; p.A = ptr; p.lda = 256; p.W0 = p.W1 = ptr; p.n_per = 688;
            p.ksplit = 1; p.ep = PG_SWIGLU; p.u = ptr; p.ldu = 688;
            return p;
        };
        struct Bad { const char* what; PrefillGemmArgs p; };
        std::vector<Bad> bad;
        { auto p = qkv(); p.ksplit = 2; bad.push_back({"QKV epilogue with a split contraction", p}); }
        { auto p = qkv(); p.Dh = 96; p.n_per = 192; p.N = 576; bad.push_back({"QKV heads of 96 columns", p}); }
        { auto p = qkv(); p.H = 3; bad.push_back({"QKV segment not whole heads", p}); }
        { auto p = qkv(); p.q = 69; bad.push_back({"QKV rows not whole sequences", p}); }
        { auto p = qkv(); p.S_max = 500; bad.push_back({"QKV cache not in 32-key blocks", p}); }
        { auto p = qkv(); p.qbuf = nullptr; bad.push_back({"QKV without a Q buffer", p}); }
        { auto p = qkv(); p.vc = nullptr; bad.push_back({"QKV without a V cache", p}); }
        { auto p = qkv(); p.N = 2 * 256; bad.push_back({"QKV with two segments", p}); }
        { auto p = qkv(); p.K = 252; bad.push_back({"contraction not in 8-element chunks", p}); }
        { auto p = qkv(); p.ep = 7; bad.push_back({"unknown epilogue", p}); }
        { auto p = swiglu(); p.u = nullptr; bad.push_back({"SwiGLU without an output", p}); }
        { auto p = swiglu(); p.ldu = 600; bad.push_back({"SwiGLU output rows too short", p}); }
        { auto p = swiglu(); p.ksplit = 2; bad.push_back({"SwiGLU epilogue with a split contraction", p}); }
        { auto p = swiglu(); p.N = 3 * 688; p.W2 = ptr; bad.push_back({"SwiGLU with three segments", p}); }
        { auto p = swiglu(); p.ep = PG_STORE; bad.push_back({"plain store without C", p}); }
        { auto p = swiglu(); p.ep = PG_STORE; p.C = reinterpret_cast<float*>(ptr); p.ldc = 100;
          bad.push_back({"plain store with C rows too short", p}); }
        { auto p = swiglu(); p.ep = PG_STORE; p.C = reinterpret_cast<float*>(ptr); p.ldc = p.N; p.ksplit = 5;
          p.c_part = (size_t)p.M * p.ldc; bad.push_back({"split into more parts than the partial buffers hold", p}); }
        { auto p = swiglu(); p.ep = PG_STORE; p.C = reinterpret_cast<float*>(ptr); p.ldc = p.N; p.ksplit = 4;
          p.c_part = (size_t)p.M * p.ldc - 1; bad.push_back({"split partials that overlap", p}); }
        for (const Bad& b : bad)
            for (int dtype : {0, 1})
                CHECK(launch_prefill_gemm(dtype, b.p, nullptr) == hipErrorInvalidValue, "prefill GEMM accepted: %s",
                      b.what);
        // split plans: O and down of a 511-row 7B block fill two workgroups per compute unit; a block of
        // 256 tiles or a short contraction stays whole; the partial buffers hold every plan
        struct Split { int M, N, K, parts; };
        for (const Split& t : {Split{511, 4096, 4096, 4}, Split{511, 4096, 11008, 4}, Split{140, 1024, 2752, 4},
                               Split{140, 1024, 1024, 2}, Split{200, 4096, 1024, 2}, Split{1024, 4096, 11008, 1},
                               Split{511, 4096, 1000, 1}, Split{2047, 5120, 13824, 1}, Split{140, 256, 688, 1}}) {
            const int k = prefill_gemm_ksplit(t.M, t.N, t.K);
            CHECK(k == t.parts && k >= 1 && k <= kPrefillMaxSplit, "prefill split of %d x %d x %d: %d parts, expected %d",
                  t.M, t.N, t.K, k, t.parts);
        }
        for (int parts : {0, kPrefillMaxSplit + 1})
            CHECK(launch_resid_norm_rows(1, reinterpret_cast<const float*>(ptr), parts, 0, 256, 4, 256,
                                         reinterpret_cast<float*>(ptr), 256, reinterpret_cast<const float*>(ptr), 1e-5f,
                                         ptr, 256, nullptr) == hipErrorInvalidValue,
                  "residual row kernel accepted %d parts", parts);
        auto rows = [&]() {
            AttnArgs a{};
            a.qbuf = reinterpret_cast<const float*>(ptr); a.kc = a.vc = ptr; a.cache_len = dummy;
            a.B = 2; a.q = 70; a.H = 2; a.S_max = 512; a.scale = 0.1f; a.out = ptr; a.ldo = 256; a.err = dummy;
            return a;
        };
        struct BadA { const char* what; AttnArgs a; int head_dim; };
        std::vector<BadA> bada;
        { auto a = rows(); a.mask = reinterpret_cast<const uint64_t*>(ptr); bada.push_back({"prefill attention with a tree mask", a, 128}); }
        { auto a = rows(); bada.push_back({"prefill attention, heads of 96 columns", a, 96}); }
        {
            auto a = rows();
            CHECK(launch_attention_rows(0, 128, a, nullptr) == hipErrorInvalidValue && !attention_rows_supported(0, 128),
                  "prefill attention accepted float heads of 128 columns");
        }
        { auto a = rows(); a.S_max = 500; bada.push_back({"prefill attention, cache not in 32-key blocks", a, 128}); }
        { auto a = rows(); a.q = 0; bada.push_back({"prefill attention without rows", a, 128}); }
        { auto a = rows(); a.ldo = 258; bada.push_back({"prefill attention, output stride not in 4s", a, 128}); }
        { auto a = rows(); a.out = nullptr; bada.push_back({"prefill attention without an output", a, 128}); }
        for (const BadA& b : bada)
            for (int dtype : {0, 1})
                CHECK(launch_attention_rows(dtype, b.head_dim, b.a, nullptr) == hipErrorInvalidValue,
                      "prefill attention accepted: %s", b.what);
    }
    std::printf("%s (%d failed)\n", failures ? "FAILED" : "ok", failures);
    return failures ? 1 : 0;
}
