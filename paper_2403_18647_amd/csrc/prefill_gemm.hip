// Matrix-core GEMM for blocks of many rows (the prompt prefill before the
// draft/verify loop, Section 2.1): C[M, N] = A[M, K] . W[N, K]^T with A the
// normalised activations (element type, rows padded with zeros), W the
// caller's row-major [out, in] weights -- up to three matrices stacked along
// N (Q | K | V, gate | up) -- and C float.  At hundreds of rows a weight byte
// feeds hundreds of flops, so unlike the decode GEMM this kernel is bound by
// the matrix cores and by how often operands are re-read, not by HBM.
//
// Tiling: a workgroup of WM x WN waves computes a BM x BN tile of C, each wave
// a (16 TM) x (16 TN) sub-tile of matrix-core 16x16 tiles (bf16: 8 waves of
// 32 x 64 in a 128 x 128 tile).  The contraction runs in stages of BK columns
// (bf16: 64, two matrix-core steps); both operands' stage tiles are staged in
// LDS (double-buffered), with the global loads of the next two stages in
// flight in registers while the current stage's fragments are read from LDS
// and multiplied; one barrier per stage.  LDS rows are padded by 32 bytes: a
// 64-lane 16-byte fragment read then takes the LDS's 4 cycles with no bank
// conflict (measured on MI355X with rocprofv3's SQ_LDS_BANK_CONFLICT: rows of
// 80 or 144 bytes conflict two-way, rows of 160 bytes or 128 bytes with the
// 16-byte chunks permuted by row do not).  Every
// element of C is accumulated by one wave in one fixed order of k, so results
// repeat bit for bit.
// Workgroups that share a weight tile (the same N tile, different M tiles) are
// placed on the same XCD (workgroups go to the 8 XCDs round-robin), so the
// weights come from HBM once and the other row tiles read them from that L2.
// Epilogues: C as float (O, down, LM head), or, from the C tile read back
// through LDS, RoPE with Q to its float buffer and K / V into the cache (QKV),
// or silu(gate) * up in the element type (gate | up, whose workgroup tiles
// pair 64 gate rows with the same 64 up rows) -- no float C round trip and no
// separate row kernel for these two.
#include "device.h"
#include "kernels.h"

namespace sdsat {

namespace {

// Stage geometry: BK contraction elements per LDS stage.  Measured on MI355X, 7B 511-row prefill
// (whole prefill, bf16, 16-byte row padding): 8 waves of 32 x 64, BK 64, two register stages in
// flight: 14.0 ms (13.2 ms with the 32-byte padding used now); the same with BK 32: 17.4 ms, with
// BK 128 (one workgroup per compute unit): 15.6 ms; 8 waves of 64 x 32: 14.1 ms; 4 waves of 64 x 64,
// BK 32: 17.3 ms, BK 64: 18.8 ms; 16 waves of 32 x 32, BK 64: 14.7 ms; one register stage instead of
// two: 14.9 ms.  Three register stages (at the register budget of two workgroups per compute unit,
// with a small spill) measured slower than two: 13.6 against 12.8 ms in one run.  With the fused
// epilogues and the four-part O / down split: 8 waves of 32 x 64 11.2-11.6 ms; 8 waves of 64 x 64 in
// 256 x 128 tiles 12.4-12.5 ms; 4 waves of 64 x 64 12.4 ms.
template <typename T, int BK_> struct PTile {
    static constexpr int BK = BK_;
    static constexpr int EPC = 16 / sizeof(T);          // elements per 16-byte chunk
    static constexpr int LDR = BK + 32 / sizeof(T);     // LDS row stride in elements (32 bytes of padding)
};

// Global -> registers: this thread's chunks of the A and W step tiles.  The loads are unconditional
// (indices clamped into the operands, the chunks past M, N or K zeroed when they are written to LDS), so
// the loop has no divergent branches and the waits for a register set count only the loads before it.
template <typename T, int BM, int BN, int NT, int BK, int EP>
struct StepLoad {
    static constexpr int EPC = PTile<T, BK>::EPC;
    static constexpr int CPR = PTile<T, BK>::BK / EPC;        // chunks per row of a stage tile
    static constexpr int NA = (BM * CPR + NT - 1) / NT, NW = (BN * CPR + NT - 1) / NT;
    static_assert(NA * NT == BM * CPR || NA == 1, "whole chunks per thread");
    static_assert(NW * NT == BN * CPR || NW == 1, "whole chunks per thread");
    u32x4_t a[NA], w[NW];
    bool ka[NA], kw[NW];

    __device__ __forceinline__ void load(const PrefillGemmArgs& p, int m0, int n0, int k0, int tid) {
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            const int c = tid + NT * i, kc = k0 + (c % CPR) * EPC, m = m0 + c / CPR;
            ka[i] = m < p.M && kc < p.K;
            a[i] = *reinterpret_cast<const u32x4_t*>(reinterpret_cast<const T*>(p.A) + (size_t)min(m, p.M - 1) * p.lda +
                                                     min(kc, p.K - EPC));
        }
#pragma unroll
        for (int i = 0; i < NW; ++i) {
            const int c = tid + NT * i, kc = k0 + (c % CPR) * EPC;
            int j, nn;
            if constexpr (EP == PG_SWIGLU) {
                // the tile's first BN / 2 rows are gate rows n0 / 2 .., the others the same up rows
                const int l = c / CPR, f = n0 / 2 + l % (BN / 2);
                j = l / (BN / 2);
                kw[i] = f < p.n_per && kc < p.K;
                nn = j * p.n_per + min(f, p.n_per - 1);
            } else {
                const int n = n0 + c / CPR;
                kw[i] = n < p.N && kc < p.K;
                nn = min(n, p.N - 1);
                j = nn / p.n_per;
            }
            // matrix j as an element offset from W0 (arithmetic, not a branch per lane; the pointer
            // stays a global one, so the load is a global load)
            const T* w0 = reinterpret_cast<const T*>(p.W0);
            const ptrdiff_t d1 = (reinterpret_cast<intptr_t>(p.W1) - reinterpret_cast<intptr_t>(p.W0)) / (ptrdiff_t)sizeof(T);
            const ptrdiff_t d2 = (reinterpret_cast<intptr_t>(p.W2) - reinterpret_cast<intptr_t>(p.W0)) / (ptrdiff_t)sizeof(T);
            const ptrdiff_t off = j == 0 ? 0 : (j == 1 ? d1 : d2);
            // cached: the other row tiles of this column tile read the same weights from L2
            w[i] = *reinterpret_cast<const u32x4_t*>(w0 + off + (ptrdiff_t)(nn - j * p.n_per) * p.K + min(kc, p.K - EPC));
        }
    }
    __device__ __forceinline__ void store(T* sa, T* sw, int tid) const {
        constexpr int LDR = PTile<T, BK>::LDR;
        const u32x4_t zero = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            const int c = tid + NT * i;
            if (NA * NT == BM * CPR || c < BM * CPR)
                *reinterpret_cast<u32x4_t*>(sa + (c / CPR) * LDR + (c % CPR) * EPC) = ka[i] ? a[i] : zero;
        }
#pragma unroll
        for (int i = 0; i < NW; ++i) {
            const int c = tid + NT * i;
            if (NW * NT == BN * CPR || c < BN * CPR)
                *reinterpret_cast<u32x4_t*>(sw + (c / CPR) * LDR + (c % CPR) * EPC) = kw[i] ? w[i] : zero;
        }
    }
};

// Fused epilogues read the workgroup's C tile back from LDS (float rows of BN + 4: the 16 columns a
// wave's lanes write per row group land in distinct banks).
template <int BM, int BN> struct CTile { static constexpr int LD = BN + 4; static constexpr int BYTES = BM * LD * 4; };

template <typename T, int WM, int WN, int TM, int TN, int BK, int EP>
__global__ void __launch_bounds__(64 * WM * WN) prefill_gemm_kernel(PrefillGemmArgs p) {
    constexpr int BM = WM * TM * 16, BN = WN * TN * 16, NT = 64 * WM * WN;
    constexpr int LDR = PTile<T, BK>::LDR;
    constexpr int STAGE_BYTES = 2 * (BM + BN) * LDR * (int)sizeof(T);
    static_assert(EP == PG_STORE || CTile<BM, BN>::BYTES + BM * 4 <= STAGE_BYTES, "C tile fits the stage buffers");
    // the two stage buffers of A and W; after the last stage, the C tile of a fused epilogue
    __shared__ __align__(16) unsigned char smem[STAGE_BYTES];
    T (*s_a)[BM * LDR] = reinterpret_cast<T (*)[BM * LDR]>(smem);
    T (*s_w)[BN * LDR] = reinterpret_cast<T (*)[BN * LDR]>(smem + 2 * BM * LDR * sizeof(T));

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int c = lane & 15, g = lane >> 4;
    // tile order: the row tiles of one column tile are consecutive on one XCD
    const int m_tiles = (p.M + BM - 1) / BM, n_tiles = (p.N + BN - 1) / BN;
    const int total = m_tiles * n_tiles;
    const int kpart = (int)blockIdx.x / total;
    int t = (int)blockIdx.x - kpart * total;
    if (total % 8 == 0) t = (t % 8) * (total / 8) + t / 8;
    const int m0 = (t % m_tiles) * BM, n0 = (t / m_tiles) * BN;
    const int wm = wave / WN, wn = wave % WN;

    f32x4_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // this workgroup's share of the contraction (split-K: part kpart of p.ksplit, whole stages)
    const int stages_all = (p.K + BK - 1) / BK;
    const int per = (stages_all + p.ksplit - 1) / p.ksplit;
    const int st0 = kpart * per;
    const int steps = max(0, min(stages_all, st0 + per) - st0);
    const int kb = st0 * BK;
    // Two stages' global loads are in flight in registers while a third is read from LDS: at stage s
    // register set (s + 1) & 1 holds stage s + 1 (written to LDS after the stage-s products) and is
    // then reloaded with stage s + 3; set s & 1 holds stage s + 2, still arriving.  Loads past the
    // last stage read clamped, in-bounds addresses; their stage tiles are never read.
    StepLoad<T, BM, BN, NT, BK, EP> r0, r1;
    r0.load(p, m0, n0, kb, tid);
    r1.load(p, m0, n0, kb + BK, tid);
    r0.store(s_a[0], s_w[0], tid);
    __syncthreads();
    r0.load(p, m0, n0, kb + 2 * BK, tid);
    auto stage = [&](int s, StepLoad<T, BM, BN, NT, BK, EP>& next) {
        const int buf = s & 1;
#pragma unroll
        for (int kk = 0; kk < BK; kk += 32) {
            Frag<T> fa[TM], fw[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                fa[i] = Frag<T>::load(&s_a[buf][((wm * TM + i) * 16 + c) * LDR + kk + 8 * g]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                fw[j] = Frag<T>::load(&s_w[buf][((wn * TN + j) * 16 + c) * LDR + kk + 8 * g]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) mma(acc[i][j], fa[i], fw[j]);
        }
        // keep the LDS write after the products and the next loads before the following stage's: left
        // to itself the scheduler moves loads next to the write that consumes them, which then waits
        // out their latency
        __builtin_amdgcn_sched_barrier(0);
        next.store(s_a[buf ^ 1], s_w[buf ^ 1], tid);
        __syncthreads();
        next.load(p, m0, n0, kb + (s + 3) * BK, tid);
        __builtin_amdgcn_sched_barrier(0);
    };
    // stages in pairs, an odd last stage after the loop: with no exit between the two halves the
    // waits before each LDS write count only the other register set's loads (a conditional second
    // half makes the compiler wait for every load at the top of the loop)
    int s = 0;
    for (; s + 1 < steps; s += 2) {
        stage(s, r1);
        stage(s + 1, r0);
    }
    if (s < steps) stage(s, r1);
    // acc[i][j][r] = C[row 16 i + 4 g + r of the wave tile][column 16 j + c]
    if constexpr (EP == PG_STORE) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int n = n0 + (wn * TN + j) * 16 + c;
                if (n >= p.N) continue;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int m = m0 + (wm * TM + i) * 16 + 4 * g + r;
                    if (m < p.M) p.C[(size_t)kpart * p.c_part + (size_t)m * p.ldc + n] = acc[i][j][r];
                }
            }
    } else {
        // the C tile to LDS (every wave is past its last fragment reads), then each thread takes
        // pairs of columns of a row
        constexpr int LDC = CTile<BM, BN>::LD;
        float* tile = reinterpret_cast<float*>(smem);
        __syncthreads();
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    tile[((wm * TM + i) * 16 + 4 * g + r) * LDC + (wn * TN + j) * 16 + c] = acc[i][j][r];
        __syncthreads();
        if constexpr (EP == PG_QKV) {
            // the tile rows' cache positions, once per row (-1: past the cache, flagged, not written)
            int* s_pos = reinterpret_cast<int*>(smem + CTile<BM, BN>::BYTES);
            for (int r = tid; r < BM; r += NT) {
                const int m = m0 + r;
                int pos = -1;
                if (m < p.M) {
                    const int b = m / p.q;
                    pos = p.cache_len[b] + (m - b * p.q);
                    if (pos >= p.S_max) {   // the host checks capacity; never write past the cache
                        atomicOr(p.err, 4);
                        pos = -1;
                    }
                }
                s_pos[r] = pos;
            }
            __syncthreads();
            const int hd = p.Dh / 2;
            if (n0 / p.n_per == 2 && (n0 + BN - 1) / p.n_per == 2) {
                // a V tile: consecutive threads take consecutive rows of a column, so the 32 keys of a
                // cache block (one key-permuted 64-byte run per dimension) are written together
#pragma unroll 4
                for (int it = tid; it < BM * BN; it += NT) {
                    const int col = it / BM, r = it % BM, n = n0 + col, pos = s_pos[r];
                    if (pos < 0 || n >= p.N) continue;
                    const int m = m0 + r, b = m / p.q, h = (n % p.n_per) / p.Dh, i = (n % p.n_per) % p.Dh;
                    T* vo = static_cast<T*>(p.vc) + (((size_t)b * p.H + h) * (p.S_max / 32) + pos / 32) * p.Dh * 32 +
                            vperm(pos & 31);
                    vo[(size_t)i * 32] = to_elem<T>(tile[r * LDC + col]);
                }
            } else {
                // RoPE pairs columns i and i + Dh / 2 of a head (heads of Dh | BN columns start at tile
                // column multiples of Dh); the segment (Q, K, V) and head follow from the column
                constexpr int ITEMS = BM * (BN / 2) / NT;
                static_assert(ITEMS * NT == BM * (BN / 2), "whole items per thread");
#pragma unroll
                for (int u = 0; u < ITEMS; ++u) {
                    const int it = tid + u * NT;
                    const int r = it / (BN / 2), pr = it % (BN / 2), pos = s_pos[r];
                    const int a = (pr / hd) * p.Dh + pr % hd, n = n0 + a;
                    if (pos < 0 || n >= p.N) continue;
                    const int m = m0 + r, b = m / p.q;
                    const int seg = n / p.n_per, h = (n % p.n_per) / p.Dh, i = pr % hd;
                    const float x1 = tile[r * LDC + a], x2 = tile[r * LDC + a + hd];
                    if (seg == 2) {
                        T* vo = static_cast<T*>(p.vc) + (((size_t)b * p.H + h) * (p.S_max / 32) + pos / 32) * p.Dh * 32 +
                                vperm(pos & 31);
                        vo[(size_t)i * 32] = to_elem<T>(x1);
                        vo[(size_t)(i + hd) * 32] = to_elem<T>(x2);
                        continue;
                    }
                    const float2 csn = *reinterpret_cast<const float2*>(p.rope + ((size_t)pos * hd + i) * 2);
                    const float cs = csn.x, sn = csn.y;
                    const float y1 = x1 * cs - x2 * sn, y2 = x1 * sn + x2 * cs;
                    if (seg == 0) {
                        float* qo = p.qbuf + ((size_t)m * p.H + h) * p.Dh;
                        qo[i] = y1;
                        qo[i + hd] = y2;
                    } else {
                        T* ko = static_cast<T*>(p.kc) + (((size_t)b * p.H + h) * p.S_max + pos) * p.Dh;
                        ko[i] = to_elem<T>(y1);
                        ko[i + hd] = to_elem<T>(y2);
                    }
                }
            }
        } else {
            // columns 0 .. BN / 2 - 1 hold gate outputs n0 / 2 .., the others the same up outputs
            for (int it = tid; it < BM * (BN / 2); it += NT) {
                const int r = it / (BN / 2), i = it % (BN / 2);
                const int m = m0 + r, f = n0 / 2 + i;
                if (m >= p.M || f >= p.n_per) continue;
                const float gate = tile[r * LDC + i], v = tile[r * LDC + BN / 2 + i];
                static_cast<T*>(p.u)[(size_t)m * p.ldu + f] = to_elem<T>(gate / (1.0f + expf(-gate)) * v);
            }
        }
    }
}

template <typename T, int WM, int WN, int TM, int TN, int BK>
hipError_t go(const PrefillGemmArgs& p, hipStream_t s) {
    constexpr int BM = WM * TM * 16, BN = WN * TN * 16;
    static_assert(BN == 128, "fused epilogues: heads of 64 or 128 columns and 64 gate | 64 up outputs per tile");
    const long tiles = (long)((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
    auto kern = prefill_gemm_kernel<T, WM, WN, TM, TN, BK, PG_STORE>;
    if (p.ep == PG_QKV) kern = prefill_gemm_kernel<T, WM, WN, TM, TN, BK, PG_QKV>;
    else if (p.ep == PG_SWIGLU) kern = prefill_gemm_kernel<T, WM, WN, TM, TN, BK, PG_SWIGLU>;
    hipLaunchKernelGGL(kern, dim3((unsigned)(tiles * p.ksplit)), dim3(64 * WM * WN), 0, s, p);
    return hipGetLastError();
}

}  // namespace

int prefill_gemm_ksplit(int M, int N, int K) {
    const long tiles = (long)((M + 127) / 128) * ((N + 127) / 128);
    if (K < 1024 || tiles >= 256) return 1;
    return tiles <= 128 && K >= 2048 ? 4 : 2;
}

// 128 x 128 tiles (bf16: 8 waves of 32 x 64, float: 4 waves of 64 x 64, 32-wide
// stages).  prefill_gemm_ksplit: a GEMM whose tiles make less than one round of
// workgroups over the 256 compute units and whose contraction is long is split
// into parts whose partials the caller adds; up to two workgroups of 80 KB of LDS
// fit a compute unit, so a split fills both (O and down at 7B, 511 rows: 128
// tiles, 4 parts, 512 workgroups).
hipError_t launch_prefill_gemm(int dtype, const PrefillGemmArgs& p, hipStream_t s) {
    if (p.M < 1 || p.N < 1 || p.K < 1 || p.K % 8 || p.n_per < 1 || p.N > 3 * p.n_per || !p.A || !p.W0 ||
        (p.N > p.n_per && !p.W1) || (p.N > 2 * p.n_per && !p.W2) || p.lda < p.K || p.ksplit < 1 || p.ksplit > kPrefillMaxSplit)
        return hipErrorInvalidValue;
    if (p.ep == PG_STORE) {
        if (!p.C || p.ldc < p.N || (p.ksplit > 1 && p.c_part < (size_t)p.M * p.ldc)) return hipErrorInvalidValue;
    } else if (p.ep == PG_QKV) {
        // heads tile the 128-column workgroup tiles; the segments are whole heads
        if (p.ksplit != 1 || p.N != 3 * p.n_per || (p.Dh != 64 && p.Dh != 128) || p.H < 1 || p.n_per != p.H * p.Dh ||
            p.q < 1 || p.M % p.q || p.S_max < 32 || p.S_max % 32 || !p.cache_len || !p.rope || !p.qbuf || !p.kc ||
            !p.vc || !p.err)
            return hipErrorInvalidValue;
    } else if (p.ep == PG_SWIGLU) {
        if (p.ksplit != 1 || p.N != 2 * p.n_per || !p.u || p.ldu < p.n_per) return hipErrorInvalidValue;
    } else {
        return hipErrorInvalidValue;
    }
    if (dtype != 1) return go<float, 2, 2, 4, 4, 32>(p, s);
    return go<uint16_t, 4, 2, 2, 4, 64>(p, s);
}

}  // namespace sdsat
