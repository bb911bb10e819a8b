// Matrix-core GEMM for blocks of many rows (the prompt prefill before the
// draft/verify loop, Section 2.1): C[M, N] = A[M, K] . W[N, K]^T with A the
// normalised activations (element type, rows padded with zeros), W the
// caller's row-major [out, in] weights -- up to three matrices stacked along
// N (Q | K | V, gate | up) -- and C float.  At hundreds of rows a weight byte
// feeds hundreds of flops, so unlike the decode GEMM this kernel is bound by
// the matrix cores and by how often operands are re-read, not by HBM.
//
// Tiling: a workgroup of 4 waves computes a BM x BN tile of C, the waves in a
// WM x WN grid, each a (16 TM) x (16 TN) sub-tile of matrix-core 16x16 tiles.
// The contraction runs in 32-wide steps; both operands' step tiles are staged
// in LDS (double-buffered), with the global loads of the next two steps in
// flight in registers while the current step's fragments are read from LDS
// and multiplied; one barrier per step.  LDS rows are padded by 16 bytes so that the 16 lanes reading one
// fragment column hit distinct banks.  Every element of C is accumulated by
// one wave in one fixed order of k, so results repeat bit for bit.
// Workgroups that share a weight tile (the same N tile, different M tiles) are
// placed on the same XCD (workgroups go to the 8 XCDs round-robin), so the
// weights come from HBM once and the other row tiles read them from that L2.
#include "device.h"
#include "kernels.h"

namespace sdsat {

namespace {

// contraction elements per LDS stage: one matrix-core step (measured on MI355X, 7B 511-row prefill:
// 21.5 ms against 22.7 ms with two steps per stage, whose larger LDS tiles allow one workgroup less
// per compute unit)
template <typename T> struct PTile {
    static constexpr int BK = 32;
    static constexpr int EPC = 16 / sizeof(T);          // elements per 16-byte chunk
    static constexpr int LDR = BK + 16 / sizeof(T);     // LDS row stride in elements (16 bytes of padding)
};

// Global -> registers: this thread's chunks of the A and W step tiles (zero past M, N or K).
template <typename T, int BM, int BN>
struct StepLoad {
    static constexpr int EPC = PTile<T>::EPC;
    static constexpr int CPR = PTile<T>::BK / EPC;        // chunks per row of a stage tile
    static constexpr int NA = BM * CPR / 256, NW = BN * CPR / 256;
    u32x4_t a[NA], w[NW];

    __device__ __forceinline__ void load(const PrefillGemmArgs& p, int m0, int n0, int k0, int tid) {
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            const int c = tid + 256 * i, row = c / CPR, kc = k0 + (c % CPR) * EPC;
            const int m = m0 + row;
            a[i] = u32x4_t{0u, 0u, 0u, 0u};
            if (m < p.M && kc < p.K)
                a[i] = *reinterpret_cast<const u32x4_t*>(reinterpret_cast<const T*>(p.A) + (size_t)m * p.lda + kc);
        }
#pragma unroll
        for (int i = 0; i < NW; ++i) {
            const int c = tid + 256 * i, row = c / CPR, kc = k0 + (c % CPR) * EPC;
            const int n = n0 + row;
            w[i] = u32x4_t{0u, 0u, 0u, 0u};
            if (n < p.N && kc < p.K) {
                const int j = n / p.n_per;
                const T* src = reinterpret_cast<const T*>(j == 0 ? p.W0 : (j == 1 ? p.W1 : p.W2));
                // cached: the other row tiles of this column tile read the same weights from L2
                w[i] = *reinterpret_cast<const u32x4_t*>(src + (size_t)(n - j * p.n_per) * p.K + kc);
            }
        }
    }
    __device__ __forceinline__ void store(T* sa, T* sw, int tid) const {
        constexpr int LDR = PTile<T>::LDR;
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            const int c = tid + 256 * i;
            *reinterpret_cast<u32x4_t*>(sa + (c / CPR) * LDR + (c % CPR) * EPC) = a[i];
        }
#pragma unroll
        for (int i = 0; i < NW; ++i) {
            const int c = tid + 256 * i;
            *reinterpret_cast<u32x4_t*>(sw + (c / CPR) * LDR + (c % CPR) * EPC) = w[i];
        }
    }
};

template <typename T, int WM, int WN, int TM, int TN>
__global__ void __launch_bounds__(256) prefill_gemm_kernel(PrefillGemmArgs p) {
    constexpr int BM = WM * TM * 16, BN = WN * TN * 16;
    constexpr int LDR = PTile<T>::LDR, BK = PTile<T>::BK;
    static_assert(WM * WN == 4, "four waves per workgroup");
    __shared__ __align__(16) T s_a[2][BM * LDR];
    __shared__ __align__(16) T s_w[2][BN * LDR];

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
    // then reloaded with stage s + 3; set s & 1 holds stage s + 2, still arriving.
    StepLoad<T, BM, BN> r0, r1;
    if (steps > 0) r0.load(p, m0, n0, kb, tid);
    if (steps > 1) r1.load(p, m0, n0, kb + BK, tid);
    if (steps > 0) r0.store(s_a[0], s_w[0], tid);
    __syncthreads();
    if (steps > 2) r0.load(p, m0, n0, kb + 2 * BK, tid);
    auto stage = [&](int s, StepLoad<T, BM, BN>& next) {
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
        if (s + 1 < steps) next.store(s_a[buf ^ 1], s_w[buf ^ 1], tid);
        __syncthreads();
        if (s + 3 < steps) next.load(p, m0, n0, kb + (s + 3) * BK, tid);
    };
    for (int s = 0; s < steps; s += 2) {
        stage(s, r1);
        if (s + 1 < steps) stage(s + 1, r0);
    }
    // acc[i][j][r] = C[row 16 i + 4 g + r of the wave tile][column 16 j + c]
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
}

template <typename T, int WM, int WN, int TM, int TN>
hipError_t go(const PrefillGemmArgs& p, hipStream_t s) {
    constexpr int BM = WM * TM * 16, BN = WN * TN * 16;
    const long tiles = (long)((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
    hipLaunchKernelGGL((prefill_gemm_kernel<T, WM, WN, TM, TN>), dim3((unsigned)(tiles * p.ksplit)), dim3(256), 0, s,
                       p);
    return hipGetLastError();
}

}  // namespace

int prefill_gemm_ksplit(int M, int N, int K) {
    const long tiles = (long)((M + 127) / 128) * ((N + 127) / 128);
    return tiles < 256 && K >= 1024 ? 2 : 1;
}

// 128 x 128 tiles.  prefill_gemm_ksplit: a GEMM whose tiles make less than
// one round of workgroups over the 256 compute units and whose contraction is
// long is better split in two (O and down at 7B: 128 -> 256 workgroups), where
// the caller can add the partials.
hipError_t launch_prefill_gemm(int dtype, const PrefillGemmArgs& p, hipStream_t s) {
    if (p.M < 1 || p.N < 1 || p.K < 1 || p.K % 8 || p.n_per < 1 || p.N > 3 * p.n_per || !p.A || !p.W0 || !p.C ||
        (p.N > p.n_per && !p.W1) || (p.N > 2 * p.n_per && !p.W2) || p.lda < p.K || p.ldc < p.N ||
        p.ksplit < 1 || p.ksplit > 2 || (p.ksplit > 1 && p.c_part < (size_t)p.M * p.ldc))
        return hipErrorInvalidValue;
    return dtype == 1 ? go<uint16_t, 2, 2, 4, 4>(p, s) : go<float, 2, 2, 4, 4>(p, s);
}

}  // namespace sdsat
