// Skinny weight-streaming GEMM for block decode: Y[M, N] = X[M, K] . W[N, K]^T with
// M = batch * block rows (<= 64) and N, K model dimensions.  At M <= 64 the
// contraction does about M flops per weight byte, far below the matrix-core
// ridge, so the kernel is bound by streaming W from HBM once.  The design:
//
//  * W is pre-packed (launch_pack) into 16-column x 32-k tiles laid out in lane
//    order, so every wave-wide load is one contiguous 1 KiB (bf16) run and each
//    lane's 16 bytes is directly its matrix-core B fragment.
//  * One workgroup per column tile (4 for prefill chunks).  Its waves split the
//    contraction into contiguous slices, stream their slice with two batches of
//    loads in flight, read the X fragments for the same steps straight from
//    global memory (the few X rows stay in L2), and reduce their partial tiles
//    through LDS in wave order: deterministic, with no device-scope fences or
//    atomics.
//  * An RMSNorm input arrives either already normalised and rounded to the
//    element type (rms_rows; blocks of several rows, whose float rows re-read by
//    every workgroup would cost as much traffic as the weights), or, for one-row
//    blocks, as the float rows x o g (gain applied by the producer): the kernel
//    then reduces the producer's per-tile sums of squares to each row's 1/rms
//    before its first matrix-core step and rounds x o g / rms to the element
//    type at the matrix-core input.  Both give the normalised activation a bf16
//    model stores, rounded once, bit for bit the same.
//  * Residual GEMMs whose tile count would leave some compute units a second
//    workgroup (13B: 320 tiles on 256 units), and long narrow ones of blocks of
//    several row tiles (four tiles per workgroup, so each row byte read feeds
//    four), spread each tile's waves over several workgroups and fold the
//    waves' partial tiles in a second kernel, in the same wave order
//    (plan_gemm_resid).
//  * Fused epilogues, run by wave 0 on the reduced tile:
//      EP_STORE   float output (LM-head logits)
//      EP_QKV     RoPE on Q and K columns, Q (float) to its buffer, K and V into
//                 the cache slots of the block rows (positions cache_len[b] + r)
//      EP_RESID   residual add into the float residual stream, the updated rows
//                 times the next RMSNorm's gain, and per-tile sums of squares
//                 that the next RMSNorm reduces
//      EP_SWIGLU  silu(gate) * up, rounded to the activation type
#include <algorithm>
#include <type_traits>

#include <hip/hip_ext.h>

#include "device.h"
#include "kernels.h"

namespace sdsat {

size_t packed_elems(int n_tiles, int k_steps) { return (size_t)n_tiles * k_steps * 64 * 8; }

template <typename T>
__global__ void pack_kernel(PackArgs a) {
    const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;   // (tile, kstep, lane)
    const size_t total = (size_t)a.n_tiles * a.k_steps * 64;
    if (idx >= total) return;
    const int lane = (int)(idx & 63);
    const size_t tk = idx >> 6;
    const int ks = (int)(tk % a.k_steps);
    const int t = (int)(tk / a.k_steps);
    const int c = lane & 15, g = lane >> 4;
    long row = -1;   // stacked source row
    if (a.perm == PACK_PLAIN) {
        row = 16L * t + c;
    } else if (a.perm == PACK_ROPE) {
        const int tph = a.head_dim / 16, half = a.head_dim / 2;
        const int head = t / tph, j = t % tph;
        const int dim = c < 8 ? 8 * j + c : half + 8 * j + (c - 8);
        row = (long)head * a.head_dim + dim;
    } else {  // PACK_GATEUP
        const int f = 8 * t + (c & 7);
        row = f < a.F ? (c < 8 ? f : (long)a.F + f) : -1;
    }
    const T* src = nullptr;
    long r = row;
    if (row >= 0 && row < a.N) {
        if (r < a.N0) src = (const T*)a.src0;
        else if ((r -= a.N0) < a.N1) src = (const T*)a.src1;
        else { r -= a.N1; src = (const T*)a.src2; }
    }
    T* dst = (T*)a.dst + idx * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int k = 32 * ks + 8 * g + e;
        float v = 0.f;
        if (src && k < a.K) v = to_f32<T>(src[r * a.K + k]);
        dst[e] = to_elem<T>(v);
    }
}

void launch_pack(const PackArgs& a, hipStream_t s) {
    const size_t total = (size_t)a.n_tiles * a.k_steps * 64;
    const int blocks = (int)((total + 255) / 256);
    if (a.dtype == 1) hipLaunchKernelGGL(pack_kernel<uint16_t>, dim3(blocks), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(pack_kernel<float>, dim3(blocks), dim3(256), 0, s, a);
}

// Plans (measured on MI355X with weights streamed from HBM):
//  * blocks of up to 16 rows: one column tile per workgroup, 8 waves for the
//    narrow [d, d] / [d, F] matrices (256 tiles, one workgroup per compute
//    unit), 4 for the wide ones; at least 4 contraction steps per wave
//    (several tiles per workgroup, or X staged in LDS, measured slower);
//  * blocks of more than 16 rows (batch 4 decode, prefill chunks) reload their
//    X fragments for every weight fragment: for the wide matrices a workgroup
//    of 4 waves takes several column tiles so that one X load feeds their
//    matrix-core steps: 4 (M = 64: QKV 55 -> 37 us, gate/up 103 -> 62 us), or
//    2 for two row tiles, which keeps more workgroups than compute units
//    (batch 4 x 6 rows: QKV 192 -> 384 workgroups, 34.4 -> 31.5 us; gate/up
//    47.5 -> 42.1 us; block 4.92 -> 4.67 ms); the narrow ones keep one tile
//    per workgroup.  The waves per workgroup depend on the matrix shape only
//    where block-size invariance needs it: one row tile and several column
//    tiles both use 4 waves on the wide matrices.
GemmPlan plan_gemm(int M, int n_tiles, int k_steps) {
    GemmPlan p;
    p.mt = (M + 15) / 16;
    p.ntw = (p.mt > 1 && n_tiles > 512) ? (p.mt == 2 ? 2 : 4) : 1;
    int w = p.ntw > 1 ? 4 : (n_tiles <= 512 ? 8 : 4);
    while (w > 1 && k_steps < 4 * w) w /= 2;
    p.waves = w;
    p.grid = (n_tiles + p.ntw - 1) / p.ntw;
    p.lds_bytes = w * p.mt * 64 * 16;
    p.ksplit = 1;
    return p;
}

// Residual GEMMs (O, down) of narrow matrices whose tile count is not a
// multiple of the 256 compute units (13B: 320 tiles) leave some units two
// workgroups and the rest one.  Their tiles' waves are then spread over
// ksplit workgroups (320 x 4 = 1280 workgroups of 2 waves, 5 per unit); each
// wave keeps its slice of the contraction, and a fold kernel adds the waves'
// partial tiles in wave order, as the single workgroup's LDS reduction does,
// so the results are the same bit for bit.  Measured at 13B, 11 rows: down
// (432 contraction steps) 39.4 -> 32.6 us; O (160 steps) 16.6 -> 17.1 us, its
// waves' work too short to cover the fold kernel's launch, so it stays whole.
// Blocks of several row tiles re-read all of their rows in every workgroup (L2 hits, but at batch
// 4 x 6 rows the down GEMM's 528 KB of rows per workgroup outweigh its 352 KB of weights).  A narrow
// residual GEMM with a long contraction then takes four column tiles per workgroup, so each row byte
// feeds four tiles, and spreads each tile's wave slices over one-wave workgroups (same slices, same
// fold order: the same values).  Measured on the 7B down GEMM: batch 4 x 6 rows 29.2 -> 27.5 us,
// batch 8 x 6 rows 45.5 -> 34.0 us (the fold included); the O GEMM (128 steps) split the same way
// was slower at batch 8 and 10.
GemmPlan plan_gemm_resid(int M, int n_tiles, int k_steps) {
    GemmPlan p = plan_gemm(M, n_tiles, k_steps);
    if (p.mt > 1 && p.ntw == 1 && n_tiles <= 512 && k_steps >= 256) {
        p.ntw = 4;
        p.ksplit = p.waves;
        p.waves = 1;
        p.grid = (n_tiles + p.ntw - 1) / p.ntw * p.ksplit;
        p.lds_bytes = p.waves * p.mt * 64 * 16;
        return p;
    }
    if (p.ntw != 1 || n_tiles <= 256 || k_steps < 256) return p;
    auto spread = [&](int k) {   // workgroup rounds over the average, per compute unit
        const long n = (long)n_tiles * k;
        return (double)((n + 255) / 256) * 256.0 / (double)n;
    };
    int best = 1;
    for (int k = 2; k <= p.waves; k *= 2)
        if (spread(k) < spread(best) - 1e-9) best = k;
    p.ksplit = best;
    p.waves /= best;
    p.grid = n_tiles * best;
    p.lds_bytes = p.waves * p.mt * 64 * 16;
    return p;
}

size_t gemm_resid_part_bytes(int n_tiles, int k_steps, int max_rows) {
    size_t most = 0;
    for (int m = 1; m <= std::min(std::max(max_rows, 1), 64); m += 16) {
        const GemmPlan p = plan_gemm_resid(std::min(m + 15, std::min(std::max(max_rows, 1), 64)), n_tiles, k_steps);
        if (p.ksplit > 1) most = std::max(most, (size_t)n_tiles * p.waves * p.ksplit * p.mt * 64 * 16);
    }
    return most;
}

// Steps per load batch (two batches in flight), sized so both batches of
// weight and X fragments fit the register budget (float X fragments of an
// RMSNorm input take twice the registers of bf16 ones).  The QKV GEMM on float
// rows takes 4 (142 VGPRs: its 3 workgroups of 4 waves per compute unit stay
// resident; 7B, 6 rows: 22.1 -> 21.2 us); the other float-row GEMMs keep 3
// (gate/up, 1376 workgroups, loses occupancy at 4: 32.4 -> 33.2 us at one row).
template <typename T, int EP, int MT, bool XF> struct Batch {
    static constexpr int U = MT == 1 ? (sizeof(T) == 2 ? (XF ? (EP == EP_QKV ? 4 : 3) : 4) : 2)
                                     : (sizeof(T) == 2 && !XF ? 2 : 1);
};

// X fragment as loaded: the element type, or raw floats of an RMSNorm input.
template <typename T, bool XF> struct XIn { using type = Frag<T>; };
template <typename T> struct XIn<T, true> { using type = Frag<float>; };

// Matrix-core A fragment from a loaded X fragment: RMSNorm inputs are scaled
// by the row's 1/rms and rounded to the element type here.
template <typename T, bool XF, typename XT>
__device__ __forceinline__ Frag<T> a_frag(const XT& x, float inv) {
    if constexpr (XF) {
        float v[8] = {x.lo.x * inv, x.lo.y * inv, x.lo.z * inv, x.lo.w * inv,
                      x.hi.x * inv, x.hi.y * inv, x.hi.z * inv, x.hi.w * inv};
        return Frag<T>::from_f32(v);
    } else {
        return x;
    }
}

// One batch of U contraction steps: the weight fragments of the NTW tiles
// (streamed, non-temporal) and the X fragments of every row tile.  TAIL
// batches may run past the wave's slice: those steps reload the last step
// with X zeroed.  Loads of the steady-state loop are unconditional so that
// the compiler's wait counts stay exact and two batches really are in flight.
template <typename T, typename XT, int MT, int NTW, int U, bool TAIL>
__device__ __forceinline__ void load_batch(Frag<T> (&w)[U][NTW], XT (&x)[U][MT], const T* const (&wp)[NTW],
                                           __amdgpu_buffer_rsrc_t xrs, const uint32_t (&xo)[MT], int s, int nks) {
    constexpr uint32_t step_bytes = 32 * (sizeof(XT) / 8);   // 32 elements of the X type
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int st = TAIL ? min(s + u, nks - 1) : s + u;
#pragma unroll
        for (int j = 0; j < NTW; ++j) w[u][j] = Frag<T>::load_nt(wp[j] + (size_t)st * 512);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            x[u][mt] = buf_frag<typename XT::elem>(xrs, xo[mt] + (uint32_t)st * step_bytes, 0);
            if (TAIL && s + u >= nks) x[u][mt] = XT::zero();
        }
    }
}

template <typename T, bool XF, typename XT, int MT, int NTW, int U>
__device__ __forceinline__ void mma_batch(f32x4_t (&acc)[NTW][MT], const Frag<T> (&w)[U][NTW],
                                          const XT (&x)[U][MT], const float (&inv)[MT]) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const Frag<T> xa = a_frag<T, XF>(x[u][mt], inv[mt]);
#pragma unroll
            for (int j = 0; j < NTW; ++j) mma(acc[j][mt], xa, w[u][j]);
        }
}

// Fused epilogue of one reduced tile (run by wave 0).
// acc[mt][r] = Y[m = 16mt + 4g + r][column c of the tile]
// gn: EP_RESID's next-RMSNorm gain at this lane's column (requested in the prologue)
template <typename T, int EP, int MT>
__device__ __forceinline__ void epilogue(const GemmArgs& a, int tile, const f32x4_t (&acc)[MT],
                                         const float (&ep_in)[MT][4], float gn, int c, int g) {
    const int M = a.M;
    if (EP == EP_STORE) {
        const int n = tile * 16 + c;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = 16 * mt + 4 * g + r;
                if (m < M && n < a.N) a.y[(size_t)m * a.ldy + n] = acc[mt][r];
            }
    } else if (EP == EP_RESID) {
        const int n = tile * 16 + c;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = 16 * mt + 4 * g + r;
                float ss = 0.f;
                if (m < M && n < a.N) {
                    const float v = ep_in[mt][r] + acc[mt][r];
                    a.resid[(size_t)m * a.ldy + n] = v;
                    a.xg_out[(size_t)m * a.ldxg + n] = v * gn;
                    ss = v * v;
                }
                ss += __shfl_xor(ss, 8, 64);
                ss += __shfl_xor(ss, 4, 64);
                ss += __shfl_xor(ss, 2, 64);
                ss += __shfl_xor(ss, 1, 64);
                if (c == 0 && m < M) a.ssq_out[(size_t)m * a.n_tiles + tile] = ss;
            }
    } else if (EP == EP_SWIGLU) {
        const int f = 8 * tile + (c & 7);
        T* u = reinterpret_cast<T*>(a.uout);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = 16 * mt + 4 * g + r;
                const float mine = acc[mt][r];
                const float other = __shfl_xor(mine, 8, 64);
                if (c < 8 && m < M && f < a.F) {
                    const float gate = mine, up = other;
                    u[(size_t)m * a.ldu + f] = to_elem<T>(gate / (1.0f + expf(-gate)) * up);
                }
            }
    } else if (EP == EP_QKV) {
        const int Dh = a.Dh, half = Dh / 2, H = a.H;
        const int tph = Dh / 16;
        const int head_all = tile / tph, j = tile % tph;
        const int sec = head_all / H, h = head_all % H;        // 0 = Q, 1 = K, 2 = V
        const int pi = 8 * j + (c & 7);
        const int dim = c < 8 ? pi : half + pi;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = 16 * mt + 4 * g + r;
                const float mine = acc[mt][r];
                const float other = __shfl_xor(mine, 8, 64);
                if (m >= M || sec > 2) continue;
                const int b = m / a.q, row = m - b * a.q;
                const int L = __float_as_int(ep_in[mt][r]);
                const int pos = L + row;                // cache slot of this block row
                if (pos >= a.S_max) {                   // the host checks capacity; never write past the cache
                    atomicOr(a.err, 4);
                    continue;
                }
                float out = mine;
                if (sec < 2) {
                    // rotary position: the row's depth in the block (its ancestors
                    // counted by the tree mask; row index for a chain), at most pos.
                    // cos / sin come from the table (angle formed in double, rounded
                    // to float).  Requesting them in the prologue, once the cache
                    // lengths are in, measured slower.
                    const int rpos = a.mask ? L + __popcll(a.mask[m]) - 1 : pos;
                    const float2 csn = *reinterpret_cast<const float2*>(a.rope + ((size_t)rpos * half + pi) * 2);
                    const float cs = csn.x, sn = csn.y;
                    out = c < 8 ? mine * cs - other * sn : other * sn + mine * cs;
                }
                if (sec == 0) {
                    reinterpret_cast<float*>(a.qbuf)[((size_t)m * H + h) * Dh + dim] = out;
                } else if (sec == 1) {
                    reinterpret_cast<T*>(a.kc)[(((size_t)b * H + h) * a.S_max + pos) * Dh + dim] = to_elem<T>(out);
                } else {
                    const size_t blk = ((size_t)b * H + h) * (a.S_max / 32) + pos / 32;
                    reinterpret_cast<T*>(a.vc)[(blk * Dh + dim) * 32 + vperm(pos & 31)] = to_elem<T>(out);
                }
            }
    }
}

template <typename T, int EP, int MT, int NTW, bool XF>
// Workgroups of several tiles have 4 waves, the others at most 8.
__global__ void __launch_bounds__(NTW > 1 ? 256 : 512) gemm_kernel(GemmArgs a) {
    constexpr int U = Batch<T, EP, MT, XF>::U;
    using XT = typename XIn<T, XF>::type;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    f32x4_t* red = reinterpret_cast<f32x4_t*>(smem_raw);   // [waves][MT][64]
    __shared__ float s_inv[64];

    const int nw = blockDim.x >> 6;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int c = lane & 15, g = lane >> 4;
    const int M = a.M;
    // a split residual GEMM: workgroup (kpart, group of NTW tiles) holds waves kpart * nw .. of each
    // of its tiles' nwt
    const bool split = EP == EP_RESID && a.ksplit > 1;
    const int n_groups = (a.n_tiles + NTW - 1) / NTW;
    const int kpart = split ? (int)blockIdx.x / n_groups : 0;
    const int tile0 = ((int)blockIdx.x - kpart * n_groups) * NTW;
    const int nwt = split ? nw * a.ksplit : nw;
    const int gw = kpart * nw + wave;

    // this wave's contiguous slice of the contraction steps
    const int chunk = (a.k_steps + nwt - 1) / nwt;
    const int ks0 = gw * chunk;
    const int nks = max(0, min(a.k_steps, ks0 + chunk) - ks0);
    const T* wp[NTW];
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
        const int t = min(tile0 + j, a.n_tiles - 1);   // a tile past the end is read, not stored
        wp[j] = reinterpret_cast<const T*>(a.W) + (((size_t)t * a.k_steps + ks0) * 64 + lane) * 8;
    }

    // RMSNorm partial sums (wave w reduces rows w, w+nw, ...; the first two
    // are requested here, ahead of the weight stream) and wave 0's epilogue
    // inputs (residual values and the next RMSNorm's gains, cache lengths).
    constexpr int NSQ = 4;   // ssq partials per lane and row (n_ssq <= 256)
    float sq[2][NSQ];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int t = 0; t < NSQ; ++t) {
            const int m = wave + j * nw, col = lane + 64 * t;
            sq[j][t] = (XF && m < M && col < a.n_ssq) ? a.ssq[(size_t)m * a.n_ssq + col] : 0.f;
        }
    // EP_RESID: residual values per tile; EP_QKV: cache_len of each row's
    // sequence (the same for every tile)
    constexpr int NEP = EP == EP_RESID ? NTW : 1;
    float ep_in[NEP][MT][4];
    float gnv[NEP];                 // EP_RESID: the next RMSNorm's gain at each tile's column
#pragma unroll
    for (int j = 0; j < NEP; ++j) {
        gnv[j] = 0.f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) ep_in[j][mt][r] = 0.f;
    }
    if (wave == 0 && !split) {
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
            const int tile = tile0 + j;
            if (tile >= a.n_tiles) break;
            if (EP != EP_RESID && j > 0) continue;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int m = 16 * mt + 4 * g + r;
                    if (EP == EP_RESID && m < M && tile * 16 + c < a.N)
                        ep_in[j < NEP ? j : 0][mt][r] = a.resid[(size_t)m * a.ldy + tile * 16 + c];
                    if (EP == EP_QKV && m < M) ep_in[0][mt][r] = __int_as_float(a.cache_len[m / a.q]);
                }
            if (EP == EP_RESID && tile * 16 + c < a.N) gnv[j < NEP ? j : 0] = a.gnext[tile * 16 + c];
        }
    }

    f32x4_t acc[NTW][MT];
#pragma unroll
    for (int j = 0; j < NTW; ++j)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[j][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // Both weight batches are in flight before anything waits, then the loop
    // keeps two in flight.
    Frag<T> w0[U][NTW], w1[U][NTW];
    XT x0[U][MT], x1[U][MT];
    // X rows [0, M) as a buffer resource; lane offsets in bytes (rows past M
    // point past its end and read zeros without a memory access)
    constexpr uint32_t xes = sizeof(XT) / 8;   // bytes per X element as stored
    const uint32_t x_bytes = (uint32_t)M * (uint32_t)a.ldx * xes;
    const __amdgpu_buffer_rsrc_t xrs = buf_rsrc(XF ? (const void*)a.xf : a.xa, x_bytes);
    uint32_t xr[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int m = 16 * mt + c;
        xr[mt] = m < M ? ((uint32_t)m * a.ldx + ks0 * 32 + 8 * g) * xes : x_bytes;
    }
    if (nks > 0) {
        load_batch<T, XT, MT, NTW, U, true>(w0, x0, wp, xrs, xr, 0, nks);
        load_batch<T, XT, MT, NTW, U, true>(w1, x1, wp, xrs, xr, U, nks);
    }

    // row scales 1/rms, needed before the first matrix-core step (rows past
    // the two prefetched ones, and partials past 64 * NSQ columns, are read now)
    float inv[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) inv[mt] = 1.f;
    if (XF) {
        for (int m = wave, j = 0; m < M; m += nw, ++j) {
            float v = 0.f;
            if (j < 2) {
#pragma unroll
                for (int t = 0; t < NSQ; ++t) v += sq[j < 1 ? 0 : 1][t];
                for (int col = lane + 64 * NSQ; col < a.n_ssq; col += 64) v += a.ssq[(size_t)m * a.n_ssq + col];
            } else {
                for (int col = lane; col < a.n_ssq; col += 64) v += a.ssq[(size_t)m * a.n_ssq + col];
            }
            v = wave_sum(v);
            if (lane == 0) s_inv[m] = 1.0f / sqrtf(v / (float)a.K + a.eps);
        }
        __syncthreads();
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int m = 16 * mt + c;
            inv[mt] = m < M ? s_inv[m] : 0.f;
        }
    }

    if (nks > 0) {
        // steady state: batches s (buffers 0) and s + U (buffers 1) are in
        // flight; each is refilled with the batch two ahead once consumed
        int s = 0;
        for (; s + 4 * U <= nks; s += 2 * U) {
            mma_batch<T, XF, XT, MT, NTW, U>(acc, w0, x0, inv);
            load_batch<T, XT, MT, NTW, U, false>(w0, x0, wp, xrs, xr, s + 2 * U, nks);
            mma_batch<T, XF, XT, MT, NTW, U>(acc, w1, x1, inv);
            load_batch<T, XT, MT, NTW, U, false>(w1, x1, wp, xrs, xr, s + 3 * U, nks);
        }
        // tail: steps s .. nks-1 (fewer than 4U), the first two batches loaded
        // (unconditional refills here, or one straight-line path per remaining
        // count, measured slower on MI355X)
        mma_batch<T, XF, XT, MT, NTW, U>(acc, w0, x0, inv);
        if (s + 2 * U < nks) load_batch<T, XT, MT, NTW, U, true>(w0, x0, wp, xrs, xr, s + 2 * U, nks);
        if (s + U < nks) mma_batch<T, XF, XT, MT, NTW, U>(acc, w1, x1, inv);
        if (s + 3 * U < nks) load_batch<T, XT, MT, NTW, U, true>(w1, x1, wp, xrs, xr, s + 3 * U, nks);
        if (s + 2 * U < nks) mma_batch<T, XF, XT, MT, NTW, U>(acc, w0, x0, inv);
        if (s + 3 * U < nks) mma_batch<T, XF, XT, MT, NTW, U>(acc, w1, x1, inv);
    }

    if (split) {   // raw partial tiles of this wave, folded by gemm_fold_kernel
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
            if (tile0 + j >= a.n_tiles) break;
            f32x4_t* pp = reinterpret_cast<f32x4_t*>(a.part) + ((size_t)(tile0 + j) * nwt + gw) * MT * 64 + lane;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) pp[mt * 64] = acc[j][mt];
        }
        return;
    }

    // cross-wave reduction in wave order, one tile at a time (LDS holds
    // waves x MT fragments); wave 0 runs the tile's epilogue
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
        if (tile0 + j >= a.n_tiles) break;
        if (j > 0) __syncthreads();   // wave 0 has read the previous tile
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) red[(wave * MT + mt) * 64 + lane] = acc[j][mt];
        __syncthreads();
        if (wave != 0) continue;
        f32x4_t t_acc[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            f32x4_t v = red[mt * 64 + lane];
            for (int w = 1; w < nw; ++w) v += red[(w * MT + mt) * 64 + lane];
            t_acc[mt] = v;
        }
        epilogue<T, EP, MT>(a, tile0 + j, t_acc, ep_in[j < NEP ? j : 0], gnv[j < NEP ? j : 0], c, g);
    }
}

// Split residual GEMM, second pass: one wave per column tile adds the nwt
// waves' partial tiles in wave order (v = p0, then v += p1, p2, ...: the
// single workgroup's LDS reduction) and runs the EP_RESID epilogue on the sum.
template <typename T, int MT>
__global__ void __launch_bounds__(64) gemm_fold_kernel(GemmArgs a, int nwt) {
    const int tile = blockIdx.x, lane = threadIdx.x, c = lane & 15, g = lane >> 4;
    const int M = a.M, n = tile * 16 + c;
    float ep_in[MT][4];
    const f32x4_t* pp = reinterpret_cast<const f32x4_t*>(a.part) + (size_t)tile * nwt * MT * 64 + lane;
    f32x4_t t_acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = 16 * mt + 4 * g + r;
            ep_in[mt][r] = (m < M && n < a.N) ? a.resid[(size_t)m * a.ldy + n] : 0.f;
        }
        f32x4_t v = pp[mt * 64];
        for (int w = 1; w < nwt; ++w) v += pp[(w * MT + mt) * 64];
        t_acc[mt] = v;
    }
    const float gn = n < a.N ? a.gnext[n] : 0.f;
    epilogue<T, EP_RESID, MT>(a, tile, t_acc, ep_in, gn, c, g);
}

template <typename T, int EP, bool XF>
static hipError_t launch_mt(const GemmPlan& p, const GemmArgs& a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    const dim3 grid(p.grid), block(64 * p.waves);
    if (p.waves > (p.ntw > 1 ? 4 : 8)) return hipErrorInvalidValue;
    const bool split = p.ksplit > 1;
    if (split && (EP != EP_RESID || !a.part || a.ksplit != p.ksplit ||
                  p.grid != (a.n_tiles + p.ntw - 1) / p.ntw * p.ksplit))
        return hipErrorInvalidValue;
    if (!split && a.ksplit > 1) return hipErrorInvalidValue;
    auto go = [&](auto kernel) {
        if (ev0) hipExtLaunchKernelGGL(kernel, grid, block, p.lds_bytes, s, ev0, split ? nullptr : ev1, 0, a);
        else hipLaunchKernelGGL(kernel, grid, block, p.lds_bytes, s, a);
    };
    switch (p.mt * 10 + p.ntw) {
        case 11: go(gemm_kernel<T, EP, 1, 1, XF>); break;
        case 21: go(gemm_kernel<T, EP, 2, 1, XF>); break;
        case 31: go(gemm_kernel<T, EP, 3, 1, XF>); break;
        case 41: go(gemm_kernel<T, EP, 4, 1, XF>); break;
        case 22: go(gemm_kernel<T, EP, 2, 2, XF>); break;
        case 24: go(gemm_kernel<T, EP, 2, 4, XF>); break;
        case 34: go(gemm_kernel<T, EP, 3, 4, XF>); break;
        case 44: go(gemm_kernel<T, EP, 4, 4, XF>); break;
        default: return hipErrorInvalidValue;
    }
    if constexpr (EP == EP_RESID && !XF) {
        if (split) {
            const hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
            const int nwt = p.waves * p.ksplit;
            auto fold = [&](auto kernel) {
                if (ev0) hipExtLaunchKernelGGL(kernel, dim3(a.n_tiles), dim3(64), 0, s, nullptr, ev1, 0, a, nwt);
                else hipLaunchKernelGGL(kernel, dim3(a.n_tiles), dim3(64), 0, s, a, nwt);
            };
            switch (p.mt) {
                case 1: fold(gemm_fold_kernel<T, 1>); break;
                case 2: fold(gemm_fold_kernel<T, 2>); break;
                case 3: fold(gemm_fold_kernel<T, 3>); break;
                case 4: fold(gemm_fold_kernel<T, 4>); break;
                default: return hipErrorInvalidValue;
            }
        }
    }
    return hipGetLastError();
}

// RMSNorm-input GEMMs (QKV, gate/up, LM head) read float x o g rows, or those
// rows already normalised and rounded (blocks of more than one row tile); O
// and down read element-type rows (attention output, SwiGLU product).
template <typename T>
static hipError_t launch_t(int ep, const GemmPlan& p, const GemmArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    const bool xf = a.xf != nullptr;
    if (xf && !a.ssq) return hipErrorInvalidValue;
    switch (ep) {
        case EP_STORE:
            return xf ? launch_mt<T, EP_STORE, true>(p, a, s, e0, e1) : launch_mt<T, EP_STORE, false>(p, a, s, e0, e1);
        case EP_QKV: return xf ? launch_mt<T, EP_QKV, true>(p, a, s, e0, e1) : launch_mt<T, EP_QKV, false>(p, a, s, e0, e1);
        case EP_RESID: return xf ? hipErrorInvalidValue : launch_mt<T, EP_RESID, false>(p, a, s, e0, e1);
        case EP_SWIGLU:
            return xf ? launch_mt<T, EP_SWIGLU, true>(p, a, s, e0, e1) : launch_mt<T, EP_SWIGLU, false>(p, a, s, e0, e1);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_gemm(int dtype, int ep, const GemmPlan& p, const GemmArgs& a, hipStream_t s, hipEvent_t ev0,
                       hipEvent_t ev1) {
    if (a.M < 1 || a.M > 64 || p.waves < 1 || p.waves > 16) return hipErrorInvalidValue;
    return dtype == 1 ? launch_t<uint16_t>(ep, p, a, s, ev0, ev1) : launch_t<float>(ep, p, a, s, ev0, ev1);
}

}  // namespace sdsat
