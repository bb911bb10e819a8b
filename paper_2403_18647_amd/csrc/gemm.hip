// Skinny weight-streaming GEMM for block decode: Y[M, N] = X[M, K] . W[N, K]^T with
// M = batch * block rows (<= 64) and N, K model dimensions.  At M <= 64 the
// contraction does about M flops per weight byte, far below the matrix-core
// ridge, so the kernel is bound by streaming W from HBM once.  The design:
//
//  * W is pre-packed (launch_pack) into 16-column x 32-k tiles laid out in lane
//    order, so every wave-wide load is one contiguous 1 KiB (bf16) run and each
//    lane's 16 bytes is directly its matrix-core B fragment: no LDS for W.
//  * A workgroup = 4 waves = 4 adjacent column tiles (64 outputs) over one
//    k-chunk.  The chunk of X (normalised and rounded to the matrix-core input
//    type when the prologue is an RMSNorm) is staged once in LDS and shared by
//    the 4 waves.
//  * Split-K over workgroups gives ~1000 workgroups per launch, enough loads in
//    flight on 256 CUs.  Partial tiles go to scratch; the last workgroup of a
//    column group (device-scope counter) sums them in split order, so results
//    are deterministic, and runs the fused epilogue:
//      EP_STORE   float output (LM-head logits)
//      EP_QKV     RoPE on Q and K columns, Q to its buffer, K and V into the
//                 cache slots of the block rows (positions cache_len[b] + r)
//      EP_RESID   residual add into the float residual stream, plus per-tile
//                 sums of squares that the next RMSNorm prologue reduces
//      EP_SWIGLU  silu(gate) * up, rounded to the activation type
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
        dst[e] = (src && k < a.K) ? src[r * a.K + k] : T(0);
    }
}

void launch_pack(const PackArgs& a, hipStream_t s) {
    const size_t total = (size_t)a.n_tiles * a.k_steps * 64;
    const int blocks = (int)((total + 255) / 256);
    if (a.dtype == 1) hipLaunchKernelGGL(pack_kernel<uint16_t>, dim3(blocks), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(pack_kernel<float>, dim3(blocks), dim3(256), 0, s, a);
}

int gemm_groups(int n_tiles) { return (n_tiles + 3) / 4; }

static constexpr int kLdsBudget = 48 * 1024;
static constexpr int kTargetWorkgroups = 1024;

GemmPlan plan_gemm(int dtype, int M, int n_tiles, int k_steps) {
    GemmPlan p;
    p.mt = (M + 15) / 16;
    const int groups = gemm_groups(n_tiles);
    const int esz = dtype == 1 ? 2 : 4;
    int splits = (kTargetWorkgroups + groups - 1) / groups;
    splits = splits < 1 ? 1 : splits;
    const int max_splits = k_steps / 4 > 0 ? k_steps / 4 : 1;
    if (splits > max_splits) splits = max_splits;
    int chunk = (k_steps + splits - 1) / splits;
    // the LDS copy of the X chunk must fit
    const int max_chunk = kLdsBudget / (M * (32 * esz) + 16 * M);
    if (chunk > max_chunk) chunk = max_chunk > 0 ? max_chunk : 1;
    splits = (k_steps + chunk - 1) / chunk;
    p.splits = splits;
    p.chunk_steps = chunk;
    p.grid = groups * splits;
    p.lds_bytes = M * (chunk * 32 * esz + 16);
    return p;
}

size_t gemm_partial_floats(const GemmPlan& p, int n_tiles) {
    if (p.splits <= 1) return 0;
    return (size_t)gemm_groups(n_tiles) * p.splits * 4 * p.mt * 64 * 4;
}

template <typename T, int XS, int EP, int MT>
__global__ void __launch_bounds__(256) gemm_kernel(GemmArgs a) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    T* xs = reinterpret_cast<T*>(smem_raw);
    __shared__ float s_inv[64];
    __shared__ int s_last;

    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int c = lane & 15, g = lane >> 4;
    const int group = blockIdx.x / a.splits, split = blockIdx.x % a.splits;
    const int ks0 = split * a.chunk_steps;
    const int ks1 = min(a.k_steps, ks0 + a.chunk_steps);
    const int nks = ks1 - ks0;
    const int kc = nks * 32;
    const int ldl = kc + 16 / (int)sizeof(T);   // LDS row stride in elements (+16 bytes)
    const int M = a.M;

    // ---- prologue: X chunk -> LDS (rows < M only)
    if (XS == XS_NORM) {
        for (int m = wave; m < M; m += 4) {
            float s = 0.f;
            for (int t = lane; t < a.n_ssq; t += 64) s += a.ssq[(size_t)m * a.n_ssq + t];
            s = wave_sum(s);
            if (lane == 0) s_inv[m] = 1.0f / sqrtf(s / (float)a.K + a.eps);
        }
        __syncthreads();
    }
    const int kbase = ks0 * 32;
    for (int idx = threadIdx.x * 4; idx < M * kc; idx += 256 * 4) {
        const int m = idx / kc, kk = idx - m * kc;
        const int k = kbase + kk;
        T* d = xs + m * ldl + kk;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float v = 0.f;
            if (k + j < a.K) {
                if (XS == XS_ACT) {
                    d[j] = reinterpret_cast<const T*>(a.xa)[(size_t)m * a.ldx + k + j];
                    continue;
                }
                v = a.x[(size_t)m * a.ldx + k + j];
                if (XS == XS_NORM) v = v * s_inv[m] * a.gain[k + j];
            }
            d[j] = to_elem<T>(v);
        }
    }
    __syncthreads();

    // ---- main loop: stream this wave's column tile over the k-chunk
    const int tile = group * 4 + wave;
    const bool tile_ok = tile < a.n_tiles;
    f32x4_t acc[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (tile_ok) {
        const T* wp = reinterpret_cast<const T*>(a.W) + (((size_t)tile * a.k_steps + ks0) * 64 + lane) * 8;
        constexpr int U = 8;
        for (int s = 0; s < nks; s += U) {
            Frag<T> w[U];
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (s + u < nks) w[u] = Frag<T>::load_nt(wp + (size_t)(s + u) * 512);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (s + u < nks) {
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        const int m = 16 * mt + c;
                        Frag<T> xf = m < M ? Frag<T>::load(xs + m * ldl + (s + u) * 32 + 8 * g) : Frag<T>::zero();
                        mma(acc[mt], xf, w[u]);
                    }
                }
            }
        }
    }

    // ---- split-K reduction: last arriving workgroup of the column group finishes
    if (a.splits > 1) {
        f32x4_t* part = reinterpret_cast<f32x4_t*>(a.partial);
        const size_t base = (((size_t)group * a.splits + split) * 4 + wave) * MT * 64;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) part[base + mt * 64 + lane] = acc[mt];
        __threadfence();
        __syncthreads();
        if (threadIdx.x == 0) s_last = atomicAdd(&a.counter[group], 1) == a.splits - 1;
        __syncthreads();
        if (!s_last) return;
        __threadfence();
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int sp = 0; sp < a.splits; ++sp) {
            const size_t b2 = (((size_t)group * a.splits + sp) * 4 + wave) * MT * 64;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc[mt] += part[b2 + mt * 64 + lane];
        }
        if (threadIdx.x == 0) a.counter[group] = 0;
    }
    if (!tile_ok) return;

    // ---- epilogues.  acc[mt][r] = Y[m = 16mt + 4g + r][column c of this tile]
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
                    float* px = a.resid + (size_t)m * a.ldy + n;
                    const float v = *px + acc[mt][r];
                    *px = v;
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
                    u[(size_t)m * a.F + f] = to_elem<T>(gate / (1.0f + expf(-gate)) * up);
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
                const int pos = a.cache_len[b] + row;   // cache slot of this block row
                if (pos >= a.S_max) {                   // the host checks capacity; never write past the cache
                    atomicOr(a.err, 4);
                    continue;
                }
                float out = mine;
                if (sec < 2) {
                    // rotary position: the row's depth in the block (its ancestors
                    // counted by the tree mask; row index for a chain)
                    const int rpos = a.mask ? a.cache_len[b] + __popcll(a.mask[m]) - 1 : pos;
                    const float cs = a.rope_cos[(size_t)rpos * half + pi];
                    const float sn = a.rope_sin[(size_t)rpos * half + pi];
                    out = c < 8 ? mine * cs - other * sn : other * sn + mine * cs;
                }
                if (sec == 0) {
                    reinterpret_cast<T*>(a.qbuf)[((size_t)m * H + h) * Dh + dim] = to_elem<T>(out);
                } else if (sec == 1) {
                    reinterpret_cast<T*>(a.kc)[(((size_t)b * H + h) * a.S_max + pos) * Dh + dim] = to_elem<T>(out);
                } else {
                    const size_t blk = ((size_t)b * H + h) * (a.S_max / 32) + pos / 32;
                    reinterpret_cast<T*>(a.vc)[(blk * Dh + dim) * 32 + vperm(pos & 31)] = to_elem<T>(out);
                }
            }
    }
}

template <typename T, int XS, int EP>
static hipError_t launch_mt(const GemmPlan& p, const GemmArgs& a, hipStream_t s) {
    switch (p.mt) {
        case 1: hipLaunchKernelGGL((gemm_kernel<T, XS, EP, 1>), dim3(p.grid), dim3(256), p.lds_bytes, s, a); break;
        case 2: hipLaunchKernelGGL((gemm_kernel<T, XS, EP, 2>), dim3(p.grid), dim3(256), p.lds_bytes, s, a); break;
        case 3: hipLaunchKernelGGL((gemm_kernel<T, XS, EP, 3>), dim3(p.grid), dim3(256), p.lds_bytes, s, a); break;
        case 4: hipLaunchKernelGGL((gemm_kernel<T, XS, EP, 4>), dim3(p.grid), dim3(256), p.lds_bytes, s, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename T>
static hipError_t launch_t(int xs, int ep, const GemmPlan& p, const GemmArgs& a, hipStream_t s) {
    if (xs == XS_NORM && ep == EP_QKV) return launch_mt<T, XS_NORM, EP_QKV>(p, a, s);
    if (xs == XS_NORM && ep == EP_SWIGLU) return launch_mt<T, XS_NORM, EP_SWIGLU>(p, a, s);
    if (xs == XS_NORM && ep == EP_STORE) return launch_mt<T, XS_NORM, EP_STORE>(p, a, s);
    if (xs == XS_ACT && ep == EP_RESID) return launch_mt<T, XS_ACT, EP_RESID>(p, a, s);
    if (xs == XS_F32 && ep == EP_STORE) return launch_mt<T, XS_F32, EP_STORE>(p, a, s);
    return hipErrorInvalidValue;
}

hipError_t launch_gemm(int dtype, int xs, int ep, const GemmPlan& p, const GemmArgs& a, hipStream_t s) {
    if (a.M < 1 || a.M > 64) return hipErrorInvalidValue;
    return dtype == 1 ? launch_t<uint16_t>(xs, ep, p, a, s) : launch_t<float>(xs, ep, p, a, s);
}

}  // namespace sdsat
