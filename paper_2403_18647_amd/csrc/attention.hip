// Block-causal decode attention over the KV cache (the target model's attention,
// run on the q rows of one SDSAT block; tree masks for Section 2.1.2).
//
// For sequence b, head h and block row r (query at position L_b + r):
//   O_r = softmax(Q_r K^T / sqrt(Dh)) V over keys 0..L_b-1 (committed) plus
//   the block rows r may see (0..r, or the rows set in its ancestor mask).
// The block's own K/V rows were written into slots L_b.. by the QKV epilogue.
//
// Work split (flash-decoding): one wave per (b, h, key chunk).  Per 32 keys a
// wave computes the 32 x q score tile S^T = K Q^T on the matrix cores (A = K
// rows straight from the cache, B = Q^T from registers), runs an online
// softmax per query row (query rows live in lanes, keys in registers and lane
// groups), and accumulates O^T = V^T P^T with A = V^T read from the cache's
// key-permuted 32-key blocks (vperm) and B = P^T taken from the score
// registers as they are.  Chunks are merged by the last-arriving wave of each
// (b, h) with a log-sum-exp combine, in chunk order.
#include "device.h"
#include "kernels.h"

namespace sdsat {

static constexpr int kMaxChunks = 32;
static constexpr int kMinChunkKeys = 64;
static constexpr int kTargetWaves = 4096;

AttnPlan plan_attention(int B, int H, int q, int max_len) {
    AttnPlan p;
    const int T = max_len + q;
    int want = kTargetWaves / (B * H);
    want = want < 1 ? 1 : (want > kMaxChunks ? kMaxChunks : want);
    int ck = (T + want - 1) / want;
    ck = (ck + 31) / 32 * 32;
    if (ck < kMinChunkKeys) ck = kMinChunkKeys;
    int n = (T + ck - 1) / ck;
    if (n > kMaxChunks) {   // cannot happen with want <= kMaxChunks, kept as a guard
        ck = ((T + kMaxChunks - 1) / kMaxChunks + 31) / 32 * 32;
        n = (T + ck - 1) / ck;
    }
    p.chunk_keys = ck;
    p.n_chunks = n;
    p.grid = B * H * n;
    return p;
}

// per (b, h, chunk): MT*16 rows x (Dh + 4) floats (unnormalised O, max, sum, 2 pad for 16-byte rows)
size_t attention_partial_floats(int B, int H, int q_max, int head_dim) {
    const int rows = (q_max + 15) / 16 * 16;
    return (size_t)B * H * kMaxChunks * rows * (head_dim + 4);
}

template <typename T, int DH, int MT>
__global__ void __launch_bounds__(64) attn_kernel(AttnArgs a) {
    constexpr int NDS = DH / 32;   // 32-wide steps over the head dimension
    constexpr int NDT = DH / 16;   // 16-row output tiles over the head dimension
    const int lane = threadIdx.x, c = lane & 15, g = lane >> 4;
    const int bh = blockIdx.x / a.n_chunks, chunk = blockIdx.x % a.n_chunks;
    const int b = bh / a.H, h = bh % a.H;
    const int q = a.q;
    const int L = a.cache_len[b];
    const int Tb = L + q;
    if (Tb > a.S_max) {   // the host checks capacity; never read past this sequence's cache
        if (lane == 0 && chunk == 0) atomicOr(a.err, 4);
        return;
    }
    const int n_chunks = (Tb + a.chunk_keys - 1) / a.chunk_keys;
    if (n_chunks > a.n_chunks) {   // launch planned for a shorter cache: flag it, touch nothing
        if (lane == 0 && chunk == 0) atomicOr(a.err, 8);
        return;
    }
    if (chunk >= n_chunks) return;
    const int k_lo = chunk * a.chunk_keys;
    const int k_hi = min(Tb, k_lo + a.chunk_keys);

    const T* qb = reinterpret_cast<const T*>(a.qbuf);
    Frag<T> qf[NDS][MT];
    uint64_t mrow[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int m = 16 * mt + c;
        mrow[mt] = (a.mask && m < q) ? a.mask[(size_t)b * q + m] : 0ull;
#pragma unroll
        for (int ds = 0; ds < NDS; ++ds)
            qf[ds][mt] = m < q ? Frag<T>::load(qb + (((size_t)b * q + m) * a.H + h) * DH + ds * 32 + 8 * g)
                               : Frag<T>::zero();
    }

    const T* kbase = reinterpret_cast<const T*>(a.kc) + ((size_t)b * a.H + h) * a.S_max * DH;
    const T* vbase = reinterpret_cast<const T*>(a.vc) + ((size_t)b * a.H + h) * a.S_max * DH;

    float rmax[MT], rsum[MT];
    f32x4_t o[NDT][MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        rmax[mt] = -INFINITY;
        rsum[mt] = 0.f;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) o[dt][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }

    for (int kb0 = k_lo; kb0 < k_hi; kb0 += 32) {
        // scores: s[kt][mt][r] = S^T[key = kb0 + 16kt + 4g + r][m = 16mt + c]
        Frag<T> kf[2][NDS];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds)
                kf[kt][ds] = Frag<T>::load(kbase + (size_t)(kb0 + 16 * kt + c) * DH + ds * 32 + 8 * g);
        Frag<T> vf[NDT];
        const T* vblk = vbase + (size_t)(kb0 / 32) * DH * 32;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) vf[dt] = Frag<T>::load(vblk + (size_t)(dt * 16 + c) * 32 + 8 * g);

#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            f32x4_t s0 = f32x4_t{0.f, 0.f, 0.f, 0.f}, s1 = s0;
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds) {
                mma(s0, kf[0][ds], qf[ds][mt]);
                mma(s1, kf[1][ds], qf[ds][mt]);
            }
            const int m = 16 * mt + c;
            float sv[8];
            bool vis[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int key = kb0 + (i < 4 ? 4 * g + i : 16 + 4 * g + (i - 4));
                bool v = key < Tb && m < q;
                if (a.mask) v = v && (key < L || ((mrow[mt] >> (key - L)) & 1ull));
                else v = v && key <= L + m;
                vis[i] = v;
                sv[i] = (i < 4 ? s0[i] : s1[i - 4]) * a.scale;
            }
            float bm = -INFINITY;
#pragma unroll
            for (int i = 0; i < 8; ++i) if (vis[i]) bm = fmaxf(bm, sv[i]);
            bm = fmaxf(bm, __shfl_xor(bm, 16, 64));
            bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
            const float nmax = fmaxf(rmax[mt], bm);
            const float alpha = rmax[mt] == -INFINITY ? 0.f : expf(rmax[mt] - nmax);
            float p[8];
            float ps = 0.f;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                p[i] = vis[i] ? expf(sv[i] - nmax) : 0.f;
                ps += p[i];
            }
            rsum[mt] = rsum[mt] * alpha + ps;
            rmax[mt] = nmax;
            const Frag<T> pf = Frag<T>::from_f32(p);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                o[dt][mt] *= alpha;
                mma(o[dt][mt], vf[dt], pf);
            }
        }
    }
    // o[dt][mt][r] = unnormalised O^T[d = 16dt + 4g + r][m = 16mt + c]
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        rsum[mt] += __shfl_xor(rsum[mt], 16, 64);
        rsum[mt] += __shfl_xor(rsum[mt], 32, 64);
    }

    if (n_chunks > 1) {
        const int rows = MT * 16;
        float* part = a.part + ((size_t)bh * kMaxChunks + chunk) * rows * (DH + 4);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int m = 16 * mt + c;
            float* pr = part + (size_t)m * (DH + 4);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
                *reinterpret_cast<f32x4_t*>(pr + 16 * dt + 4 * g) = o[dt][mt];
            if (g == 0) { pr[DH] = rmax[mt]; pr[DH + 1] = rsum[mt]; }
        }
        __threadfence();
        __shared__ int s_last;
        if (lane == 0) s_last = atomicAdd(&a.counter[bh], 1) == n_chunks - 1;
        __syncthreads();
        if (!s_last) return;
        __threadfence();
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int m = 16 * mt + c;
            float gmax = -INFINITY;
            for (int ch = 0; ch < n_chunks; ++ch) {
                const float* pr = a.part + (((size_t)bh * kMaxChunks + ch) * rows + m) * (DH + 4);
                gmax = fmaxf(gmax, pr[DH]);
            }
            float den = 0.f;
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) o[dt][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            for (int ch = 0; ch < n_chunks; ++ch) {
                const float* pr = a.part + (((size_t)bh * kMaxChunks + ch) * rows + m) * (DH + 4);
                const float cm = pr[DH];
                const float w = cm == -INFINITY ? 0.f : expf(cm - gmax);
                den += w * pr[DH + 1];
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt)
                    o[dt][mt] += w * *reinterpret_cast<const f32x4_t*>(pr + 16 * dt + 4 * g);
            }
            rsum[mt] = den;
        }
        if (lane == 0) a.counter[bh] = 0;
    }
    // normalise and store O[b*q + m][h*DH + d]
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int m = 16 * mt + c;
        if (m >= q) continue;
        const float inv = 1.0f / rsum[mt];
        const size_t row = ((size_t)b * q + m) * a.H * DH + (size_t)h * DH;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            const int d = 16 * dt + 4 * g;
            if (a.out_f32) {
                float* po = reinterpret_cast<float*>(a.out) + row + d;
#pragma unroll
                for (int r = 0; r < 4; ++r) po[r] = o[dt][mt][r] * inv;
            } else {
                T* po = reinterpret_cast<T*>(a.out) + row + d;
#pragma unroll
                for (int r = 0; r < 4; ++r) po[r] = to_elem<T>(o[dt][mt][r] * inv);
            }
        }
    }
}

template <typename T, int DH>
static hipError_t launch_dh(const AttnArgs& a, int grid, hipStream_t s) {
    const int mt = (a.q + 15) / 16;
    switch (mt) {
        case 1: hipLaunchKernelGGL((attn_kernel<T, DH, 1>), dim3(grid), dim3(64), 0, s, a); break;
        case 2: hipLaunchKernelGGL((attn_kernel<T, DH, 2>), dim3(grid), dim3(64), 0, s, a); break;
        case 3: hipLaunchKernelGGL((attn_kernel<T, DH, 3>), dim3(grid), dim3(64), 0, s, a); break;
        case 4: hipLaunchKernelGGL((attn_kernel<T, DH, 4>), dim3(grid), dim3(64), 0, s, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_attention(int dtype, int head_dim, const AttnArgs& a, hipStream_t s) {
    const int grid = a.B * a.H * a.n_chunks;
    if (a.q < 1 || a.q > 64 || a.n_chunks > kMaxChunks) return hipErrorInvalidValue;
    if (dtype == 1) {
        if (head_dim == 128) return launch_dh<uint16_t, 128>(a, grid, s);
        if (head_dim == 64) return launch_dh<uint16_t, 64>(a, grid, s);
    } else {
        if (head_dim == 128) return launch_dh<float, 128>(a, grid, s);
        if (head_dim == 64) return launch_dh<float, 64>(a, grid, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace sdsat
