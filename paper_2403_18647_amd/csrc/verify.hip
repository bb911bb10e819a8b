// Verification kernels (Section 2.1.1 Eq. 3 and Section 2.1.2).
//
// One workgroup per logits row (b, j) reduces over the vocabulary; the last
// workgroup of sequence b to finish (device-scope counter) then scans the rows
// for the accepted prefix: m = number of leading j >= 1 with
// drafts[b][j-1] == token[b][j-1].
//
// Greedy: arg-max with ties to the lowest id.
// Nucleus: float64 arithmetic on z = logit / T.  Optional top-k (ties keep
// lower ids) and the top-p threshold are found by radix descent over the
// order-preserving 32-bit keys of the float logits (4 bits per pass, 8
// passes): the threshold is the largest key K with S(K) = sum of e^(z - zmax)
// over kept ids with key >= K at least p * E.  Each pass sums its 16 digits
// through per-thread columns in LDS (one writer per word) and a fixed-order
// reduction.  The token is the smallest id of the nucleus whose ascending-id
// cumulative mass exceeds u * S(K*), with the cumulative sums formed by a
// block-wide prefix scan in id order.  All sums use a fixed reduction order,
// so results are reproducible run to run.
#include "device.h"
#include "kernels.h"

namespace sdsat {

// ---------------------------------------------------------------- helpers
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
    return v > bv || (v == bv && i < bi);
}

template <int NT>
__device__ int block_argmax(const float* row, int V, float* s_val, int* s_idx) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    if ((V & 3) == 0) {
        // all of a round's loads are issued before any is compared
        constexpr int PF = 8;
        const float4* r4 = reinterpret_cast<const float4*>(row);
        const int n4 = V / 4;
        for (int i0 = threadIdx.x; i0 < n4; i0 += NT * PF) {
            float4 v[PF];
#pragma unroll
            for (int p = 0; p < PF; ++p) v[p] = r4[min(i0 + p * NT, n4 - 1)];
#pragma unroll
            for (int p = 0; p < PF; ++p) {
                const int i = i0 + p * NT;
                if (i >= n4) break;
                if (better(v[p].x, 4 * i, bv, bi)) { bv = v[p].x; bi = 4 * i; }
                if (better(v[p].y, 4 * i + 1, bv, bi)) { bv = v[p].y; bi = 4 * i + 1; }
                if (better(v[p].z, 4 * i + 2, bv, bi)) { bv = v[p].z; bi = 4 * i + 2; }
                if (better(v[p].w, 4 * i + 3, bv, bi)) { bv = v[p].w; bi = 4 * i + 3; }
            }
        }
    } else {
        for (int i = threadIdx.x; i < V; i += NT) {
            const float v = row[i];
            if (better(v, i, bv, bi)) { bv = v; bi = i; }
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float ov = __shfl_xor(bv, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) { s_val[wave] = bv; s_idx[wave] = bi; }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < NT / 64; ++w)
            if (better(s_val[w], s_idx[w], bv, bi)) { bv = s_val[w]; bi = s_idx[w]; }
        s_idx[0] = bi == 0x7fffffff ? 0 : bi;
    }
    __syncthreads();
    const int r = s_idx[0];
    __syncthreads();
    return r;
}

// last workgroup of sequence b computes the accepted prefix length
__device__ void finish_sequence(int b, int q, const int* drafts, int drafts_ld, const int* tokens_out,
                                int* n_accept, int* counter) {
    __shared__ int s_last;
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) s_last = atomicAdd(&counter[b], 1) == q - 1;
    __syncthreads();
    if (!s_last || threadIdx.x != 0) return;
    __threadfence();
    int m = 0;
    if (drafts) {
        for (int j = 1; j < q; ++j) {
            if (drafts[(size_t)b * drafts_ld + j - 1] != tokens_out[(size_t)b * q + j - 1]) break;
            m = j;
        }
    }
    if (n_accept) n_accept[b] = m;
    counter[b] = 0;
}

__global__ void __launch_bounds__(1024) verify_greedy_kernel(const float* logits, int q, int V, const int* drafts,
                                                             int drafts_ld, int* tokens_out, int* n_accept,
                                                             int* counter) {
    __shared__ float s_val[16];
    __shared__ int s_idx[16];
    const int row = blockIdx.x, b = row / q;
    const int t = block_argmax<1024>(logits + (size_t)row * V, V, s_val, s_idx);
    if (threadIdx.x == 0) tokens_out[row] = t;
    finish_sequence(b, q, drafts, drafts_ld, tokens_out, n_accept, counter);
}

hipError_t launch_verify_greedy(const float* logits, int B, int q, int V, const int* drafts, int drafts_ld,
                                int* tokens_out, int* n_accept, int* counter, hipStream_t s) {
    hipLaunchKernelGGL(verify_greedy_kernel, dim3(B * q), dim3(1024), 0, s, logits, q, V, drafts, drafts_ld,
                       tokens_out, n_accept, counter);
    return hipGetLastError();
}

// ---------------------------------------------------------------- nucleus
// 1024 threads x 32 contiguous ids (V <= 32768); each thread keeps its ids' keys and float64
// weights in registers and a bit mask (one bit per id) of the kept and nucleus ids.  Longer
// vocabularies go chunk by chunk (sample_row_chunked).
static constexpr int kNT = 1024;
static constexpr int kCPT = 32;
using Bits = uint32_t;
static_assert(kCPT <= 32, "one mask bit per id");
static constexpr int kWaves = kNT / 64;
static constexpr int kBins = 16;    // radix digits of 4 bits
static_assert(kBins % kWaves == 0, "digit totals: each wave sums kBins / kWaves digits");
static constexpr int kArgNT = 1024; // threads of the arg-max-only tree kernel

__device__ __forceinline__ double readlane_d(double v, int lane) {
    const int2 p = __builtin_bit_cast(int2, v);
    return __builtin_bit_cast(double, make_int2(__builtin_amdgcn_readlane(p.x, lane),
                                                __builtin_amdgcn_readlane(p.y, lane)));
}

__device__ __forceinline__ uint32_t order_key(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;   // -0 and +0 compare equal
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_value(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// SplitMix64 (Steele, Lea, Flood 2014): output number n of the generator started at `state`
__device__ __forceinline__ uint64_t splitmix64(uint64_t state, uint64_t n) {
    uint64_t z = state + n * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ double keyed_uniform(uint64_t seed, int b, int pos) {
    const uint64_t c = ((uint64_t)(uint32_t)b << 32) | (uint32_t)pos;
    return (double)(splitmix64(seed, c + 1) >> 11) * (1.0 / 9007199254740992.0);
}

__device__ __forceinline__ double dshfl_xor(double v, int o) {
    int2 p = __builtin_bit_cast(int2, v);
    p.x = __shfl_xor(p.x, o, 64);
    p.y = __shfl_xor(p.y, o, 64);
    return __builtin_bit_cast(double, p);
}

__device__ __forceinline__ double dshfl_up(double v, int o) {
    int2 p = __builtin_bit_cast(int2, v);
    p.x = __shfl_up(p.x, o, 64);
    p.y = __shfl_up(p.y, o, 64);
    return __builtin_bit_cast(double, p);
}

// Sum of NV doubles per thread over the block, fixed order; result in every thread.
template <int NV>
__device__ void block_sum_d(double (&v)[NV], double* s_buf /* [kWaves][NV] */) {
#pragma unroll
    for (int i = 0; i < NV; ++i)
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) v[i] += dshfl_xor(v[i], o);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0)
#pragma unroll
        for (int i = 0; i < NV; ++i) s_buf[wave * NV + i] = v[i];
    __syncthreads();
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        double s = 0.0;
        for (int w = 0; w < kWaves; ++w) s += s_buf[w * NV + i];
        v[i] = s;
    }
    __syncthreads();
}

__device__ int block_sum_i(int v, int* s_buf) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) s_buf[wave] = v;
    __syncthreads();
    int s = 0;
    for (int w = 0; w < kWaves; ++w) s += s_buf[w];
    __syncthreads();
    return s;
}

// exclusive prefix sum of one int per thread, thread order
__device__ int block_exscan_i(int v, int* s_buf) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    int inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(inc, o, 64);
        if (lane >= o) inc += t;
    }
    if (lane == 63) s_buf[wave] = inc;
    __syncthreads();
    int base = 0;
    for (int w = 0; w < wave; ++w) base += s_buf[w];
    __syncthreads();
    return base + inc - v;
}

// exclusive prefix sum of one double per thread, thread order
__device__ double block_exscan_d(double v, double* s_buf) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    double inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const double t = dshfl_up(inc, o);
        if (lane >= o) inc += t;
    }
    if (lane == 63) s_buf[wave] = inc;
    __syncthreads();
    double base = 0.0;
    for (int w = 0; w < wave; ++w) base += s_buf[w];
    __syncthreads();
    return base + (inc - v);
}

__device__ int block_min_i(int v, int* s_buf) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) s_buf[wave] = v;
    __syncthreads();
    int s = s_buf[0];
    for (int w = 1; w < kWaves; ++w) s = min(s, s_buf[w]);
    __syncthreads();
    return s;
}

__device__ int block_max_i(int v, int* s_buf) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) s_buf[wave] = v;
    __syncthreads();
    int s = s_buf[0];
    for (int w = 1; w < kWaves; ++w) s = max(s, s_buf[w]);
    __syncthreads();
    return s;
}

__device__ float block_max_f(float v, float* s_buf) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) s_buf[wave] = v;
    __syncthreads();
    float s = s_buf[0];
    for (int w = 1; w < kWaves; ++w) s = fmaxf(s, s_buf[w]);
    __syncthreads();
    return s;
}

// Radix descent over the order-preserving keys, 4 bits per pass from the top.
// Every thread keeps private per-digit sums of its own ids in LDS (column t of
// hist[digit][thread]), so no atomics are needed and the totals of each digit
// are formed in a fixed order: wave w sums digit w, lane l over threads l,
// l + 64, ... in turn, then a butterfly.  The result is the largest key K whose
// weight sum over kept ids with key >= K reaches `goal` (the lowest key of the
// final range if rounding leaves every sum short of it) and, in *mass, that
// sum.

// One id's weight into the thread's own column of the pass's digit histogram
// (a no-return LDS add: no round trip, and the adds to one word land in
// program order, one writer, so the sums repeat bit for bit).
__device__ __forceinline__ void radix_add(double* hist, uint32_t key, int shift, double w) {
    __hip_atomic_fetch_add(&hist[((key >> shift) & 15u) * kNT + threadIdx.x], w, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ void radix_clear(double* hist) {
#pragma unroll
    for (int v = 0; v < kBins; ++v) hist[v * kNT + threadIdx.x] = 0.0;
}

// After a pass's adds: the digit totals in a fixed order, then the digit whose
// running sum from the top first reaches `goal` (every wave takes the same
// decision); extends `prefix` and the mass above / at it.
__device__ __forceinline__ void radix_pick(const double* hist, double* s_tot, int shift, double goal,
                                           uint32_t& prefix, double& above, double& at) {
    const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
    __syncthreads();
#pragma unroll
    for (int h = 0; h < kBins / kWaves; ++h) {
        const int bin = wave + h * kWaves;
        double sum = 0.0;
#pragma unroll
        for (int j = 0; j < kNT / 64; ++j) sum += hist[bin * kNT + j * 64 + lane];
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) sum += dshfl_xor(sum, o);
        if (lane == 0) s_tot[bin] = sum;
    }
    __syncthreads();
    // lane v holds digit v's total; walk the digits from the top
    const double mine = s_tot[lane & (kBins - 1)];
    double acc = above, before = above;
    int best = 0;
    for (int v = kBins - 1; v >= 0; --v) {
        before = acc;
        acc += readlane_d(mine, v);
        if (acc >= goal) { best = v; break; }
    }
    prefix |= (uint32_t)best << shift;
    above = before;
    at = acc;
}

// w_of(i) gives id id0 + i's weight (0 for ids outside the kept set).
template <typename WeightFn>
__device__ __forceinline__ uint32_t radix_threshold(const uint32_t (&keys)[kCPT], Bits kept, WeightFn w_of, double goal,
                                    double* hist, double* s_tot, double* mass) {
    uint32_t prefix = 0;
    double above = 0.0, at = 0.0;
#pragma unroll 1
    for (int shift = 28; shift >= 0; shift -= 4) {
        const uint32_t hi = shift == 28 ? 0u : 0xFFFFFFFFu << (shift + 4);
        radix_clear(hist);
#pragma unroll
        for (int i = 0; i < kCPT; ++i) {
            if (!((kept >> i) & 1u)) continue;
            const uint32_t key = keys[i];
            if ((key & hi) != (prefix & hi)) continue;
            radix_add(hist, key, shift, w_of(i));
        }
        radix_pick(hist, s_tot, shift, goal, prefix, above, at);
    }
    *mass = at;
    return prefix;
}

// ---- top-k of at most kSmallK ids: candidate list
static constexpr int kSmallK = 64;

__device__ __forceinline__ uint32_t shfl_xor_any(uint32_t v, int o) { return (uint32_t)__shfl_xor((int)v, o, 64); }
__device__ __forceinline__ uint64_t shfl_xor_any(uint64_t v, int o) {
    return ((uint64_t)shfl_xor_any((uint32_t)(v >> 32), o) << 32) | shfl_xor_any((uint32_t)v, o);
}
__device__ __forceinline__ uint32_t readlane_u(uint32_t v, int lane) {
    return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}

// Bitonic sort of one value per lane across the wave, descending (lane 0 holds the largest).
template <typename U>
__device__ __forceinline__ U wave_sort_desc(U v) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int size = 2; size <= 64; size <<= 1)
#pragma unroll
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            const U o = shfl_xor_any(v, stride);
            const bool keep_max = ((lane & stride) == 0) == ((lane & size) == 0);
            v = keep_max ? (v > o ? v : o) : (v < o ? v : o);
        }
    return v;
}

// Top-k with k <= kSmallK (ties keep lower ids), then top-p and the inverse
// CDF, on a candidate list.  The k-th largest of the 1024 threads' maxima is at
// most the row's k-th largest key (k distinct ids reach it), so every id at or
// above it is a candidate and the kept ids are among them; it is found by
// sorting each wave's maxima and a k-round tournament over the waves' sorted
// lists.  The candidates are gathered in
// id order; wave 0 sorts them by (key descending, id ascending), keeps the
// first k and finishes in float64: the total mass and the threshold in that
// order, the inverse CDF over the nucleus in ascending id order.  Returns false
// (nothing decided) when more than kSmallK ids reach the bound.
__device__ __forceinline__ bool sample_small_topk(const uint32_t (&keys)[kCPT], Bits kept, int id0, double T,
                                                  double p, int top_k, double u, int* s_i, int* out) {
    __shared__ uint32_t s_top[kWaves * kSmallK];   // each wave's k largest thread maxima, descending
    __shared__ uint32_t s_bound;
    __shared__ uint32_t s_ck[kSmallK];
    __shared__ int s_cid[kSmallK];
    __shared__ double s_ne[kSmallK];
    __shared__ int s_nid[kSmallK];
    __shared__ int s_tok;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    uint32_t tmax = 0;
#pragma unroll
    for (int i = 0; i < kCPT; ++i) if ((kept >> i) & 1u) tmax = max(tmax, keys[i]);
    const uint32_t srt = wave_sort_desc(tmax);
    if (lane < top_k) s_top[wave * kSmallK + lane] = srt;
    __syncthreads();
    if (wave == 0) {
        // k rounds of a tournament over the waves' lists: the k-th largest thread maximum
        int pos = 0;
        uint32_t head = lane < kWaves ? s_top[lane * kSmallK] : 0u;
        uint32_t last = 0;
        for (int r = 0; r < top_k; ++r) {
            uint64_t c = lane < kWaves ? ((uint64_t)head << 32) | (uint32_t)(63 - lane) : 0ull;
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) {
                const uint64_t t = shfl_xor_any(c, o);
                c = c > t ? c : t;
            }
            last = (uint32_t)(c >> 32);
            if (lane == 63 - (int)(uint32_t)c) {   // the list that held it moves on
                ++pos;
                head = pos < top_k ? s_top[lane * kSmallK + pos] : 0u;
            }
        }
        if (lane == 0) s_bound = last;
    }
    __syncthreads();
    const uint32_t bound = s_bound;
    int cnt = 0;
#pragma unroll
    for (int i = 0; i < kCPT; ++i) cnt += ((kept >> i) & 1u) && keys[i] >= bound;
    const int C = block_sum_i(cnt, s_i);   // >= top_k
    if (C > kSmallK) return false;
    int slot = block_exscan_i(cnt, s_i);
#pragma unroll
    for (int i = 0; i < kCPT; ++i)
        if (((kept >> i) & 1u) && keys[i] >= bound) { s_ck[slot] = keys[i]; s_cid[slot] = id0 + i; ++slot; }
    __syncthreads();
    if (wave == 0) {
        // (key descending, id ascending) as the composite (key, ~id) sorted descending;
        // lanes past C hold 0 and sort last
        uint64_t v = lane < C ? ((uint64_t)s_ck[lane] << 32) | (uint32_t)~(uint32_t)s_cid[lane] : 0ull;
        v = wave_sort_desc(v);
        const uint32_t key = (uint32_t)(v >> 32);
        const int id = (int)~(uint32_t)v;
        const int k = top_k;
        const double zmax = (double)key_value(readlane_u(key, 0)) / T;
        const double e = lane < k ? exp((double)key_value(key) / T - zmax) : 0.0;
        double tot = 0.0;
        for (int j = 0; j < k; ++j) tot += readlane_d(e, j);
        const double pE = (p < 1.0 ? p : 1.0) * tot;
        // threshold: the first group of equal keys (in descending order) at which the mass
        // from the top reaches p * E; the whole group is in the nucleus
        double acc = 0.0, mass = -1.0;
        int nstar = k;
        for (int j = 0; j < k; ++j) {
            acc += readlane_d(e, j);
            const bool group_end = j + 1 == k || readlane_u(key, min(j + 1, 63)) != readlane_u(key, j);
            if (group_end && acc >= pE) { nstar = j + 1; mass = acc; break; }
        }
        if (mass < 0.0) mass = acc;   // rounding left every sum short of p * E: all k
        // the nucleus in ascending id order, then the inverse CDF
        if (lane < nstar) {
            int rank = 0;
            for (int i = 0; i < nstar; ++i) rank += (int)__builtin_amdgcn_readlane(id, i) < id;
            s_nid[rank] = id;
            s_ne[rank] = e;
        }
        const double target = u * mass;
        double cum = 0.0;
        int tok = -1;
        for (int r = 0; r < nstar; ++r) {
            cum += s_ne[r];
            if (cum > target) { tok = s_nid[r]; break; }
        }
        if (tok < 0) tok = s_nid[nstar - 1];
        if (lane == 0) s_tok = tok;
    }
    __syncthreads();
    *out = s_tok;
    return true;
}

// ids id0 .. id0+31 of a row as order-preserving keys (ids past V: -inf)
__device__ __forceinline__ void load_keys(const float* row, int V, int id0, uint32_t (&keys)[kCPT]) {
#pragma unroll
    for (int i = 0; i < kCPT; i += 4) {
        if (id0 + i + 3 < V && (V & 3) == 0) {
            const float4 v = *reinterpret_cast<const float4*>(row + id0 + i);
            keys[i] = order_key(v.x); keys[i + 1] = order_key(v.y);
            keys[i + 2] = order_key(v.z); keys[i + 3] = order_key(v.w);
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) keys[i + j] = order_key(id0 + i + j < V ? row[id0 + i + j] : -INFINITY);
        }
    }
}

__device__ __forceinline__ int sample_row(const float* row, int V, double T, double p, int top_k, double u) {
    __shared__ double s_hist[kBins * kNT];   // 128 KiB: per-thread digit columns
    __shared__ double s_tot[kBins];          // digit totals (read by every thread after the last pass)
    __shared__ double s_d[kWaves];
    __shared__ int s_i[kWaves];
    __shared__ float s_f[kWaves];
    const int id0 = threadIdx.x * kCPT;
    // ids id0 .. id0+31 as order-preserving keys (the float is recovered from the key where needed)
    uint32_t keys[kCPT];
    load_keys(row, V, id0, keys);
    Bits kept = 0;   // bit i: id0+i is kept by top-k
#pragma unroll
    for (int i = 0; i < kCPT; ++i) if (id0 + i < V) kept |= 1u << i;

    // k up to 3/4 of the list: the candidates (about k) rarely overflow it
    if (top_k > 0 && top_k <= kSmallK * 3 / 4 && top_k < V) {
        int tok;
        if (sample_small_topk(keys, kept, id0, T, p, top_k, u, s_i, &tok)) return tok;
    }
    if (top_k > 0 && top_k < V) {
        // largest key Kk with count(key >= Kk) >= top_k (counts are exact in double)
        double cnt;
        const uint32_t Kk = radix_threshold(keys, kept, [&](int) { return 1.0; }, (double)top_k, s_hist, s_tot, &cnt);
        int gt = 0, eq = 0;
#pragma unroll
        for (int i = 0; i < kCPT; ++i) {
            if (!((kept >> i) & 1u)) continue;
            gt += keys[i] > Kk;
            eq += keys[i] == Kk;
        }
        const int need = top_k - block_sum_i(gt, s_i);
        int rank = block_exscan_i(eq, s_i);
        Bits nk = 0;
#pragma unroll
        for (int i = 0; i < kCPT; ++i) {
            if (!((kept >> i) & 1u)) continue;
            if (keys[i] > Kk) nk |= 1u << i;
            else if (keys[i] == Kk) { if (rank < need) nk |= 1u << i; ++rank; }
        }
        kept = nk;
    }

    uint32_t kmax = 0;
#pragma unroll
    for (int i = 0; i < kCPT; ++i) if ((kept >> i) & 1u) kmax = max(kmax, keys[i]);
    const float lmax = block_max_f(key_value(kmax), s_f);
    const double zmax = (double)lmax / T;
    double e[kCPT];
    double tot[1] = {0.0};
#pragma unroll
    for (int i = 0; i < kCPT; ++i) {
        e[i] = ((kept >> i) & 1u) ? exp((double)key_value(keys[i]) / T - zmax) : 0.0;
        tot[0] += e[i];
    }
    block_sum_d<1>(tot, s_d);
    const double pE = (p < 1.0 ? p : 1.0) * tot[0];

    // top-p threshold key and the mass of the nucleus
    double mass;
    const uint32_t Kstar = radix_threshold(keys, kept, [&](int i) { return e[i]; }, pE, s_hist, s_tot, &mass);

    // inverse CDF over the nucleus in ascending id order
    double loc = 0.0;
    Bits inN = 0;
#pragma unroll
    for (int i = 0; i < kCPT; ++i)
        if (((kept >> i) & 1u) && keys[i] >= Kstar) { inN |= 1u << i; loc += e[i]; }
    const double pre = block_exscan_d(loc, s_d);
    const double target = u * mass;
    int cand = 0x7fffffff;
    int last = -1;
    double cum = pre;
#pragma unroll
    for (int i = 0; i < kCPT; ++i) {
        if (!((inN >> i) & 1u)) continue;
        cum += e[i];
        last = id0 + i;
        if (cand == 0x7fffffff && cum > target) cand = id0 + i;
    }
    cand = block_min_i(cand, s_i);
    if (cand == 0x7fffffff) cand = block_max_i(last, s_i);
    return cand;
}

// ---- vocabularies past one chunk of kNT * kCPT ids
// Chunk c covers ids [c * kChunk, (c + 1) * kChunk); thread t holds ids
// c * kChunk + 32 t + i of each.  Only the kept bits stay resident (in LDS);
// every pass reloads a chunk's keys from the row (from L2 after the first) and
// recomputes their float64 weights, so registers do not grow with V.  The
// chunks are visited in order, so each lower-ids-first rule (top-k ties, the
// inverse CDF) keeps ascending id order.  Same decisions as sample_row: top-k
// by a count threshold, top-p by a weight threshold, inverse CDF.
static constexpr int kChunk = kNT * kCPT;
static constexpr int kMaxChunks = 4;   // V <= 131072

__device__ __forceinline__ int sample_row_chunked(const float* row, int V, double T, double p, int top_k, double u) {
    __shared__ double s_hist[kBins * kNT];     // 128 KiB: per-thread digit columns
    __shared__ Bits s_kept[kMaxChunks * kNT];  // thread t's kept bits of chunk c at [c * kNT + t]
    __shared__ double s_tot[kBins];
    __shared__ double s_d[kWaves];
    __shared__ int s_i[kWaves];
    __shared__ float s_f[kWaves];
    const int t = threadIdx.x, tb = t * kCPT;
    const int nch = (V + kChunk - 1) / kChunk;
    uint32_t keys[kCPT];
    for (int c = 0; c < nch; ++c) {   // each thread reads back only its own words
        Bits kb = 0;
#pragma unroll
        for (int i = 0; i < kCPT; ++i) if (c * kChunk + tb + i < V) kb |= 1u << i;
        s_kept[c * kNT + t] = kb;
    }
    if (top_k > 0 && top_k < V) {
        // largest key Kk with count(key >= Kk) >= top_k (counts are exact in double)
        uint32_t Kk = 0;
        double above = 0.0, at = 0.0;
#pragma unroll 1
        for (int shift = 28; shift >= 0; shift -= 4) {
            const uint32_t hi = shift == 28 ? 0u : 0xFFFFFFFFu << (shift + 4);
            radix_clear(s_hist);
            for (int c = 0; c < nch; ++c) {
                load_keys(row, V, c * kChunk + tb, keys);
                const Bits kb = s_kept[c * kNT + t];
#pragma unroll
                for (int i = 0; i < kCPT; ++i)
                    if (((kb >> i) & 1u) && (keys[i] & hi) == (Kk & hi)) radix_add(s_hist, keys[i], shift, 1.0);
            }
            radix_pick(s_hist, s_tot, shift, (double)top_k, Kk, above, at);
        }
        int gt = 0;
        for (int c = 0; c < nch; ++c) {
            load_keys(row, V, c * kChunk + tb, keys);
            const Bits kb = s_kept[c * kNT + t];
#pragma unroll
            for (int i = 0; i < kCPT; ++i) gt += ((kb >> i) & 1u) && keys[i] > Kk;
        }
        const int need = top_k - block_sum_i(gt, s_i);
        int base = 0;   // ids at Kk in earlier chunks
        for (int c = 0; c < nch; ++c) {
            load_keys(row, V, c * kChunk + tb, keys);
            const Bits kb = s_kept[c * kNT + t];
            int eq = 0;
#pragma unroll
            for (int i = 0; i < kCPT; ++i) eq += ((kb >> i) & 1u) && keys[i] == Kk;
            int rank = base + block_exscan_i(eq, s_i);
            base += block_sum_i(eq, s_i);
            Bits nk = 0;
#pragma unroll
            for (int i = 0; i < kCPT; ++i) {
                if (!((kb >> i) & 1u)) continue;
                if (keys[i] > Kk) nk |= 1u << i;
                else if (keys[i] == Kk) { if (rank < need) nk |= 1u << i; ++rank; }
            }
            s_kept[c * kNT + t] = nk;
        }
    }
    uint32_t kmax = 0;
    for (int c = 0; c < nch; ++c) {
        load_keys(row, V, c * kChunk + tb, keys);
        const Bits kb = s_kept[c * kNT + t];
#pragma unroll
        for (int i = 0; i < kCPT; ++i) if ((kb >> i) & 1u) kmax = max(kmax, keys[i]);
    }
    const float lmax = block_max_f(key_value(kmax), s_f);
    const double zmax = (double)lmax / T;
    double tot[1] = {0.0};
    for (int c = 0; c < nch; ++c) {
        load_keys(row, V, c * kChunk + tb, keys);
        const Bits kb = s_kept[c * kNT + t];
#pragma unroll
        for (int i = 0; i < kCPT; ++i)
            if ((kb >> i) & 1u) tot[0] += exp((double)key_value(keys[i]) / T - zmax);
    }
    block_sum_d<1>(tot, s_d);
    const double pE = (p < 1.0 ? p : 1.0) * tot[0];

    // top-p threshold key and the mass of the nucleus
    uint32_t Ks = 0;
    double above = 0.0, mass = 0.0;
#pragma unroll 1
    for (int shift = 28; shift >= 0; shift -= 4) {
        const uint32_t hi = shift == 28 ? 0u : 0xFFFFFFFFu << (shift + 4);
        radix_clear(s_hist);
        for (int c = 0; c < nch; ++c) {
            load_keys(row, V, c * kChunk + tb, keys);
            const Bits kb = s_kept[c * kNT + t];
#pragma unroll
            for (int i = 0; i < kCPT; ++i)
                if (((kb >> i) & 1u) && (keys[i] & hi) == (Ks & hi))
                    radix_add(s_hist, keys[i], shift, exp((double)key_value(keys[i]) / T - zmax));
        }
        radix_pick(s_hist, s_tot, shift, pE, Ks, above, mass);
    }

    // inverse CDF over the nucleus in ascending id order, chunk by chunk
    const double target = u * mass;
    double run = 0.0;   // nucleus mass of the earlier chunks
    int last = -1;
    for (int c = 0; c < nch; ++c) {
        load_keys(row, V, c * kChunk + tb, keys);
        const Bits kb = s_kept[c * kNT + t];
        double e[kCPT];
        double loc[1] = {0.0};
        Bits inN = 0;
#pragma unroll
        for (int i = 0; i < kCPT; ++i) {
            e[i] = 0.0;
            if (((kb >> i) & 1u) && keys[i] >= Ks) {
                e[i] = exp((double)key_value(keys[i]) / T - zmax);
                loc[0] += e[i];
                inN |= 1u << i;
            }
        }
        double cum = run + block_exscan_d(loc[0], s_d);
        int cand = 0x7fffffff;
#pragma unroll
        for (int i = 0; i < kCPT; ++i) {
            if (!((inN >> i) & 1u)) continue;
            cum += e[i];
            last = c * kChunk + tb + i;
            if (cand == 0x7fffffff && cum > target) cand = c * kChunk + tb + i;
        }
        cand = block_min_i(cand, s_i);
        if (cand != 0x7fffffff) return cand;
        block_sum_d<1>(loc, s_d);
        run += loc[0];
    }
    return block_max_i(last, s_i);
}

template <bool CHUNKED>
__global__ void __launch_bounds__(kNT) verify_nucleus_kernel(const float* logits, int q, int V, const int* drafts,
                                                             int drafts_ld, float temperature, float top_p,
                                                             int top_k, uint64_t seed, const int* pos0,
                                                             const int* row_depth, int* tokens_out, int* n_accept,
                                                             int* counter) {
    __shared__ float s_val[kWaves];
    __shared__ int s_idx[kWaves];
    const int row = blockIdx.x, b = row / q, j = row % q;
    const float* lg = logits + (size_t)row * V;
    // row_depth (a draft tree): every row is sampled, keyed by the position of its node's next token
    const bool sample = temperature > 0.f && (drafts != nullptr || row_depth != nullptr || j == 0);
    int t;
    if (sample) {
        const double u = keyed_uniform(seed, b, pos0[b] + (row_depth ? row_depth[row] : j));
        if constexpr (CHUNKED) t = sample_row_chunked(lg, V, (double)temperature, (double)top_p, top_k, u);
        else t = sample_row(lg, V, (double)temperature, (double)top_p, top_k, u);
    } else {
        t = block_argmax<kNT>(lg, V, s_val, s_idx);
    }
    if (threadIdx.x == 0) tokens_out[row] = t;
    if (drafts || n_accept) finish_sequence(b, q, drafts, drafts_ld, tokens_out, n_accept, counter);
}

hipError_t launch_verify_nucleus(const float* logits, int B, int q, int V, const int* drafts, int drafts_ld,
                                 float temperature, float top_p, int top_k, uint64_t seed, const int* pos0,
                                 int* tokens_out, int* n_accept, int* counter, hipStream_t s, const int* row_depth) {
    if (V > kChunk * kMaxChunks || (row_depth && drafts)) return hipErrorInvalidValue;
    auto kern = V > kChunk ? verify_nucleus_kernel<true> : verify_nucleus_kernel<false>;
    hipLaunchKernelGGL(kern, dim3(B * q), dim3(kNT), 0, s, logits, q, V, drafts, drafts_ld, temperature, top_p, top_k,
                       seed, pos0, row_depth, tokens_out, n_accept, counter);
    return hipGetLastError();
}

// ---------------------------------------------------------------- draft tree (Section 2.1.2)
// Tree of width w over draft step 1's adaptive rows: depth j holds the w
// largest logits of row j (ties to the lower id).  Block rows: 0 the root t1,
// 1..k the chain of each depth's first candidate (parent: the row above),
// then depth by depth the other candidates, leaves under the chain node one
// level up (row k + 1 + (j - 1)(w - 1) + i - 1 for candidate i of depth j).

// arg-max of a row over the ids not in excl[0..n_excl) (ties to the lower id)
template <int NT>
__device__ int block_argmax_excl(const float* row, int V, const int* excl, int n_excl, float* s_val, int* s_idx) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    for (int i = threadIdx.x; i < V; i += NT) {
        bool skip = false;
        for (int e = 0; e < n_excl; ++e) skip |= excl[e] == i;
        if (skip) continue;
        const float v = row[i];
        if (better(v, i, bv, bi)) { bv = v; bi = i; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float ov = __shfl_xor(bv, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) { s_val[wave] = bv; s_idx[wave] = bi; }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < NT / 64; ++w)
            if (better(s_val[w], s_idx[w], bv, bi)) { bv = s_val[w]; bi = s_idx[w]; }
        s_idx[0] = bi == 0x7fffffff ? 0 : bi;
    }
    __syncthreads();
    const int r = s_idx[0];
    __syncthreads();
    return r;
}

// One workgroup per (sequence, depth j): the depth's candidates, their block
// rows' tokens, ancestor masks (bit r: block row r is visible) and depths;
// depth 1 also writes the root.
__global__ void __launch_bounds__(kArgNT) tree_build_kernel(const float* logits1, int q1, int V, const int* out1, int k,
                                                         int w, int q2, int* tok2, uint64_t* mask2, int* depth2) {
    __shared__ float s_val[kArgNT / 64];
    __shared__ int s_idx[kArgNT / 64];
    __shared__ int s_ch[kMaxTreeWidth];
    const int b = blockIdx.x, j = blockIdx.y + 1;
    const float* row = logits1 + ((size_t)b * q1 + j) * V;
    for (int p = 0; p < w; ++p) {
        const int t = block_argmax_excl<kArgNT>(row, V, s_ch, p, s_val, s_idx);
        if (threadIdx.x == 0) s_ch[p] = t;
        __syncthreads();
    }
    if (threadIdx.x != 0) return;
    int* tk = tok2 + (size_t)b * q2;
    uint64_t* mk = mask2 + (size_t)b * q2;
    int* dp = depth2 + (size_t)b * q2;
    const uint64_t up = (1ull << j) - 1;   // the root and chain rows 1..j-1
    tk[j] = s_ch[0];
    mk[j] = up | (1ull << j);
    dp[j] = j;
    for (int i = 1; i < w; ++i) {
        const int r = k + 1 + (j - 1) * (w - 1) + (i - 1);
        tk[r] = s_ch[i];
        mk[r] = up | (1ull << r);
        dp[r] = j;
    }
    if (j == 1) {
        tk[0] = out1[(size_t)b * q1];
        mk[0] = 1ull;
        dp[0] = 0;
    }
}

// Longest confirmed branch, one thread per sequence: from the root, emit the
// target's token at the node (targets[node]) and descend into the child that
// carries it (chain child first, then the leaves in row order), else stop.
// Writes the emitted tokens, m, the branch's block rows (for the gathered
// commit), the next pending token and the rows to commit (0 when inactive).
__global__ void tree_walk_kernel(int B, int q2, int k, int w, const int* tok2, const int* targets, const int* active,
                                 int* emitted, int* n_accept, int* rows, int* pending, int* n_commit) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    const int* tk = tok2 + (size_t)b * q2;
    const int* tg = targets + (size_t)b * q2;
    int node = 0, m = 0;
    rows[(size_t)b * q2] = 0;
    for (;;) {
        const int t = tg[node];
        emitted[(size_t)b * q2 + m] = t;
        int nxt = -1;
        if (node < k) {   // a chain node (the root is depth 0); leaves have no children
            if (tk[node + 1] == t) {
                nxt = node + 1;
            } else {
                for (int i = 0; i < w - 1; ++i) {
                    const int r = k + 1 + node * (w - 1) + i;
                    if (tk[r] == t) { nxt = r; break; }
                }
            }
        }
        if (nxt < 0) break;
        ++m;
        rows[(size_t)b * q2 + m] = nxt;
        node = nxt;
    }
    n_accept[b] = m;
    const bool act = active[b] != 0;
    if (act) pending[b] = tg[node];
    n_commit[b] = act ? m + 1 : 0;
}

hipError_t launch_tree_build(const float* logits1, int B, int q1, int V, const int* out1, int k, int w, int q2,
                             int* tok2, uint64_t* mask2, int* depth2, hipStream_t s) {
    if (k < 1 || w < 1 || w > kMaxTreeWidth || q2 != 1 + k * w || q2 > 64) return hipErrorInvalidValue;
    hipLaunchKernelGGL(tree_build_kernel, dim3(B, k), dim3(kArgNT), 0, s, logits1, q1, V, out1, k, w, q2, tok2, mask2,
                       depth2);
    return hipGetLastError();
}

hipError_t launch_tree_walk(int B, int q2, int k, int w, const int* tok2, const int* targets, const int* active,
                            int* emitted, int* n_accept, int* rows, int* pending, int* n_commit, hipStream_t s) {
    hipLaunchKernelGGL(tree_walk_kernel, dim3((B + 63) / 64), dim3(64), 0, s, B, q2, k, w, tok2, targets, active,
                       emitted, n_accept, rows, pending, n_commit);
    return hipGetLastError();
}

}  // namespace sdsat
