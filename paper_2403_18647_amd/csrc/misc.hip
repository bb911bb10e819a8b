// Small kernels of the block forward and the decode loop: embedding gather,
// KV-cache commit (length bump, or in-place gather for tree-shaped blocks),
// cache writes for tests, and the device-side bookkeeping of a draft/verify
// loop (Section 2.1: draft step 1 keeps one row, verification keeps m+1).
#include "device.h"
#include "kernels.h"

namespace sdsat {

// x[m] = E[token[m]] as float, x o g (g: the first RMSNorm's gain, the QKV
// GEMM's input) and per-16-column sums of squares of x (the partials its
// RMSNorm scale reduces).  One thread per 16-column tile, vector loads and
// stores.  Out-of-range ids set *err and read row 0.
template <typename T>
__global__ void embed_kernel(const T* emb, int n_rows, int d, const int* tokens, float* x, float* xg,
                             const float* gain, int ldxg, float* ssq, int n_ssq, int* err) {
    const int m = blockIdx.y;
    const int t = blockIdx.x * blockDim.x + threadIdx.x;   // 16-column tile
    int tok = tokens[m];
    if (tok < 0 || tok >= n_rows) {
        if (t == 0) atomicOr(err, 1);
        tok = 0;
    }
    if (t >= n_ssq) return;
    const T* src = emb + (size_t)tok * d + 16 * t;
    float v[16];
    if ((d & 15) == 0) {
        const Frag<T> a = Frag<T>::load(src), b = Frag<T>::load(src + 8);
#pragma unroll
        for (int j = 0; j < 8; ++j) { v[j] = a.get(j); v[8 + j] = b.get(j); }
    } else {
#pragma unroll
        for (int j = 0; j < 16; ++j) v[j] = 16 * t + j < d ? to_f32<T>(src[j]) : 0.f;
    }
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) ss += v[j] * v[j];
    if ((d & 15) == 0 && (ldxg & 3) == 0 && ((uintptr_t)gain & 15) == 0) {
        f32x4_t* xo = reinterpret_cast<f32x4_t*>(x + (size_t)m * d + 16 * t);
        f32x4_t* go = reinterpret_cast<f32x4_t*>(xg + (size_t)m * ldxg + 16 * t);
        const f32x4_t* gi = reinterpret_cast<const f32x4_t*>(gain + 16 * t);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const f32x4_t e = f32x4_t{v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]};
            xo[i] = e;
            go[i] = e * gi[i];
        }
    } else {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int k = 16 * t + j;
            if (k < d) {
                x[(size_t)m * d + k] = v[j];
                xg[(size_t)m * ldxg + k] = v[j] * gain[k];
            }
        }
    }
    ssq[(size_t)m * n_ssq + t] = ss;
}

hipError_t launch_embed(int dtype, const void* embed, int n_rows_emb, int d, const int* tokens, int M,
                        float* x, float* xg, const float* gain, int ldxg, float* ssq, int n_ssq, int* err,
                        hipStream_t s) {
    if (dtype == 1)
        hipLaunchKernelGGL(embed_kernel<uint16_t>, dim3((n_ssq + 63) / 64, M), dim3(64), 0, s,
                           (const uint16_t*)embed, n_rows_emb, d, tokens, x, xg, gain, ldxg, ssq, n_ssq, err);
    else
        hipLaunchKernelGGL(embed_kernel<float>, dim3((n_ssq + 63) / 64, M), dim3(64), 0, s, (const float*)embed,
                           n_rows_emb, d, tokens, x, xg, gain, ldxg, ssq, n_ssq, err);
    return hipGetLastError();
}

// float rows [rows][cols] -> element rows [rows][ld], zero in columns cols..ld-1
template <typename T>
__global__ void to_elem_rows_kernel(const float* src, int rows, int cols, T* dst, int ld) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (size_t)rows * ld) return;
    const int r = (int)(i / ld), c = (int)(i % ld);
    dst[i] = to_elem<T>(c < cols ? src[(size_t)r * cols + c] : 0.f);
}

hipError_t launch_to_elem_rows(int dtype, const float* src, int rows, int cols, void* dst, int ld, hipStream_t s) {
    const size_t n = (size_t)rows * ld;
    const int blocks = (int)((n + 255) / 256);
    if (blocks == 0) return hipSuccess;
    if (dtype == 1)
        hipLaunchKernelGGL(to_elem_rows_kernel<uint16_t>, dim3(blocks), dim3(256), 0, s, src, rows, cols,
                           (uint16_t*)dst, ld);
    else
        hipLaunchKernelGGL(to_elem_rows_kernel<float>, dim3(blocks), dim3(256), 0, s, src, rows, cols, (float*)dst,
                           ld);
    return hipGetLastError();
}

// K/V rows [B][n][H][Dh] float -> cache slots pos[b*n + i]
template <typename T>
__global__ void kv_write_kernel(T* kc, T* vc, int B, int n, int H, int Dh, int S_max, const float* k,
                                const float* v, const int* pos) {
    const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t total = (size_t)B * n * H * Dh;
    if (idx >= total) return;
    const int d = (int)(idx % Dh);
    const int h = (int)((idx / Dh) % H);
    const int i = (int)((idx / ((size_t)Dh * H)) % n);
    const int b = (int)(idx / ((size_t)Dh * H * n));
    const int p = pos[(size_t)b * n + i];
    if (p < 0 || p >= S_max) return;
    kc[(((size_t)b * H + h) * S_max + p) * Dh + d] = to_elem<T>(k[idx]);
    const size_t blk = ((size_t)b * H + h) * (S_max / 32) + p / 32;
    vc[(blk * Dh + d) * 32 + vperm(p & 31)] = to_elem<T>(v[idx]);
}

hipError_t launch_kv_write(int dtype, void* kc, void* vc, int B, int n, int H, int Dh, int S_max,
                           const float* k, const float* v, const int* pos, hipStream_t s) {
    const size_t total = (size_t)B * n * H * Dh;
    const int blocks = (int)((total + 255) / 256);
    if (blocks == 0) return hipSuccess;
    if (dtype == 1)
        hipLaunchKernelGGL(kv_write_kernel<uint16_t>, dim3(blocks), dim3(256), 0, s, (uint16_t*)kc, (uint16_t*)vc,
                           B, n, H, Dh, S_max, k, v, pos);
    else
        hipLaunchKernelGGL(kv_write_kernel<float>, dim3(blocks), dim3(256), 0, s, (float*)kc, (float*)vc, B, n, H,
                           Dh, S_max, k, v, pos);
    return hipGetLastError();
}

template <typename T>
__global__ void to_elem_kernel(const float* src, T* dst, size_t n) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) dst[i] = to_elem<T>(src[i]);
}

hipError_t launch_to_elem(int dtype, const float* src, void* dst, size_t n, hipStream_t s) {
    const int blocks = (int)((n + 255) / 256);
    if (blocks == 0) return hipSuccess;
    if (dtype == 1) hipLaunchKernelGGL(to_elem_kernel<uint16_t>, dim3(blocks), dim3(256), 0, s, src, (uint16_t*)dst, n);
    else hipLaunchKernelGGL(to_elem_kernel<float>, dim3(blocks), dim3(256), 0, s, src, (float*)dst, n);
    return hipGetLastError();
}

// cache_len[b] += n[b], kept within [0, S_max] (an out-of-range n sets err bit 4)
__global__ void commit_kernel(int* cache_len, int B, const int* n_commit, int S_max, int* err) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    const int v = cache_len[b] + n_commit[b];
    if (v < 0 || v > S_max) {
        atomicOr(err, 4);
        cache_len[b] = v < 0 ? 0 : S_max;
    } else {
        cache_len[b] = v;
    }
}

hipError_t launch_commit(int* cache_len, int B, const int* n_commit, int S_max, int* err, hipStream_t s) {
    hipLaunchKernelGGL(commit_kernel, dim3((B + 63) / 64), dim3(64), 0, s, cache_len, B, n_commit, S_max, err);
    return hipGetLastError();
}

// Tree case: move block rows rows[b][j] (strictly ascending, rows[b][j] >= j)
// to slot L + j.  Walking j upwards never overwrites a row still to be read.
// One thread per (layer, b, h, d); the length bump is a separate launch.
template <typename T>
__global__ void gather_kernel(T* kc, T* vc, size_t layer_stride, int n_layers, int B, int H, int Dh, int S_max,
                              const int* cache_len, const int* n_commit, const int* rows, int q, int* err) {
    const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t total = (size_t)n_layers * B * H * Dh;
    if (idx >= total) return;
    const int d = (int)(idx % Dh);
    const int h = (int)((idx / Dh) % H);
    const int b = (int)((idx / ((size_t)Dh * H)) % B);
    const int layer = (int)(idx / ((size_t)Dh * H * B));
    const int L = cache_len[b];
    const int n = n_commit[b];
    T* K = kc + layer * layer_stride + ((size_t)b * H + h) * S_max * Dh;
    T* V = vc + layer * layer_stride + ((size_t)b * H + h) * S_max * Dh;
    int prev = -1;
    for (int j = 0; j < n; ++j) {
        const int r = rows[(size_t)b * q + j];
        if (r <= prev || r < j || r >= q || L + r >= S_max) {
            if (d == 0 && h == 0 && layer == 0) atomicOr(err, 2);
            return;
        }
        prev = r;
        if (r == j) continue;
        const int src = L + r, dst = L + j;
        K[(size_t)dst * Dh + d] = K[(size_t)src * Dh + d];
        V[((size_t)(dst / 32) * Dh + d) * 32 + vperm(dst & 31)] = V[((size_t)(src / 32) * Dh + d) * 32 + vperm(src & 31)];
    }
}

hipError_t launch_commit_gather(int dtype, void* kc, void* vc, size_t layer_stride_elems, int n_layers, int B,
                                int H, int Dh, int S_max, const int* cache_len, const int* n_commit,
                                const int* rows, int q, int* err, hipStream_t s) {
    const size_t total = (size_t)n_layers * B * H * Dh;
    const int blocks = (int)((total + 255) / 256);
    if (dtype == 1)
        hipLaunchKernelGGL(gather_kernel<uint16_t>, dim3(blocks), dim3(256), 0, s, (uint16_t*)kc, (uint16_t*)vc,
                           layer_stride_elems, n_layers, B, H, Dh, S_max, cache_len, n_commit, rows, q, err);
    else
        hipLaunchKernelGGL(gather_kernel<float>, dim3(blocks), dim3(256), 0, s, (float*)kc, (float*)vc,
                           layer_stride_elems, n_layers, B, H, Dh, S_max, cache_len, n_commit, rows, q, err);
    return hipGetLastError();
}

__global__ void set_len_kernel(int* cache_len, int B, const int* vals, int value) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b < B) cache_len[b] = vals ? vals[b] : value;
}

hipError_t launch_set_len(int* cache_len, int B, const int* vals_or_null, int value, hipStream_t s) {
    hipLaunchKernelGGL(set_len_kernel, dim3((B + 63) / 64), dim3(64), 0, s, cache_len, B, vals_or_null, value);
    return hipGetLastError();
}

__global__ void fill_i32_kernel(int* p, size_t n, int value) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = value;
}

hipError_t launch_fill_i32(int* p, size_t n, int value, hipStream_t s) {
    const int blocks = (int)((n + 255) / 256);
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(fill_i32_kernel, dim3(blocks), dim3(256), 0, s, p, n, value);
    return hipGetLastError();
}

__global__ void rope_table_kernel(const double* inv_freq, int S, int half, float* rope) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (size_t)S * half) return;
    const int pos = (int)(i / half), p = (int)(i % half);
    double sd, cd;
    sincos((double)pos * inv_freq[p], &sd, &cd);
    rope[2 * i] = (float)cd;
    rope[2 * i + 1] = (float)sd;
}

// Read-only stream for measuring the device's achievable HBM read rate: workgroup g reads bytes
// [16 KiB g, 16 KiB (g + 1)), its four waves interleaved 1 KiB at a time with all four of a wave's
// 16-byte nontemporal loads in flight (many small workgroups measured fastest on MI355X).
__global__ void __launch_bounds__(256) stream_read_kernel(const u32x4_t* __restrict__ src, size_t n16) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const size_t base = (size_t)blockIdx.x * 1024 + lane;
    u32x4_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const size_t i = base + (size_t)(wave + 4 * u) * 64;
        v[u] = i < n16 ? __builtin_nontemporal_load(src + i) : u32x4_t{0, 0, 0, 0};
    }
    uint32_t acc = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) acc ^= v[u].x ^ v[u].w;
    asm volatile("" ::"v"(acc));   // keeps the loads; nothing is written
}

hipError_t launch_stream_read(const void* src, size_t bytes, hipStream_t s) {
    const size_t n16 = bytes / 16;
    if (n16 == 0) return hipSuccess;
    hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)((n16 + 1023) / 1024)), dim3(256), 0, s,
                       static_cast<const u32x4_t*>(src), n16);
    return hipGetLastError();
}

hipError_t launch_rope_table(const double* inv_freq, int S, int half, float* rope, hipStream_t s) {
    const size_t n = (size_t)S * half;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, inv_freq, S, half, rope);
    return hipGetLastError();
}

// draft step 1 block: [pending_b, a_1..a_k]
__global__ void build_draft1_kernel(const int* pending, const int* adaptive, int B, int k, int* tokens) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= B * (k + 1)) return;
    const int b = i / (k + 1), j = i % (k + 1);
    tokens[i] = j == 0 ? pending[b] : adaptive[j - 1];
}

hipError_t launch_build_draft1(const int* pending, const int* adaptive, int B, int k, int* tokens, hipStream_t s) {
    const int n = B * (k + 1);
    hipLaunchKernelGGL(build_draft1_kernel, dim3((n + 63) / 64), dim3(64), 0, s, pending, adaptive, B, k, tokens);
    return hipGetLastError();
}

// after verification: active sequences commit m+1 rows and take o_m as the
// next pending token; finished ones commit nothing.
__global__ void loop_commit_kernel(int* cache_len, int B, int q, const int* active, const int* n_accept,
                                   const int* tokens2, int* pending, int* n_commit_out) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    const int m = n_accept[b];
    const int n = active[b] ? m + 1 : 0;
    n_commit_out[b] = n;
    if (n) {
        cache_len[b] += n;
        pending[b] = tokens2[(size_t)b * q + m];
    }
}

hipError_t launch_loop_commit(int* cache_len, int B, int q, const int* active, const int* n_accept,
                              const int* tokens2, int* pending, int* n_commit_out, hipStream_t s) {
    hipLaunchKernelGGL(loop_commit_kernel, dim3((B + 63) / 64), dim3(64), 0, s, cache_len, B, q, active, n_accept,
                       tokens2, pending, n_commit_out);
    return hipGetLastError();
}

// After a loop's verification: its record [m, t1, emitted 0..k] for the host,
// and the sequence's progress (a loop emits m + 2 tokens: draft step 1's token
// and verified rows 0..m); a sequence stays active while it has emitted fewer
// than max_new, the rule the host applies when it replays the records.
__global__ void loop_record_kernel(int* rec, int B, int q1, int q2, int k, int max_new, const int* out1,
                                   const int* out2, const int* n_accept, int* active, int* produced) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    int* r = rec + (size_t)b * kLoopRecCols;
    const int m = n_accept[b];
    r[0] = m;
    r[1] = out1[(size_t)b * q1];
    for (int j = 0; j <= k; ++j) r[2 + j] = out2[(size_t)b * q2 + j];
    if (active[b]) {
        produced[b] += m + 2;
        active[b] = produced[b] < max_new;
    }
}

hipError_t launch_loop_record(int* rec, int B, int q1, int q2, int k, int max_new, const int* out1, const int* out2,
                              const int* n_accept, int* active, int* produced, hipStream_t s) {
    if (k + 3 > kLoopRecCols) return hipErrorInvalidValue;
    hipLaunchKernelGGL(loop_record_kernel, dim3((B + 63) / 64), dim3(64), 0, s, rec, B, q1, q2, k, max_new, out1, out2,
                       n_accept, active, produced);
    return hipGetLastError();
}

__global__ void pos0_kernel(const int* cache_len, int B, int offset, int* pos0) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b < B) pos0[b] = cache_len[b] + offset;
}

hipError_t launch_pos0(const int* cache_len, int B, int offset, int* pos0, hipStream_t s) {
    hipLaunchKernelGGL(pos0_kernel, dim3((B + 63) / 64), dim3(64), 0, s, cache_len, B, offset, pos0);
    return hipGetLastError();
}

}  // namespace sdsat
