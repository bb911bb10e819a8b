// Row-wise kernels around the matrix-core GEMMs of large blocks (prompt prefill).
//
// A block of more than 64 rows is weight-reuse bound rather than weight-stream
// bound, so its linear layers run as tiled matrix-core GEMMs (prefill_gemm.hip:
// bf16 or float inputs, float accumulation and output) on the caller's
// row-major weights.  The model's other arithmetic stays here and
// rounds exactly where the decode kernels round (the values a bf16 model
// stores): the RMSNorm output bf16(x o g / rms), K and V, the SwiGLU product;
// Q and the residual stream stay float.  Rotary cos / sin come from the same
// table as the decode path.
#include "device.h"
#include "kernels.h"

namespace sdsat {

// h[m][k] = elem(xg[m][k] / rms_m), rms_m = sqrt(sum_t ssq[m][t] / K + eps).
// Workgroup (m, chunk) writes 4 * 256 columns of row m; every thread's four
// values are requested first, then the first wave sums the row's partials in
// the order the decode GEMM does (lane-strided, then a wave butterfly).
template <typename T>
__global__ void __launch_bounds__(256) rms_rows_kernel(const float* xg, int ldxg, const float* ssq, int n_ssq, int K,
                                                       float eps, T* h, int ldh) {
    __shared__ float s_inv;
    const int m = blockIdx.x;
    const int k0 = (blockIdx.y * 256 + threadIdx.x) * 4;
    const float* xr = xg + (size_t)m * ldxg;
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    const bool whole = k0 + 3 < K;   // ldxg and the row start are multiples of 4 floats
    if (whole) {
        const float4 t = *reinterpret_cast<const float4*>(xr + k0);
        v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = k0 + i < K ? xr[k0 + i] : 0.f;
    }
    if (threadIdx.x < 64) {
        float sum = 0.f;
        for (int col = threadIdx.x; col < n_ssq; col += 64) sum += ssq[(size_t)m * n_ssq + col];
        sum = wave_sum(sum);
        if (threadIdx.x == 0) s_inv = 1.0f / sqrtf(sum / (float)K + eps);
    }
    __syncthreads();
    const float inv = s_inv;
    T* hr = h + (size_t)m * ldh;
#pragma unroll
    for (int i = 0; i < 4; ++i)
        if (k0 + i < K) hr[k0 + i] = to_elem<T>(v[i] * inv);
}

// Q, K, V of row m from the float GEMM output c[m][0..3d) (Q | K | V): rotary
// rotation of the pair (i, i + Dh/2) of Q and K at the row's position, Q to
// its float buffer, K and V into the cache slot cache_len[b] + row.  One
// workgroup per (row, head), one thread per pair.
template <typename T>
__global__ void qkv_rope_kernel(const float* c, int ldc, int q, int H, int Dh, const int* cache_len, int S_max,
                                const float* rope, float* qbuf, T* kc, T* vc, int* err) {
    const int m = blockIdx.x, h = blockIdx.y, i = threadIdx.x, half = Dh / 2;
    if (i >= half) return;
    const int b = m / q, row = m - b * q;
    const int pos = cache_len[b] + row;
    if (pos >= S_max) {   // the host checks capacity; never write past the cache
        if (i == 0 && h == 0) atomicOr(err, 4);
        return;
    }
    const int d = H * Dh;
    const float* cr = c + (size_t)m * ldc + h * Dh;
    const float2 csn = *reinterpret_cast<const float2*>(rope + ((size_t)pos * half + i) * 2);
    const float cs = csn.x, sn = csn.y;
    const float q1 = cr[i], q2 = cr[i + half];
    float* qo = qbuf + ((size_t)m * H + h) * Dh;
    qo[i] = q1 * cs - q2 * sn;
    qo[i + half] = q1 * sn + q2 * cs;
    const float k1 = cr[d + i], k2 = cr[d + i + half];
    T* ko = kc + (((size_t)b * H + h) * S_max + pos) * Dh;
    ko[i] = to_elem<T>(k1 * cs - k2 * sn);
    ko[i + half] = to_elem<T>(k1 * sn + k2 * cs);
    const size_t blk = ((size_t)b * H + h) * (S_max / 32) + pos / 32;
    T* vo = vc + blk * Dh * 32 + vperm(pos & 31);
    vo[(size_t)i * 32] = to_elem<T>(cr[2 * d + i]);
    vo[(size_t)(i + half) * 32] = to_elem<T>(cr[2 * d + i + half]);
}

// x[m][n] += y[m][n]; xg[m][n] = x[m][n] * gnext[n]; ssq[m][n/16] = the sum of
// squares over each 16-column group (butterfly in the decode epilogue's order).
__global__ void __launch_bounds__(256) resid_rows_kernel(const float* y, const float* y1, int ldy, int N, float* x,
                                                         int ldx, float* xg, int ldxg, const float* gnext, float* ssq,
                                                         int n_tiles) {
    const int m = blockIdx.y, n = blockIdx.x * blockDim.x + threadIdx.x;
    float ss = 0.f;
    if (n < N) {
        const float yv = y1 ? y[(size_t)m * ldy + n] + y1[(size_t)m * ldy + n] : y[(size_t)m * ldy + n];
        const float v = x[(size_t)m * ldx + n] + yv;
        x[(size_t)m * ldx + n] = v;
        xg[(size_t)m * ldxg + n] = v * gnext[n];
        ss = v * v;
    }
    ss += __shfl_xor(ss, 8, 64);
    ss += __shfl_xor(ss, 4, 64);
    ss += __shfl_xor(ss, 2, 64);
    ss += __shfl_xor(ss, 1, 64);
    if ((n & 15) == 0 && n < N) ssq[(size_t)m * n_tiles + n / 16] = ss;
}

// u[m][f] = elem(silu(g) * up) from the float gate and up GEMM outputs.
template <typename T>
__global__ void __launch_bounds__(256) swiglu_rows_kernel(const float* g, const float* up, int ldg, int F, T* u, int ldu) {
    const int m = blockIdx.y, f = blockIdx.x * blockDim.x + threadIdx.x;
    if (f >= F) return;
    const float gate = g[(size_t)m * ldg + f], v = up[(size_t)m * ldg + f];
    u[(size_t)m * ldu + f] = to_elem<T>(gate / (1.0f + expf(-gate)) * v);
}

hipError_t launch_rms_rows(int dtype, const float* xg, int ldxg, const float* ssq, int n_ssq, int K, float eps, int M,
                           void* h, int ldh, hipStream_t s) {
    if (M < 1) return hipSuccess;
    if (ldxg % 4) return hipErrorInvalidValue;   // float4 row loads
    const dim3 grid(M, (K + 1023) / 1024);
    if (dtype == 1)
        hipLaunchKernelGGL(rms_rows_kernel<uint16_t>, grid, dim3(256), 0, s, xg, ldxg, ssq, n_ssq, K, eps,
                           static_cast<uint16_t*>(h), ldh);
    else
        hipLaunchKernelGGL(rms_rows_kernel<float>, grid, dim3(256), 0, s, xg, ldxg, ssq, n_ssq, K, eps,
                           static_cast<float*>(h), ldh);
    return hipGetLastError();
}

hipError_t launch_qkv_rope(int dtype, const float* c, int ldc, int M, int q, int H, int Dh, const int* cache_len,
                           int S_max, const float* rope, float* qbuf, void* kc, void* vc, int* err, hipStream_t s) {
    if (M < 1) return hipSuccess;
    if (dtype == 1)
        hipLaunchKernelGGL(qkv_rope_kernel<uint16_t>, dim3(M, H), dim3(Dh / 2), 0, s, c, ldc, q, H, Dh, cache_len,
                           S_max, rope, qbuf, static_cast<uint16_t*>(kc), static_cast<uint16_t*>(vc), err);
    else
        hipLaunchKernelGGL(qkv_rope_kernel<float>, dim3(M, H), dim3(Dh / 2), 0, s, c, ldc, q, H, Dh, cache_len, S_max,
                           rope, qbuf, static_cast<float*>(kc), static_cast<float*>(vc), err);
    return hipGetLastError();
}

hipError_t launch_resid_rows(const float* y, const float* y1, int ldy, int M, int N, float* x, int ldx, float* xg,
                             int ldxg, const float* gnext, float* ssq, int n_tiles, hipStream_t s) {
    if (M < 1) return hipSuccess;
    hipLaunchKernelGGL(resid_rows_kernel, dim3((N + 255) / 256, M), dim3(256), 0, s, y, y1, ldy, N, x, ldx, xg, ldxg,
                       gnext, ssq, n_tiles);
    return hipGetLastError();
}

hipError_t launch_swiglu_rows(int dtype, const float* g, const float* up, int ldg, int M, int F, void* u, int ldu,
                              hipStream_t s) {
    if (M < 1) return hipSuccess;
    if (dtype == 1)
        hipLaunchKernelGGL(swiglu_rows_kernel<uint16_t>, dim3((F + 255) / 256, M), dim3(256), 0, s, g, up, ldg, F,
                           static_cast<uint16_t*>(u), ldu);
    else
        hipLaunchKernelGGL(swiglu_rows_kernel<float>, dim3((F + 255) / 256, M), dim3(256), 0, s, g, up, ldg, F,
                           static_cast<float*>(u), ldu);
    return hipGetLastError();
}

}  // namespace sdsat
