// Row-wise kernels around the matrix-core GEMMs of large blocks (prompt prefill).
//
// A block of more than 64 rows is weight-reuse bound rather than weight-stream
// bound, so its linear layers run as tiled matrix-core GEMMs (prefill_gemm.hip:
// bf16 or float inputs, float accumulation and output) on the caller's
// row-major weights.  RoPE with the Q / K / V writes and SwiGLU run in the
// epilogues of those GEMMs; the RMSNorm and the residual stream run here.
// Both round exactly where the decode kernels round (the values a bf16 model
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

// The residual add and the next RMSNorm of a large block in one pass over each
// row: x[m] += y[m] (the sum of a split contraction's parts, in part order), then
// h[m] = elem((x[m] o g) / rms_m).  One workgroup per row; each thread keeps
// its columns' x o g in registers.  The sums of squares are formed per 16-column
// group in the decode residual epilogue's butterfly and reduced in rms_rows'
// order (lane-strided, then a wave butterfly), so h is bitwise what a separate
// residual pass and rms_rows give.
static constexpr int kNormRowThreads = 1024;
static constexpr int kNormRowMaxPer = 8;   // columns per thread: rows of up to 8192
template <typename T>
__global__ void __launch_bounds__(kNormRowThreads) resid_norm_rows_kernel(const float* y, int parts, size_t part_stride,
                                                                          int ldy, int N, float* x, int ldx,
                                                                          const float* g, float eps, T* h, int ldh) {
    constexpr int NT = kNormRowThreads, P = kNormRowMaxPer;
    __shared__ float s_ssq[P * NT / 16];
    __shared__ float s_inv;
    const int m = blockIdx.x, t = threadIdx.x;
    const int nch = (N + NT - 1) / NT;
    // every load first (indices clamped into the row), then the arithmetic
    float yv[P], xv[P], gv[P];
#pragma unroll
    for (int c = 0; c < P; ++c) {
        const int n = min(c * NT + t, N - 1);
        yv[c] = xv[c] = gv[c] = 0.f;
        if (c < nch) {
            float pv[kPrefillMaxSplit];
#pragma unroll
            for (int q = 0; q < kPrefillMaxSplit; ++q)
                pv[q] = q < parts ? y[q * part_stride + (size_t)m * ldy + n] : 0.f;
            yv[c] = pv[0];
#pragma unroll
            for (int q = 1; q < kPrefillMaxSplit; ++q)
                if (q < parts) yv[c] += pv[q];
            xv[c] = x[(size_t)m * ldx + n];
            gv[c] = g[n];
        }
    }
#pragma unroll
    for (int c = 0; c < P; ++c) {
        if (c >= nch) continue;
        const int n = c * NT + t;
        float ss = 0.f;
        if (n < N) {
            const float v = xv[c] + yv[c];
            x[(size_t)m * ldx + n] = v;
            xv[c] = v * gv[c];   // x o g from here on
            ss = v * v;
        }
        ss += __shfl_xor(ss, 8, 64);
        ss += __shfl_xor(ss, 4, 64);
        ss += __shfl_xor(ss, 2, 64);
        ss += __shfl_xor(ss, 1, 64);
        if ((n & 15) == 0 && n < N) s_ssq[n / 16] = ss;
    }
    __syncthreads();
    if (t < 64) {
        const int n_ssq = (N + 15) / 16;
        float sum = 0.f;
        for (int col = t; col < n_ssq; col += 64) sum += s_ssq[col];
        sum = wave_sum(sum);
        if (t == 0) s_inv = 1.0f / sqrtf(sum / (float)N + eps);
    }
    __syncthreads();
    const float inv = s_inv;
    T* hr = h + (size_t)m * ldh;
#pragma unroll
    for (int c = 0; c < P; ++c) {
        const int n = c * NT + t;
        if (c < nch && n < N) hr[n] = to_elem<T>(xv[c] * inv);
    }
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

hipError_t launch_resid_norm_rows(int dtype, const float* y, int parts, size_t part_stride, int ldy, int M, int N,
                                  float* x, int ldx, const float* g, float eps, void* h, int ldh, hipStream_t s) {
    if (M < 1) return hipSuccess;
    if (N < 1 || N > kNormRowMaxPer * kNormRowThreads || parts < 1 || parts > kPrefillMaxSplit) return hipErrorInvalidValue;
    if (dtype == 1)
        hipLaunchKernelGGL(resid_norm_rows_kernel<uint16_t>, dim3(M), dim3(kNormRowThreads), 0, s, y, parts,
                           part_stride, ldy, N, x, ldx, g, eps, static_cast<uint16_t*>(h), ldh);
    else
        hipLaunchKernelGGL(resid_norm_rows_kernel<float>, dim3(M), dim3(kNormRowThreads), 0, s, y, parts, part_stride,
                           ldy, N, x, ldx, g, eps, static_cast<float*>(h), ldh);
    return hipGetLastError();
}

}  // namespace sdsat
