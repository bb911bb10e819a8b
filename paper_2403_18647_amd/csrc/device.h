// Device-side helpers shared by the SDSAT kernels (gfx950 / CDNA4).
//
// Element types: a template parameter T is either `float` (fp32 models) or
// `uint16_t` holding bf16 bit patterns (bf16 models).  Matrix-core operands are
// "fragments" of 8 consecutive elements per lane: lane l of a wave covers
// row/column (l % 16) and the 8 contraction indices 8*(l/16) .. 8*(l/16)+7 of a
// 32-wide contraction step.  A and B operands use the same index sets, so
// v_mfma_f32_16x16x32_bf16 (one instruction) or eight v_mfma_f32_16x16x4_f32
// (one per element) accumulate the full 32-term dot products into a 16x16 tile
// whose lane l holds column (l % 16), rows 4*(l/16) .. 4*(l/16)+3.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sdsat {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two floats to a packed bf16 pair (low half = a), round to nearest even: one
// v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{a, b}), bf16x2_t));
}

// Round to nearest even.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) { return (uint16_t)f32x2_to_bf16x2(f, 0.f); }

template <typename T> struct Frag;

template <> struct Frag<uint16_t> {
    using elem = uint16_t;
    u32x4_t v;
    __device__ __forceinline__ static Frag zero() { Frag f; f.v = u32x4_t{0u, 0u, 0u, 0u}; return f; }
    __device__ __forceinline__ static Frag load(const uint16_t* p) { Frag f; f.v = *reinterpret_cast<const u32x4_t*>(p); return f; }
    __device__ __forceinline__ static Frag load_nt(const uint16_t* p) {
        Frag f; f.v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p)); return f;
    }
    __device__ __forceinline__ void store(uint16_t* p) const { *reinterpret_cast<u32x4_t*>(p) = v; }
    __device__ __forceinline__ float get(int j) const {   // element j as float
        const uint32_t w = v[j >> 1];
        return __uint_as_float((j & 1) ? (w & 0xFFFF0000u) : (w << 16));
    }
    // 8 floats rounded to bf16
    __device__ __forceinline__ static Frag from_f32(const float* x) {
        Frag f;
        f.v.x = f32x2_to_bf16x2(x[0], x[1]);
        f.v.y = f32x2_to_bf16x2(x[2], x[3]);
        f.v.z = f32x2_to_bf16x2(x[4], x[5]);
        f.v.w = f32x2_to_bf16x2(x[6], x[7]);
        return f;
    }
};

template <> struct Frag<float> {
    using elem = float;
    f32x4_t lo, hi;
    __device__ __forceinline__ static Frag zero() {
        Frag f; f.lo = f32x4_t{0.f, 0.f, 0.f, 0.f}; f.hi = f.lo; return f;
    }
    __device__ __forceinline__ static Frag load(const float* p) {
        Frag f; f.lo = reinterpret_cast<const f32x4_t*>(p)[0]; f.hi = reinterpret_cast<const f32x4_t*>(p)[1]; return f;
    }
    __device__ __forceinline__ static Frag load_nt(const float* p) {
        Frag f;
        f.lo = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(p));
        f.hi = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(p) + 1);
        return f;
    }
    __device__ __forceinline__ void store(float* p) const {
        reinterpret_cast<f32x4_t*>(p)[0] = lo; reinterpret_cast<f32x4_t*>(p)[1] = hi;
    }
    __device__ __forceinline__ float get(int j) const { return j < 4 ? lo[j] : hi[j - 4]; }
    __device__ __forceinline__ static Frag from_f32(const float* x) {
        Frag f; f.lo = f32x4_t{x[0], x[1], x[2], x[3]}; f.hi = f32x4_t{x[4], x[5], x[6], x[7]}; return f;
    }
};

// Buffer resource over [p, p + bytes): loads through it take a 32-bit lane
// offset (VGPR) plus a wave-uniform one (SGPR), and lanes whose offset lies
// past the end read zeros without touching memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

template <typename T>
__device__ __forceinline__ Frag<T> buf_frag(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    Frag<T> f;
    if constexpr (sizeof(T) == 2) {
        f.v = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
    } else {
        f.lo = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
        f.hi = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, voff + 16, soff, 0));
    }
    return f;
}

// acc += A(16 x 32) * B(32 x 16) with the fragment convention above.
__device__ __forceinline__ void mma(f32x4_t& acc, const Frag<uint16_t>& a, const Frag<uint16_t>& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a.v),
                                                  __builtin_bit_cast(bf16x8_t, b.v), acc, 0, 0, 0);
}

__device__ __forceinline__ void mma(f32x4_t& acc, const Frag<float>& a, const Frag<float>& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.x, b.lo.x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.y, b.lo.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.z, b.lo.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.w, b.lo.w, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.x, b.hi.x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.y, b.hi.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.z, b.hi.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.w, b.hi.w, acc, 0, 0, 0);
}

template <typename T> __device__ __forceinline__ T to_elem(float x);
template <> __device__ __forceinline__ float to_elem<float>(float x) { return x; }
template <> __device__ __forceinline__ uint16_t to_elem<uint16_t>(float x) { return f32_to_bf16(x); }

template <typename T> __device__ __forceinline__ float to_f32(T x);
template <> __device__ __forceinline__ float to_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ float to_f32<uint16_t>(uint16_t x) { return bf16_to_f32(x); }

// Position of key kb (0..31) inside a 32-key block of the V cache.  Block
// positions 8g..8g+7 hold keys {4g..4g+3, 16+4g..16+4g+3}: the keys a lane of
// lane-group g holds after the score tile, so P^T needs no shuffle.
__device__ __forceinline__ int vperm(int kb) {
    return kb < 16 ? ((kb >> 2) << 3) + (kb & 3) : (((kb - 16) >> 2) << 3) + 4 + ((kb - 16) & 3);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

}  // namespace sdsat
