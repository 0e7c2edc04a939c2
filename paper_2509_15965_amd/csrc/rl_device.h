// rl_device.h -- device-side helpers for the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rl {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16 bits, round to nearest even (NaN stays a quiet NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return 0x7FC0u;
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

// Model-dtype element access.
// silu(g) * u for bf16-stored activations: hardware exponential and
// reciprocal (a few fp32 ulp; the value is rounded to bf16 right after).
__device__ __forceinline__ float swiglu_bf16(float g, float u) {
    return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
}
// The same for fp32 storage: IEEE division and the accurate exponential.
__device__ __forceinline__ float swiglu_f32(float g, float u) {
    return g / (1.0f + expf(-g)) * u;
}
template <typename T> __device__ __forceinline__ float swiglu(float g, float u);
template <> __device__ __forceinline__ float swiglu<uint16_t>(float g, float u) { return swiglu_bf16(g, u); }
template <> __device__ __forceinline__ float swiglu<float>(float g, float u) { return swiglu_f32(g, u); }

template <typename T> struct Elem;
template <> struct Elem<float> {
    static __device__ __forceinline__ float load(const float* p, size_t i) { return p[i]; }
    static __device__ __forceinline__ void store(float* p, size_t i, float v) { p[i] = v; }
};
template <> struct Elem<uint16_t> {
    static __device__ __forceinline__ float load(const uint16_t* p, size_t i) { return bf16_to_f32(p[i]); }
    static __device__ __forceinline__ void store(uint16_t* p, size_t i, float v) { p[i] = f32_to_bf16(v); }
};

// 16-byte global load (p must be 16-byte aligned).
__device__ __forceinline__ u32x4 ld16(const void* p) {
    return *reinterpret_cast<const u32x4*>(p);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// D = A . B + C for one 16x16x32 bf16 tile (fp32 accumulate).
// Lane l supplies A[l % 16][k-group l / 16] and B[k-group l / 16][l % 16]
// (8 k values each, paired element by element) and receives
// D[4 * (l / 16) + e][l % 16] in element e.
__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

typedef float f32x16 __attribute__((ext_vector_type(16)));

// D = A . B + C for one 32x32x16 bf16 tile (fp32 accumulate).
// Lane l supplies A[l % 32][8 (l / 32) + j] and B[8 (l / 32) + j][l % 32]
// (j = 0..7) and receives D[8 (e / 4) + 4 (l / 32) + e % 4][l % 32] in
// element e (0..15).  One wave per SIMD issuing these keeps the matrix core
// close to its peak, unlike the 16x16x32 form.
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float wave_max(float v) {
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ __forceinline__ float wave_sum(float v) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

}  // namespace rl
