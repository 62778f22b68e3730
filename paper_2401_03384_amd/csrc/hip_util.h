// Device helpers shared by the HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace ce {

typedef uint16_t bf16_t;   // raw bfloat16 bit pattern

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) { return __uint_as_float((uint32_t)v << 16); }

// float32 -> bfloat16, round to nearest even (a NaN stays a NaN): gfx950's
// hardware conversion.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
    const __bf16 h = (__bf16)f;
    bf16_t u;
    __builtin_memcpy(&u, &h, 2);
    return u;
}

// two float32 -> one word of two bfloat16 (lo in the low half), one
// conversion instruction
__device__ __forceinline__ uint32_t pk_bf16(float lo, float hi) {
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    const b2 r = __builtin_convertvector((f2){lo, hi}, b2);
    uint32_t u;
    __builtin_memcpy(&u, &r, 4);
    return u;
}

__device__ __forceinline__ void store(float* p, int64_t i, float v) { p[i] = v; }
__device__ __forceinline__ void store(bf16_t* p, int64_t i, float v) { p[i] = f32_to_bf16(v); }

template <typename T>
__device__ __forceinline__ float load(const T* p, int64_t i) { return to_f32(p[i]); }

// Sum over the 64 lanes of a wavefront (butterfly, same order on every call).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}

}  // namespace ce
