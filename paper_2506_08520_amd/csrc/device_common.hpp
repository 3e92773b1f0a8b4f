// Device-side helpers shared by the HIP kernels: element access for the two
// storage types, rounding to bfloat16, and wavefront reductions (wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nystra {

constexpr float kLog2e = 1.4426950408889634f;

// ---- element access ------------------------------------------------------

struct F32 {
    using T = float;
    static constexpr int bytes = 4;
    __device__ static inline float load(const T *p, int64_t i) { return p[i]; }
    __device__ static inline void store(T *p, int64_t i, float x) { p[i] = x; }
};

// bfloat16 held as raw 16-bit patterns.
__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// Round-to-nearest-even fp32 -> bf16 (NaN kept quiet).
__device__ inline uint16_t f32_to_bf16(float x)
{
    uint32_t u = __float_as_uint(x);
    if ((u & 0x7fffffffu) > 0x7f800000u)
        return uint16_t((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

struct BF16 {
    using T = uint16_t;
    static constexpr int bytes = 2;
    __device__ static inline float load(const T *p, int64_t i) { return bf16_to_f32(p[i]); }
    __device__ static inline void store(T *p, int64_t i, float x) { p[i] = f32_to_bf16(x); }
};

// ---- wavefront reductions (64 lanes) -------------------------------------

__device__ inline float wave_max(float x)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        x = fmaxf(x, __shfl_xor(x, o, 64));
    return x;
}

__device__ inline float wave_sum(float x)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        x += __shfl_xor(x, o, 64);
    return x;
}

// 2^x on the hardware transcendental unit (v_exp_f32).
__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

}  // namespace nystra
