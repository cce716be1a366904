// Device helpers shared by the gfx950 kernels: vector types, bf16 bit
// conversions, wave/block scans.  Wave size is 64 throughout.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace relaxkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

// Round-to-nearest-even float -> bf16 bits (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ int wave_inclusive_scan(int x) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    return x;
}

// Exclusive prefix sum over the block (NT threads, NT % 64 == 0, NT <= 4096).
// `scratch` holds NT/64 ints of LDS.  Returns the exclusive prefix of `v` and
// writes the block total to `total`.  Contains barriers: every thread must call.
template <int NT>
__device__ __forceinline__ int block_exclusive_scan(int v, int* scratch, int& total) {
    constexpr int NW = NT / 64;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int x = wave_inclusive_scan(v);
    if (lane == 63) scratch[w] = x;
    __syncthreads();
    if (w == 0) {
        int t = lane < NW ? scratch[lane] : 0;
        t = wave_inclusive_scan(t);
        if (lane < NW) scratch[lane] = t;
    }
    __syncthreads();
    const int base = w ? scratch[w - 1] : 0;
    total = scratch[NW - 1];
    __syncthreads();
    return base + x - v;
}

template <typename T>
__device__ __forceinline__ T wave_sum(T x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    return x;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
    return x;
}

// Exchange a 32-bit value with the lane 32 positions away (lane ^ 32).
__device__ __forceinline__ float swap_half(float x) { return __shfl_xor(x, 32, 64); }

}  // namespace relaxkv
