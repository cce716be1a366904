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

// ------------------------------------------------ swizzled LDS tiles (bf16)
//
// Tiles of rows of D bf16 values (D = 64 or 128) filled by 16-byte direct
// global->LDS loads (global_load_lds_dwordx4): one wave-wide load writes 64 x 16
// bytes of consecutive LDS, so tiles are unpadded and each lane picks the
// global chunk that belongs at its slot.  Logical 16-byte chunk c of tile row r
// is stored at chunk c ^ tile_swz<D>(r), which makes
// - MFMA fragment reads (16 consecutive rows, one chunk per row) and
// - transposing reads (4 consecutive rows x 4 chunks per 32 lanes)
// hit distinct bank groups of the 256-byte LDS bank line.
typedef __attribute__((address_space(3))) void lds_void;

template <int D>
__device__ __forceinline__ int tile_swz(int r) {
    static_assert(D == 64 || D == 128, "tile row width");
    if constexpr (D == 128) {
        return ((r & 3) << 2) | ((r >> 2) & 3);              // 16 chunks per row
    } else {
        const int m = (r >> 1) & 7;                          // 8 chunks, 2 rows per bank line
        return ((m & 1) << 2) | (m >> 1);
    }
}

// 16-byte load of global memory into LDS: lane l's chunk lands at lds + 16 l.
// lds must be wave-uniform.
__device__ __forceinline__ void load_lds16(const void* src, void* lds) {
    __builtin_amdgcn_global_load_lds(src, (lds_void*)lds, 16, 0, 0);
}

// Wait until at most N vector-memory loads of this wave are outstanding and
// all its LDS accesses are done, then join the workgroup barrier.  Unlike
// __syncthreads() this does not drain every outstanding load, so direct LDS
// loads of later pipeline stages stay in flight.  Loads complete in order, so
// "at most N outstanding" means every load issued before the last N is done.
template <int N>
__device__ __forceinline__ void wait_loads_barrier() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// The same fills written as inline assembly (M0 = the wave's LDS byte address,
// lane l's bytes land at M0 + size * l).  The compiler does not see an LDS write
// here, so it adds no vector-memory waits before later LDS reads: the caller
// orders each fill and its readers with explicit s_waitcnt vmcnt counts and
// barriers.  Waits the compiler inserts for its own loads stay correct, since
// fills it does not count only make an in-order count wait longer.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(lds_void*)p;
}
// M0 is reserved to the compiler, which ignores it in a clobber list: these
// helpers are only used in kernels that contain no compiler-generated use of
// M0 (on gfx950 LDS instructions do not read it), so the value they leave in
// M0 cannot reach another instruction.
__device__ __forceinline__ void fill_lds16(const void* src, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :: "v"(src), "s"(lds) : "memory", "m0");
}
__device__ __forceinline__ void fill_lds4(const void* src, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
                 :: "v"(src), "s"(lds) : "memory", "m0");
}

}  // namespace relaxkv
