// Shared device helpers for the gfx950 kernels: bf16 bit handling, RoPE angle
// reduction and wave-level utilities.  Host-side code never includes device
// intrinsics from here except through the kernels' launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kMaxHalfDim = 64;  // head_dim <= 128

// theta_i / (2 pi) for i < head_dim / 2, computed on the host in fp64.
struct RopeRev {
    double rev[kMaxHalfDim];
};

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// Round-to-nearest-even pack of two floats into one dword of two bf16
// (low half = a).  gfx950 has a native instruction for this.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    f32x2 x = {a, b};
    bf16x2 y = __builtin_convertvector(x, bf16x2);
    return __builtin_bit_cast(uint32_t, y);
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float a) {
    return (uint16_t)(pack_bf16x2(a, 0.0f) & 0xffffu);
}

// Angle pos * theta_i reduced to revolutions in [-0.5, 0.5]: the product and
// the reduction are done in fp64, so the float result is accurate to ~1e-16
// revolutions whatever the position.
__device__ __forceinline__ float rope_revolutions(int pos, double rev_i) {
    double a = (double)pos * rev_i;
    a -= rint(a);
    return (float)a;
}

// cos / sin of 2 pi r for r in [-0.5, 0.5] revolutions, accurate to a few
// float ulps (libm-quality sincosf on a reduced argument).
__device__ __forceinline__ void sincos_rev(float r, float* s, float* c) {
    sincosf(r * 6.28318530717958647692f, s, c);
}

// Same with the hardware transcendental unit (v_sin_f32 / v_cos_f32 take
// revolutions).  Used where the rotated value is rounded to bf16 afterwards.
__device__ __forceinline__ void sincos_rev_fast(float r, float* s, float* c) {
    *s = __builtin_amdgcn_sinf(r);
    *c = __builtin_amdgcn_cosf(r);
}

// Combine the values of lanes l and l ^ 32 with one v_permlane32_swap.  Fed
// the same register twice, the swap leaves {own value, partner value} in its
// two results in every lane, so max / sum of the pair do not depend on which
// result holds which.
__device__ __forceinline__ float pair_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float pair_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float wave_max(float x) {
    for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
    return x;
}

__device__ __forceinline__ float wave_sum(float x) {
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

// Exclusive prefix sum of `part` over the threads of an NW-wave block, in
// thread order, and the block total: lane shuffles inside each wave, then
// the NW wave totals through `wave_tot` (LDS, NW ints).  One barrier; every
// thread of the block must call it.
template <int NW>
__device__ __forceinline__ int block_exclusive_scan(int part, int* wave_tot, int* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int incl = part;
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
    }
    if (lane == 63) wave_tot[wave] = incl;
    __syncthreads();
    int before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        const int t = wave_tot[w];
        if (w < wave) before += t;
        tot += t;
    }
    *total = tot;
    return before + incl - part;
}

__device__ __forceinline__ int block4_exclusive_scan(int part, int* wave_tot, int* total) {
    return block_exclusive_scan<4>(part, wave_tot, total);
}

}  // namespace rc
