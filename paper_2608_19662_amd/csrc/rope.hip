// RoPE at explicit or resource-local positions, with optional head-major
// cache write (ReCache Sec. 3, "Resource-Wise Attention": resource tokens get
// pos(t_ij) = j; the surrounding context keeps its original positions).
//
// A block handles a few consecutive tokens.  It first evaluates cos / sin of
// pos * theta_f once per (token, frequency) into LDS (fp64 angle reduction,
// then float sincos), then every thread rotates one 8-element chunk pair
// (f .. f+7, f+d/2 .. f+d/2+7) of one head with 16-byte loads and stores, and
// copies the matching V chunks bit for bit.  HBM-bound.
#include "common.hpp"
#include "kernels.hpp"

namespace rc {

namespace {

constexpr int kThreads = 256;

template <typename T>
struct Vec8;  // 8 elements as raw 32-bit words
template <>
struct Vec8<float> {
    u32x4 w[2];
    __device__ __forceinline__ void load(const float* p) {
        w[0] = reinterpret_cast<const u32x4*>(p)[0];
        w[1] = reinterpret_cast<const u32x4*>(p)[1];
    }
    __device__ __forceinline__ void store(float* p) const {
        reinterpret_cast<u32x4*>(p)[0] = w[0];
        reinterpret_cast<u32x4*>(p)[1] = w[1];
    }
    __device__ __forceinline__ float get(int e) const { return __uint_as_float(w[e >> 2][e & 3]); }
    __device__ __forceinline__ void set(const float* v) {
        for (int e = 0; e < 8; ++e) w[e >> 2][e & 3] = __float_as_uint(v[e]);
    }
};
template <>
struct Vec8<uint16_t> {
    u32x4 w;
    __device__ __forceinline__ void load(const uint16_t* p) { w = *reinterpret_cast<const u32x4*>(p); }
    __device__ __forceinline__ void store(uint16_t* p) const { *reinterpret_cast<u32x4*>(p) = w; }
    __device__ __forceinline__ float get(int e) const {
        return bf16_bits_to_f32((w[e >> 1] >> (16 * (e & 1))) & 0xffffu);
    }
    __device__ __forceinline__ void set(const float* v) {
        for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
    }
};

template <typename T>
__global__ __launch_bounds__(kThreads) void rope_kernel(const RopeArgs a) {
    __shared__ float2 cs[kThreads];  // (cos, sin) per (token in block, frequency)
    const int half = a.head_dim / 2;
    const int tpb = kThreads / half;  // tokens per block
    const long t0 = (long)blockIdx.x * tpb;
    {
        const int tk = threadIdx.x / half, f = threadIdx.x % half;
        const long t = t0 + tk;
        float s = 0.f, c = 1.f;
        if (t < a.T) {
            int pos;
            if (a.pos) {
                pos = a.pos[t];
            } else {
                int lo = 0, hi = a.n_res - 1;  // resource r with cu_len[r] <= t < cu_len[r + 1]
                while (lo < hi) {
                    const int mid = (lo + hi + 1) >> 1;
                    if (a.cu_len[mid] <= t) lo = mid; else hi = mid - 1;
                }
                pos = (a.pos_base ? a.pos_base[lo] : 0) + (int)(t - a.cu_len[lo]);
            }
            sincos_rev(rope_revolutions(pos, a.rope.rev[f]), &s, &c);
        }
        cs[threadIdx.x] = make_float2(c, s);
    }
    __syncthreads();
    const int chunks = half / 8;  // chunk pairs per head
    const int units = tpb * a.n_heads * chunks;
    const T* x = static_cast<const T*>(a.x);
    T* y = static_cast<T*>(a.y);
    const T* v = static_cast<const T*>(a.v);
    T* vd = static_cast<T*>(a.v_dst);
    const int d = a.head_dim;
    for (int u = threadIdx.x; u < units; u += kThreads) {
        const int tk = u / (a.n_heads * chunks);
        const int h = (u / chunks) % a.n_heads;
        const int ch = u % chunks;
        const long t = t0 + tk;
        if (t >= a.T) continue;
        const size_t src = ((size_t)t * a.n_heads + h) * d + ch * 8;
        const size_t dst = a.to_cache ? ((size_t)h * a.cache_rows + a.row0 + t) * d + ch * 8 : src;
        Vec8<T> x1, x2;
        x1.load(x + src);
        x2.load(x + src + half);
        float y1[8], y2[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float2 k = cs[tk * half + ch * 8 + e];
            const float a1 = x1.get(e), a2 = x2.get(e);
            // one product rounded, the other fused: written out, so that the
            // rounding does not depend on how the compiler contracts
            y1[e] = fmaf(a1, k.x, -(a2 * k.y));
            y2[e] = fmaf(a2, k.x, a1 * k.y);
        }
        x1.set(y1);
        x2.set(y2);
        x1.store(y + dst);
        x2.store(y + dst + half);
        if (v) {
            // values are copied bit for bit
            Vec8<T> v1, v2;
            v1.load(v + src);
            v2.load(v + src + half);
            v1.store(vd + dst);
            v2.store(vd + dst + half);
        }
    }
}

}  // namespace

hipError_t launch_rope(const RopeArgs& a, hipStream_t stream) {
    if (a.T == 0) return hipSuccess;
    const int tpb = kThreads / (a.head_dim / 2);
    const long blocks = (a.T + tpb - 1) / tpb;
    if (blocks > 0x7fffffffL) return hipErrorInvalidValue;
    if (a.dtype == 0)
        hipLaunchKernelGGL(rope_kernel<float>, dim3((unsigned)blocks), dim3(kThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(rope_kernel<uint16_t>, dim3((unsigned)blocks), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace rc
