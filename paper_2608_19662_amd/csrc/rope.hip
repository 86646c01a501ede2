// RoPE at explicit or resource-local positions, with optional head-major
// cache write (ReCache Sec. 3, "Resource-Wise Attention": resource tokens get
// pos(t_ij) = j; the surrounding context keeps its original positions).
//
// One thread per (token, frequency f): it evaluates cos / sin of pos*theta_f
// once (fp64 angle reduction, then float sincos) and applies them to element
// pair (f, f + d/2) of every head of the token.  HBM-bound; the access
// pattern reads and writes contiguous half-rows per head.
#include "common.hpp"
#include "kernels.hpp"

namespace rc {

namespace {

template <typename T>
__device__ __forceinline__ float ld(const T* p, size_t i);
template <>
__device__ __forceinline__ float ld<float>(const float* p, size_t i) { return p[i]; }
template <>
__device__ __forceinline__ float ld<uint16_t>(const uint16_t* p, size_t i) {
    return bf16_bits_to_f32(p[i]);
}
template <typename T>
__device__ __forceinline__ void st(T* p, size_t i, float x);
template <>
__device__ __forceinline__ void st<float>(float* p, size_t i, float x) { p[i] = x; }
template <>
__device__ __forceinline__ void st<uint16_t>(uint16_t* p, size_t i, float x) {
    p[i] = f32_to_bf16_bits(x);
}

template <typename T>
__global__ __launch_bounds__(256) void rope_kernel(const RopeArgs a) {
    const int half = a.head_dim / 2;
    const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
    const long t = idx / half;
    const int f = (int)(idx % half);
    if (t >= a.T) return;
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
    float s, c;
    sincos_rev(rope_revolutions(pos, a.rope.rev[f]), &s, &c);
    const T* x = static_cast<const T*>(a.x);
    T* y = static_cast<T*>(a.y);
    const T* v = static_cast<const T*>(a.v);
    T* vd = static_cast<T*>(a.v_dst);
    const int d = a.head_dim;
    for (int h = 0; h < a.n_heads; ++h) {
        const size_t src = ((size_t)t * a.n_heads + h) * d;
        const size_t dst = a.to_cache ? ((size_t)h * a.cache_rows + a.row0 + t) * d : src;
        const float x1 = ld(x, src + f), x2 = ld(x, src + f + half);
        st(y, dst + f, x1 * c - x2 * s);
        st(y, dst + f + half, x2 * c + x1 * s);
        if (v) {
            // values are copied bit for bit
            vd[dst + f] = v[src + f];
            vd[dst + f + half] = v[src + f + half];
        }
    }
}

}  // namespace

hipError_t launch_rope(const RopeArgs& a, hipStream_t stream) {
    const long n = (long)a.T * (a.head_dim / 2);
    if (n == 0) return hipSuccess;
    const long blocks = (n + 255) / 256;
    if (blocks > 0x7fffffffL) return hipErrorInvalidValue;
    if (a.dtype == 0)
        hipLaunchKernelGGL(rope_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL(rope_kernel<uint16_t>, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace rc
