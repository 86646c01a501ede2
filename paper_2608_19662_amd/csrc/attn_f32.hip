// fp32 attention for the reference-precision path (encode and conversation
// attend).  One wave per (query row, head): the lanes split head_dim, each
// key's logit is a wave reduction, and the softmax is accumulated online in
// fp32 with exp2.  It exists to run the method exactly at fp32 input
// precision (no bf16 rounding anywhere); the bf16 MFMA kernels are the
// throughput path.
//
// Visibility follows the same definitions as the bf16 kernels: encode rows
// see the shared prefix and their own resource causally (ReCache Sec. 3,
// "Resource-Wise Attention"); conversation rows see the kept rows of their routed resources
// in request order and then the context causally, bottom-right aligned
// (Fig. 2, final mask).
#include "common.hpp"
#include "kernels.hpp"

namespace rc {

namespace {

struct OnlineSoftmax {
    float m = -INFINITY, l = 0.f, o0 = 0.f, o1 = 0.f;
    __device__ __forceinline__ void add(float s2, float v0, float v1) {
        const float mn = fmaxf(m, s2);
        const float alpha = exp2f(m - mn);
        const float p = exp2f(s2 - mn);
        l = l * alpha + p;
        o0 = o0 * alpha + p * v0;
        o1 = o1 * alpha + p * v1;
        m = mn;
    }
};

template <bool ENCODE>
__global__ __launch_bounds__(256) void attn_f32_kernel(const AttnF32Args a) {
    const int lane = threadIdx.x & 63;
    const long w = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int head = (int)(w % a.n_q_heads);
    const long rest = w / a.n_q_heads;
    const int unit = (int)(rest % a.n_units);
    const int row = (int)(rest / a.n_units);
    if (row >= a.max_rows) return;
    const int g = head / a.ratio;
    const int d = a.head_dim;
    const bool two = d == 128;  // lanes hold elements lane and lane + 64

    int q_row0, q_len;
    if constexpr (ENCODE) {
        q_row0 = a.cu_len[unit];
        q_len = a.cu_len[unit + 1] - q_row0;
    } else {
        q_row0 = a.cu_q[unit];
        q_len = a.cu_q[unit + 1] - q_row0;
    }
    if (row == a.max_rows - 1 && q_len > a.max_rows) {
        // rows past the grid's max_rows: NaN, so that a caller's size error
        // shows in the outputs instead of leaving them unwritten
        for (int r = a.max_rows; r < q_len && (long)q_row0 + r < a.lse_rows; ++r) {
            float* op = a.out + ((size_t)(q_row0 + r) * a.n_q_heads + head) * a.head_dim;
            op[lane] = __builtin_nanf("");
            if (a.head_dim == 128) op[lane + 64] = __builtin_nanf("");
            if (a.lse && lane == 0) a.lse[(size_t)head * a.lse_rows + q_row0 + r] = __builtin_nanf("");
        }
    }
    if (row >= q_len || q_row0 + row >= a.lse_rows) return;

    const float* qp = a.q + ((size_t)(q_row0 + row) * a.n_q_heads + head) * d;
    float q0 = qp[lane];
    float q1 = two ? qp[lane + 64] : 0.f;
    if constexpr (ENCODE) {
        const int pos = (a.pos_base ? a.pos_base[unit] : 0) + row;
        float s, c;
        if (two) {
            // pair (lane, lane + 64), frequency lane
            sincos_rev(rope_revolutions(pos, a.rope.rev[lane]), &s, &c);
            // the rounding of the key rotation, written out
            const float y0 = fmaf(q0, c, -(q1 * s)), y1 = fmaf(q1, c, q0 * s);
            q0 = y0;
            q1 = y1;
        } else {
            // pair (lane, lane + 32), frequency lane % 32
            sincos_rev(rope_revolutions(pos, a.rope.rev[lane & 31]), &s, &c);
            const float partner = __shfl_xor(q0, 32);
            q0 = (lane < 32) ? fmaf(q0, c, -(partner * s)) : fmaf(q0, c, partner * s);
        }
    }
    const float sc = a.scale * 1.44269504088896340736f;

    OnlineSoftmax acc;
    auto visit = [&](const float* kr, const float* vr) {
        float part = q0 * kr[lane] + (two ? q1 * kr[lane + 64] : 0.f);
        const float s2 = wave_sum(part) * sc;
        acc.add(s2, vr[lane], two ? vr[lane + 64] : 0.f);
    };

    if constexpr (ENCODE) {
        // the shared prefix, fully visible, then the resource's own rows
        const float* pk = a.k + (size_t)g * a.k_gstride * d;
        const float* pv = a.v + (size_t)g * a.k_gstride * d;
        for (int u = 0; u < a.p_len; ++u) visit(pk + (size_t)u * d, pv + (size_t)u * d);
        const float* kb = a.ck + ((size_t)g * a.c_rows + q_row0) * d;
        const float* vb = a.cv + ((size_t)g * a.c_rows + q_row0) * d;
        for (int u = 0; u <= row; ++u) visit(kb + (size_t)u * d, vb + (size_t)u * d);
    } else {
        const size_t e = ((size_t)unit * a.n_layers + a.layer) * a.n_kv_heads + g;
        const float* kb = a.k + (size_t)g * a.k_gstride * d;
        const float* vb = a.v + (size_t)g * a.k_gstride * d;
        for (int s = a.route_off[e]; s < a.route_off[e + 1]; ++s) {
            const int r = a.route_res[s];
            const int r_beg = a.res_off ? a.res_off[(size_t)r * a.n_kv_heads + g] : a.cu_kept[r];
            const int r_end = min(r_beg + (a.cu_kept[r + 1] - a.cu_kept[r]), (int)a.k_rows);
            for (int u = r_beg; u < r_end; ++u) visit(kb + (size_t)u * d, vb + (size_t)u * d);
        }
        const int c0 = a.cu_ctx[unit];
        const int tc = a.cu_ctx[unit + 1] - c0;
        const int last = min(tc - q_len + row, (int)a.c_rows - 1 - c0);
        const float* ckb = a.ck + ((size_t)g * a.c_rows + c0) * d;
        const float* cvb = a.cv + ((size_t)g * a.c_rows + c0) * d;
        for (int u = 0; u <= last; ++u) visit(ckb + (size_t)u * d, cvb + (size_t)u * d);
    }

    const float inv = 1.0f / acc.l;
    float* op = a.out + ((size_t)(q_row0 + row) * a.n_q_heads + head) * d;
    op[lane] = acc.o0 * inv;
    if (two) op[lane + 64] = acc.o1 * inv;
    if (a.lse && lane == 0)
        a.lse[(size_t)head * a.lse_rows + q_row0 + row] =
            (acc.m + log2f(acc.l)) * 0.69314718055994531f;
}

}  // namespace

hipError_t launch_attn_f32(const AttnF32Args& a, bool encode, hipStream_t stream) {
    const long waves = (long)a.max_rows * a.n_units * a.n_q_heads;
    if (waves == 0) return hipSuccess;
    const long blocks = (waves + 3) / 4;
    if (blocks > 0x7fffffffL) return hipErrorInvalidValue;
    if (encode)
        hipLaunchKernelGGL(attn_f32_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL(attn_f32_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace rc
