// Split-KV decode: one new conversation token per request attends the kept
// rows of the resources routed to its (layer, KV group) and the whole
// conversation context (final ReCache mask, Fig. 2, with Tq = 1), followed
// by a log-sum-exp merge of the splits.
//
// Memory-bound: every visible K/V row is read from HBM once.  One block
// handles one contiguous range of the (request, group) key stream for all
// query heads of the group.  Rows are read 16 bytes per lane, 16 lanes per
// 256-byte row, so each wave instruction covers 4 whole rows.  Pass 1 forms
// logits with bf16 dot2 instructions and DPP row reductions and keeps them in
// LDS; the weights exp2(s - max) are then formed once per (row, head); pass 2
// streams V and accumulates P V in fp32.  Ranges longer than the LDS logit
// buffer are processed in sub-chunks with online rescaling, so any stream
// length is handled.
#include "common.hpp"
#include "kernels.hpp"

namespace rc {

namespace {

constexpr int kThreads = 256;
constexpr int kSub = 512;  // rows per sub-chunk held in LDS
constexpr int kMaxSeg = 1024;

template <int CTRL>
__device__ __forceinline__ float dpp_sum_step(float x) {
    return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum over groups of LPR consecutive lanes (LPR = 16 or 8); every lane of the
// group ends with the group sum.
template <int LPR>
__device__ __forceinline__ float row_sum(float x) {
    x = dpp_sum_step<0xB1>(x);   // quad_perm [1,0,3,2]
    x = dpp_sum_step<0x4E>(x);   // quad_perm [2,3,0,1]
    x = dpp_sum_step<0x141>(x);  // row_half_mirror: pairs the two quads of 8 lanes
    if constexpr (LPR == 16) x = dpp_sum_step<0x140>(x);  // row_mirror: pairs the two halves
    return x;
}

// acc + sum of the 8 products of two rows of 8 bf16 (fp32 accumulation).
// The dwords are taken out of the 16-byte vectors first: handed the vector
// elements directly, the compiler's dot2 lowering reads the first dword four
// times.
__device__ __forceinline__ float dot8_bf16(const u32x4& k, const u32x4& q, float acc) {
    const uint32_t ks[4] = {k.x, k.y, k.z, k.w}, qs[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int w = 0; w < 4; ++w)
        acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, ks[w]),
                                              __builtin_bit_cast(bf16x2, qs[w]), acc, false);
    return acc;
}

// One row's R logits into LDS with as few vector stores as alignment allows.
template <int R>
__device__ __forceinline__ void store_row(float* dst, const float* v) {
    // dst = sc + i * R is 16-byte aligned when R % 4 == 0, 8-byte when R is even
    if constexpr (R % 4 == 0) {
#pragma unroll
        for (int j = 0; j < R; j += 4)
            *reinterpret_cast<float4*>(dst + j) = make_float4(v[j], v[j + 1], v[j + 2], v[j + 3]);
    } else if constexpr (R % 2 == 0) {
#pragma unroll
        for (int j = 0; j < R; j += 2) *reinterpret_cast<float2*>(dst + j) = make_float2(v[j], v[j + 1]);
    } else {
#pragma unroll
        for (int j = 0; j < R; ++j) dst[j] = v[j];
    }
}

template <int HD, int R>
struct DecSmem {
    int seg_start[kMaxSeg + 1];
    int seg_row[kMaxSeg];
    int scan[kThreads];
    alignas(16) float sc[kSub * R];  // logits, then weights, [row][head]
    float red[4][R];           // per-wave maxima
    float bm[R];               // block running max (log2 units)
    float ored[4][R][HD];      // cross-wave O reduction
    float lred[4][R];
};

template <int HD, int R>
__global__ __launch_bounds__(kThreads) void decode_kernel(const DecodeArgs a) {
    constexpr int LPR = HD / 8;     // lanes per row
    constexpr int RPW = 64 / LPR;   // rows per wave instruction
    constexpr int RPB = 4 * RPW;    // rows per block step
    constexpr int UNR = 4;
    __shared__ DecSmem<HD, R> sm;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int c = lane % LPR, sub = lane / LPR;

    int bid = blockIdx.x;
    const int split = bid % a.n_splits;
    bid /= a.n_splits;
    const int g = bid % a.n_kv_heads;
    const int b = bid / a.n_kv_heads;

    // ---- visible segments of this (request, layer, group)
    const size_t e = ((size_t)b * a.n_layers + a.layer) * a.n_kv_heads + g;
    const int r0 = a.route_off[e];
    const int n_seg = min(a.route_off[e + 1] - r0, kMaxSeg);
    int lens[4], part = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int s = tid * 4 + i;
        lens[i] = 0;
        if (s < n_seg) {
            const int r = a.route_res[r0 + s];
            const int k0 = a.cu_kept[r];
            lens[i] = a.cu_kept[r + 1] - k0;
            sm.seg_row[s] = k0;
        }
        part += lens[i];
    }
    sm.scan[tid] = part;
    __syncthreads();
    for (int o = 1; o < kThreads; o <<= 1) {
        const int add = tid >= o ? sm.scan[tid - o] : 0;
        __syncthreads();
        sm.scan[tid] += add;
        __syncthreads();
    }
    {
        int run = sm.scan[tid] - part;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int s = tid * 4 + i;
            if (s < n_seg) sm.seg_start[s] = run;
            run += lens[i];
        }
    }
    const int s_vis = sm.scan[kThreads - 1];
    const int c0 = a.cu_ctx[b];
    const int tc = a.cu_ctx[b + 1] - c0;
    const int n_keys = s_vis + tc;
    int chunk = (n_keys + a.n_splits - 1) / a.n_splits;
    chunk = (chunk + RPB - 1) / RPB * RPB;
    const int s0 = min(split * chunk, n_keys);
    const int s1 = min(s0 + chunk, n_keys);
    __syncthreads();

    const uint16_t* rk = a.rk + (size_t)g * a.r_rows * HD;
    const uint16_t* rv = a.rv + (size_t)g * a.r_rows * HD;
    const uint16_t* ck = a.ck + ((size_t)g * a.c_rows + c0) * HD;
    const uint16_t* cv = a.cv + ((size_t)g * a.c_rows + c0) * HD;
    auto row_off = [&](int p, bool& is_ctx) -> size_t {
        if (p < s_vis) {
            int lo = 0, hi = n_seg - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (sm.seg_start[mid] <= p) lo = mid; else hi = mid - 1;
            }
            is_ctx = false;
            return min((size_t)(sm.seg_row[lo] + (p - sm.seg_start[lo])), (size_t)a.r_rows - 1) * HD;
        }
        is_ctx = true;
        return min((size_t)(p - s_vis), (size_t)(a.c_rows - 1 - c0)) * HD;
    };

    // ---- query heads of the group, raw bf16 pairs for dot2
    const int qrow = min(a.cu_q[b], (int)a.lse_rows - 1);
    u32x4 qv[R];
#pragma unroll
    for (int h = 0; h < R; ++h)
        qv[h] = *reinterpret_cast<const u32x4*>(a.q + ((size_t)qrow * a.n_q_heads + g * R + h) * HD + c * 8);

    float o[R][8];
    float lacc[R];
#pragma unroll
    for (int h = 0; h < R; ++h) {
        lacc[h] = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[h][i] = 0.f;
    }
    if (tid < R) sm.bm[tid] = -INFINITY;
    const float sl2 = a.scale_log2;

    for (int base = s0; base < s1; base += kSub) {
        const int n = min(kSub, s1 - base);
        // pass 1: logits
        float mloc[R];
#pragma unroll
        for (int h = 0; h < R; ++h) mloc[h] = -INFINITY;
        for (int i0 = wave * RPW + sub; i0 < n; i0 += RPB * UNR) {
            u32x4 kr[UNR];
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                const int i = i0 + u * RPB;
                if (i < n) {
                    bool is_ctx;
                    const size_t ro = row_off(base + i, is_ctx);
                    kr[u] = *reinterpret_cast<const u32x4*>((is_ctx ? ck : rk) + ro + c * 8);
                }
            }
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                const int i = i0 + u * RPB;
                if (i < n) {
                    float sv[R];
#pragma unroll
                    for (int h = 0; h < R; ++h) {
                        sv[h] = row_sum<LPR>(dot8_bf16(kr[u], qv[h], 0.f)) * sl2;
                        mloc[h] = fmaxf(mloc[h], sv[h]);
                    }
                    if (c == 0) store_row<R>(&sm.sc[i * R], sv);
                }
            }
        }
#pragma unroll
        for (int h = 0; h < R; ++h) {
            const float wm = wave_max(mloc[h]);
            if (lane == 0) sm.red[wave][h] = wm;
        }
        __syncthreads();
        float alpha[R];
#pragma unroll
        for (int h = 0; h < R; ++h) {
            const float mold = sm.bm[h];
            const float mnew = fmaxf(fmaxf(mold, fmaxf(sm.red[0][h], sm.red[1][h])),
                                     fmaxf(sm.red[2][h], sm.red[3][h]));
            alpha[h] = __builtin_amdgcn_exp2f(mold - mnew);  // 0 when mold == -inf
            lacc[h] *= alpha[h];
#pragma unroll
            for (int i = 0; i < 8; ++i) o[h][i] *= alpha[h];
        }
        __syncthreads();  // everyone has read the old maxima
        if (tid < R) {
            const int h = tid;
            sm.bm[h] = fmaxf(fmaxf(sm.bm[h], fmaxf(sm.red[0][h], sm.red[1][h])),
                             fmaxf(sm.red[2][h], sm.red[3][h]));
        }
        __syncthreads();
        // weights, once per (row, head)
        for (int idx = tid; idx < n * R; idx += kThreads)
            sm.sc[idx] = __builtin_amdgcn_exp2f(sm.sc[idx] - sm.bm[idx % R]);
        __syncthreads();
        // pass 2: P V
        for (int i0 = wave * RPW + sub; i0 < n; i0 += RPB * UNR) {
            u32x4 vr[UNR];
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                const int i = i0 + u * RPB;
                if (i < n) {
                    bool is_ctx;
                    const size_t ro = row_off(base + i, is_ctx);
                    vr[u] = *reinterpret_cast<const u32x4*>((is_ctx ? cv : rv) + ro + c * 8);
                }
            }
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                const int i = i0 + u * RPB;
                if (i < n) {
                    float v[8];
#pragma unroll
                    for (int w = 0; w < 4; ++w) {
                        v[2 * w] = __uint_as_float(vr[u][w] << 16);
                        v[2 * w + 1] = __uint_as_float(vr[u][w] & 0xffff0000u);
                    }
#pragma unroll
                    for (int h = 0; h < R; ++h) {
                        const float p = sm.sc[i * R + h];
                        if (c == 0) lacc[h] += p;
#pragma unroll
                        for (int k = 0; k < 8; ++k) o[h][k] = fmaf(p, v[k], o[h][k]);
                    }
                }
            }
        }
        __syncthreads();  // sc is rewritten by the next sub-chunk
    }

    // ---- reduce over the row groups of a wave, then over waves
#pragma unroll
    for (int h = 0; h < R; ++h) {
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            float x = o[h][k];
            for (int m = LPR; m < 64; m <<= 1) x += __shfl_xor(x, m);
            o[h][k] = x;
        }
        float l = lacc[h];
        for (int m = LPR; m < 64; m <<= 1) l += __shfl_xor(l, m);
        lacc[h] = l;
    }
    if (sub == 0) {
#pragma unroll
        for (int h = 0; h < R; ++h) {
#pragma unroll
            for (int k = 0; k < 8; ++k) sm.ored[wave][h][c * 8 + k] = o[h][k];
            if (c == 0) sm.lred[wave][h] = lacc[h];
        }
    }
    __syncthreads();
    for (int idx = tid; idx < R * HD; idx += kThreads) {
        const int h = idx / HD, d = idx % HD;
        const float sum = sm.ored[0][h][d] + sm.ored[1][h][d] + sm.ored[2][h][d] + sm.ored[3][h][d];
        const size_t slot = ((size_t)b * a.n_q_heads + g * R + h) * a.n_splits + split;
        a.ws_o[slot * HD + d] = sum;
        if (d == 0) {
            a.ws_ml[slot * 2 + 0] = sm.bm[h];
            a.ws_ml[slot * 2 + 1] = sm.lred[0][h] + sm.lred[1][h] + sm.lred[2][h] + sm.lred[3][h];
        }
    }
}

// out[b][h] = sum_s w_s O_s / sum_s w_s l_s with w_s = exp2(m_s - max m).
template <int HD>
__global__ __launch_bounds__(HD) void combine_kernel(const DecodeArgs a) {
    const int bh = blockIdx.x;
    const int b = bh / a.n_q_heads, h = bh % a.n_q_heads;
    const int d = threadIdx.x;
    const size_t slot0 = (size_t)bh * a.n_splits;
    float mx = -INFINITY;
    for (int s = 0; s < a.n_splits; ++s) mx = fmaxf(mx, a.ws_ml[(slot0 + s) * 2]);
    float num = 0.f, den = 0.f;
    for (int s = 0; s < a.n_splits; ++s) {
        const float w = exp2f(a.ws_ml[(slot0 + s) * 2] - mx);
        den += w * a.ws_ml[(slot0 + s) * 2 + 1];
        num += w * a.ws_o[(slot0 + s) * HD + d];
    }
    const int row = a.cu_q[b];
    if (row < 0 || row >= a.lse_rows) return;
    a.out[((size_t)row * a.n_q_heads + h) * HD + d] = f32_to_bf16_bits(num / den);
    if (a.lse && d == 0) a.lse[(size_t)h * a.lse_rows + row] = (mx + log2f(den)) * 0.69314718055994531f;
}

template <int HD, int R>
hipError_t launch_dec(const DecodeArgs& a, hipStream_t s) {
    const long blocks = (long)a.n_req * a.n_kv_heads * a.n_splits;
    hipLaunchKernelGGL((decode_kernel<HD, R>), dim3((unsigned)blocks), dim3(kThreads), 0, s, a);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL((combine_kernel<HD>), dim3((unsigned)(a.n_req * a.n_q_heads)), dim3(HD), 0, s, a);
    return hipGetLastError();
}

}  // namespace

int decode_splits(int n_req, int n_kv_heads, int max_kv) {
    const long units = (long)n_req * n_kv_heads;
    long s = (8192 + units - 1) / units;        // aim at ~32 blocks per CU
    const long by_len = (max_kv + 255) / 256;   // and at least ~256 rows per block
    if (s > by_len) s = by_len;
    if (s > 64) s = 64;
    if (s < 1) s = 1;
    return (int)s;
}

size_t decode_workspace_bytes(int n_req, int n_q_heads, int head_dim, int n_splits) {
    const size_t slots = (size_t)n_req * n_q_heads * n_splits;
    return slots * head_dim * sizeof(float) + slots * 2 * sizeof(float);
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t s) {
    if ((long)a.n_req * a.n_kv_heads * a.n_splits > 0x7fffffffL) return hipErrorInvalidValue;
    const int R = a.ratio;
    if (a.head_dim == 128) {
        switch (R) {
            case 1: return launch_dec<128, 1>(a, s);
            case 2: return launch_dec<128, 2>(a, s);
            case 3: return launch_dec<128, 3>(a, s);
            case 4: return launch_dec<128, 4>(a, s);
            case 5: return launch_dec<128, 5>(a, s);
            case 6: return launch_dec<128, 6>(a, s);
            case 7: return launch_dec<128, 7>(a, s);
            case 8: return launch_dec<128, 8>(a, s);
        }
    } else {
        switch (R) {
            case 1: return launch_dec<64, 1>(a, s);
            case 2: return launch_dec<64, 2>(a, s);
            case 3: return launch_dec<64, 3>(a, s);
            case 4: return launch_dec<64, 4>(a, s);
            case 5: return launch_dec<64, 5>(a, s);
            case 6: return launch_dec<64, 6>(a, s);
            case 7: return launch_dec<64, 7>(a, s);
            case 8: return launch_dec<64, 8>(a, s);
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace rc
