// Split-KV decode: one new conversation token per request attends the kept
// rows of the resources routed to its (layer, KV group) and the whole
// conversation context (final ReCache mask, Fig. 2, with Tq = 1), followed
// by a log-sum-exp merge of the splits.
//
// Memory-bound: every visible K/V row is read from HBM once per (request,
// layer, group), whatever the number of query heads in the group.  The
// products run on the matrix cores with the group's query heads as the N
// dimension of 16x16x32 bf16 MFMAs:
//     S^T = K Q^T      (A = 16 keys x 32 dims of K, straight from HBM into VGPRs)
//     O^T += V^T P^T   (A = V^T read from LDS with transpose reads, B = P^T
//                       packed from the S^T accumulators without shuffles)
// which leaves the VALU a few dozen instructions per 32 keys (the softmax),
// so the kernel streams at the memory system's pace.
//
// One block handles one contiguous range of the (request, group) key stream.
// Its four waves take 32-key tiles of the range in turn and run independent
// pipelines (own registers, own LDS buffers, no barriers in the loop): K and
// V of tile t + 1 are in flight while tile t is computed.  The four partial
// softmax states are merged in LDS at the end, and a second kernel merges the
// splits.
#include "common.hpp"
#include "kernels.hpp"

namespace rc {

namespace {

constexpr int kThreads = 256;
constexpr int kTk = 32;  // keys per wave tile
constexpr int kMaxSeg = 1024;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

template <int C>
struct Tag {
    static constexpr int value = C;
};

template <int HD>
struct DT {
    static constexpr int CPR = HD / 8;        // 16-byte chunks per row
    static constexpr int ROWB = HD * 2;       // bytes per row
    static constexpr int TILEB = kTk * ROWB;  // bytes of one V tile
    static constexpr int NKS = HD / 32;       // k-steps of S^T over head_dim
    static constexpr int NDB = HD / 16;       // 16-dim blocks of O^T
    static constexpr int RPI = 64 / CPR;      // rows per 1 KB wave copy
    static constexpr int NJ = kTk / RPI;      // copies per V tile
    static constexpr int NLOAD = 2 * NKS + NJ;  // vector memory operations per tile
    // s_waitcnt immediate for vmcnt(NLOAD) (the loads of the newer tile may
    // still be in flight), other counters unconstrained
    static constexpr int WAIT_PREV = (NLOAD & 15) | ((NLOAD >> 4) << 14) | 0x0F70;
};

template <int HD>
struct DecSmem {
    int seg_start[kMaxSeg + 1];
    int seg_row[kMaxSeg];
    int scan[4];  // wave totals of the segment-length scan
    // per wave: two V tile buffers; reused for the cross-wave merge
    alignas(16) char v[4][2][DT<HD>::TILEB];
};

// Chunk swizzle of a V tile row: the 16 rows x 32 bytes that one transpose
// read touches spread over all 64 banks exactly twice.
template <int CPR>
__device__ __forceinline__ int v_mask(int row) {
    return CPR == 16 ? 2 * (row & 7) : 2 * ((row >> 1) & 3);
}

__device__ __forceinline__ float xor16_max(float x) { return fmaxf(x, __shfl_xor(x, 16)); }
__device__ __forceinline__ float xor16_sum(float x) { return x + __shfl_xor(x, 16); }

template <int HD>
__global__ __launch_bounds__(kThreads, 2) void decode_kernel(const DecodeArgs a) {
    using T = DT<HD>;
    __shared__ DecSmem<HD> sm;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, grp = lane >> 4;  // MFMA column and row group of this lane

    int bid = blockIdx.x;
    const int split = bid % a.n_splits;
    bid /= a.n_splits;
    int g = bid % a.n_kv_heads;
    int b = bid / a.n_kv_heads;
    if (a.plan) {
        // with a work order the streams run longest first, so that the grid
        // does not end on a tail of long ones
        const int n_pairs = a.n_req * a.n_kv_heads;
        int p = a.plan[(size_t)a.layer * n_pairs + bid];
        p = min(max(p, 0), n_pairs - 1);  // in bounds whatever the plan holds
        b = p / a.n_kv_heads;
        g = p % a.n_kv_heads;
    }
    const int R = a.ratio;

    // ---- Q^T (B operand), loaded first since it depends on nothing else
    // (but the pair):
    // lane holds head l16 of the group (zero beyond R), dims ks*32 + grp*8 + [0, 8).
    const int qrow = min(a.cu_q[b], (int)a.lse_rows - 1);
    bf16x8_t qf[T::NKS];
#pragma unroll
    for (int ks = 0; ks < T::NKS; ++ks) {
        u32x4 w = {0u, 0u, 0u, 0u};
        if (l16 < R)
            w = *reinterpret_cast<const u32x4*>(a.q + ((size_t)qrow * a.n_q_heads + g * R + l16) * HD +
                                                ks * 32 + grp * 8);
        qf[ks] = __builtin_bit_cast(bf16x8_t, w);
    }

    // ---- visible segments of this (request, layer, group): kept rows of the
    // routed resources, request order.  Exclusive scan of their lengths.
    const size_t e = ((size_t)b * a.n_layers + a.layer) * a.n_kv_heads + g;
    const int r0 = a.route_off[e];
    const int n_seg = a.route_off[e + 1] - r0;
    if (n_seg > kMaxSeg || a.cu_q[b + 1] - a.cu_q[b] != 1) {
        // A route list longer than the segment table, or a request that does
        // not have exactly one query: this split's partial becomes NaN with
        // an infinite max, which the merge turns into NaN outputs for the
        // group (a caller's size error shows instead of dropped keys).
        for (int idx = tid; idx < R * HD; idx += kThreads) {
            const size_t slot = ((size_t)b * a.n_q_heads + g * R + idx / HD) * a.n_splits + split;
            a.ws_o[slot * HD + idx % HD] = __builtin_nanf("");
            if (idx % HD == 0) {
                a.ws_ml[slot * 2 + 0] = INFINITY;
                a.ws_ml[slot * 2 + 1] = __builtin_nanf("");
            }
        }
        return;
    }
    int lens[4], part = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int s = tid * 4 + i;
        lens[i] = 0;
        if (s < n_seg) {
            const int r = a.route_res[r0 + s];
            const int k0 = a.cu_kept[r];
            lens[i] = a.cu_kept[r + 1] - k0;
            sm.seg_row[s] = a.res_off ? a.res_off[(size_t)r * a.n_kv_heads + g] : k0;
        }
        part += lens[i];
    }
    int s_vis;
    {
        int run = block4_exclusive_scan(part, sm.scan, &s_vis);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int s = tid * 4 + i;
            if (s < n_seg) sm.seg_start[s] = run;
            run += lens[i];
        }
    }
    if (tid == 0) sm.seg_start[n_seg] = s_vis;
    const int c0 = a.cu_ctx[b];
    const int tc = a.cu_ctx[b + 1] - c0;
    const int n_keys = s_vis + tc;
    // this split's key range: whole 32-key tiles, the last one possibly partial
    int chunk = (n_keys + a.n_splits - 1) / a.n_splits;
    chunk = (chunk + kTk - 1) / kTk * kTk;
    const int s0 = min(split * chunk, n_keys);
    const int s1 = min(s0 + chunk, n_keys);
    const int n_tiles = (s1 - s0 + kTk - 1) / kTk;
    __syncthreads();

    const uint16_t* rk = a.rk + (size_t)g * a.r_gstride * HD;
    const uint16_t* rv = a.rv + (size_t)g * a.r_gstride * HD;
    const uint16_t* ck = a.ck + (size_t)g * a.c_rows * HD;
    const uint16_t* cv = a.cv + (size_t)g * a.c_rows * HD;
    // Row of stream key p in its buffer (p < s_vis: kept resource rows, else
    // context rows), clamped into the buffer.  A lane's segment index only
    // moves forward, since each lane visits its keys in increasing order.
    auto row_of = [&](int p, int& sidx, int& hi, int& dl) -> size_t {
        if (p < s_vis) {
            while (p >= hi && sidx + 1 < n_seg) {
                ++sidx;
                hi = sm.seg_start[sidx + 1];
                dl = sm.seg_row[sidx] - sm.seg_start[sidx];
            }
            return min((size_t)(dl + p), (size_t)a.r_rows - 1);
        }
        return min((size_t)c0 + (p - s_vis), (size_t)a.c_rows - 1);
    };
    const int seg_hi0 = n_seg > 0 ? sm.seg_start[1] : 0;
    const int seg_dl0 = n_seg > 0 ? sm.seg_row[0] : 0;
    int ks_i = 0, ks_hi = seg_hi0, ks_dl = seg_dl0;  // walk for this lane's K keys
    int vs_i = 0, vs_hi = seg_hi0, vs_dl = seg_dl0;  // walk for this lane's V keys
    int us_i = 0;                                     // wave-uniform walk (fast test)
    int us_hi = __builtin_amdgcn_readfirstlane(seg_hi0), us_dl = __builtin_amdgcn_readfirstlane(seg_dl0);

    // ---- loads of one tile.  K: lane holds key kb*16 + l16 of the tile,
    // dims ks*32 + grp*8 + [0, 8), in registers.  V: copy j of the wave moves
    // rows j*RPI + i / CPR of the tile; lane i lands at byte 16 i, i.e.
    // physical chunk i % CPR, which holds logical chunk (i % CPR) ^ v_mask(row).
    char* vbuf = sm.v[wave][0];
    u32x4 kreg[2][2][T::NKS];  // [buffer][key block][k-step]
    auto load_tile = [&](auto buf_tag, int t) {
        constexpr int buf = decltype(buf_tag)::value;
        const int tb = s0 + (wave + 4 * t) * kTk;  // first key of the tile
        // fast tile: all 32 keys consecutive in one buffer (wave-uniform test)
        bool fast = false;
        const uint16_t* kb0 = rk;
        const uint16_t* vb0 = rv;
        if (tb + kTk <= s1) {
            if (tb + kTk <= s_vis) {
                while (tb >= us_hi && us_i + 1 < n_seg) {
                    ++us_i;
                    us_hi = __builtin_amdgcn_readfirstlane(sm.seg_start[us_i + 1]);
                    us_dl = __builtin_amdgcn_readfirstlane(sm.seg_row[us_i]) -
                            __builtin_amdgcn_readfirstlane(sm.seg_start[us_i]);
                }
                const long row0 = (long)us_dl + tb;
                if (tb + kTk <= us_hi && row0 >= 0 && row0 + kTk <= a.r_rows) {
                    fast = true;
                    kb0 = rk + row0 * HD;
                    vb0 = rv + row0 * HD;
                }
            } else if (tb >= s_vis) {
                const long row0 = (long)c0 + (tb - s_vis);
                if (row0 + kTk <= a.c_rows) {
                    fast = true;
                    kb0 = ck + row0 * HD;
                    vb0 = cv + row0 * HD;
                }
            }
        }
        u64x2 ksrc;
        if (fast) {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) ksrc[kb] = (uint64_t)(kb0 + (kb * 16 + l16) * HD);
        } else {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const int p = min(tb + kb * 16 + l16, s1 - 1);
                const size_t r = row_of(p, ks_i, ks_hi, ks_dl);
                ksrc[kb] = (uint64_t)((p < s_vis ? rk : ck) + r * HD);
            }
        }
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int ks = 0; ks < T::NKS; ++ks)
                kreg[buf][kb][ks] =
                    *reinterpret_cast<const u32x4*>((const uint16_t*)ksrc[kb] + ks * 32 + grp * 8);
        char* dst = vbuf + buf * T::TILEB;
#pragma unroll
        for (int j = 0; j < T::NJ; ++j) {
            const int row = j * T::RPI + lane / T::CPR;
            const int chunk = (lane % T::CPR) ^ v_mask<T::CPR>(row);
            const uint16_t* src;
            if (fast) {
                src = vb0 + row * HD + chunk * 8;
            } else {
                const int p = min(tb + row, s1 - 1);
                const size_t r = row_of(p, vs_i, vs_hi, vs_dl);
                src = (p < s_vis ? rv : cv) + r * HD + chunk * 8;
            }
            __builtin_amdgcn_global_load_lds(src, (lds_void*)(dst + j * 1024), 16, 0, 0);
        }
    };

    // ---- transpose-read offsets: lane (grp, i) of a 16-lane group points at
    // row w*16 + grp*4 + i/4, dims db*16 + 4*(i % 4), so that it receives dim
    // db*16 + i of rows w*16 + grp*4 + [0, 4): keys grp*4 + [0, 4) (w = 0) and
    // 16 + grp*4 + [0, 4) (w = 1), the keys whose weights this lane holds in
    // the S^T accumulators of the two 16-key blocks.
    auto tr_off = [&](int db, int w) -> uint32_t {
        const int row = w * 16 + grp * 4 + (l16 >> 2);
        const int col = db * 16 + 4 * (l16 & 3);
        return (uint32_t)(row * T::ROWB + (((col >> 3) ^ v_mask<T::CPR>(row)) << 4) + (col & 7) * 2);
    };

    const float sl2 = a.scale_log2;
    const bf16x2 ones2 = __builtin_bit_cast(bf16x2, 0x3F803F80u);  // (1.0, 1.0) in bf16
    float m = -INFINITY;  // running max (log2 units) for head l16
    float lsum = 0.f;     // this lane's part of the row sum
    f32x4 oacc[T::NDB];   // O^T: dims db*16 + grp*4 + [0, 4) of head l16
#pragma unroll
    for (int db = 0; db < T::NDB; ++db) oacc[db] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto compute = [&](auto buf_tag, int t) {
        constexpr int buf = decltype(buf_tag)::value;
        const int tb = s0 + (wave + 4 * t) * kTk;
        f32x4 sacc[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            sacc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < T::NKS; ++ks)
                sacc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    __builtin_bit_cast(bf16x8_t, kreg[buf][kb][ks]), qf[ks], sacc[kb], 0, 0, 0);
        }
        // keys past the range end (last tile of the range only)
        if (tb + kTk > s1) {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (tb + kb * 16 + grp * 4 + r >= s1) sacc[kb][r] = -INFINITY;
        }
        float mt = fmaxf(fmaxf(fmaxf(sacc[0][0], sacc[0][1]), fmaxf(sacc[0][2], sacc[0][3])),
                         fmaxf(fmaxf(sacc[1][0], sacc[1][1]), fmaxf(sacc[1][2], sacc[1][3])));
        mt = pair_max(xor16_max(mt)) * sl2;  // over the tile's 32 keys, log2 units
        // lazy rescale: m moves only when a logit exceeds it by more than 8
        // (weights stay <= 2^8); O and the row sum share m, so this is exact
        if (__builtin_amdgcn_ballot_w64(mt > m + 8.f)) {
            const float m_new = fmaxf(m, mt);
            const float alpha = __builtin_amdgcn_exp2f(m - m_new);  // 0 when m == -inf
            lsum *= alpha;
#pragma unroll
            for (int db = 0; db < T::NDB; ++db) oacc[db] *= alpha;
            m = m_new;
        }
        uint32_t w[4];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int r = 0; r < 4; r += 2) {
                const float p0 = __builtin_amdgcn_exp2f(fmaf(sacc[kb][r], sl2, -m));
                const float p1 = __builtin_amdgcn_exp2f(fmaf(sacc[kb][r + 1], sl2, -m));
                const uint32_t pk = pack_bf16x2(p0, p1);
                w[kb * 2 + r / 2] = pk;
                // row sum of the weights as rounded for the P V product
                lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk), ones2, lsum, false);
            }
        const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, u32x4{w[0], w[1], w[2], w[3]});
        const char* st = vbuf + buf * T::TILEB;
#pragma unroll
        for (int db = 0; db < T::NDB; ++db) {
            const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(st + tr_off(db, 0)));
            const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(st + tr_off(db, 1)));
            const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
            const bf16x8_t av = __builtin_bit_cast(bf16x8_t, u32x4{l2[0], l2[1], h2[0], h2[1]});
            oacc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, pf, oacc[db], 0, 0, 0);
        }
    };

    // This wave's tiles are wave, wave + 4, ... of the range; the loads of
    // the next one are in flight while one is computed.  Only this wave
    // reads its V buffers, so waiting for its own copies is enough.
    const int my_tiles = n_tiles > wave ? (n_tiles - wave + 3) / 4 : 0;
    if (my_tiles > 0) load_tile(Tag<0>{}, 0);
    for (int t = 0; t < my_tiles; t += 2) {
        if (t + 1 < my_tiles) {
            load_tile(Tag<1>{}, t + 1);
            __builtin_amdgcn_s_waitcnt(T::WAIT_PREV);
        } else {
            __builtin_amdgcn_s_waitcnt(0x0F70);
        }
        compute(Tag<0>{}, t);
        if (t + 1 < my_tiles) {
            if (t + 2 < my_tiles) {
                load_tile(Tag<0>{}, t + 2);
                __builtin_amdgcn_s_waitcnt(T::WAIT_PREV);
            } else {
                __builtin_amdgcn_s_waitcnt(0x0F70);
            }
            compute(Tag<1>{}, t + 1);
        }
    }

    // ---- merge: the four row groups of a head hold disjoint dims of O^T and
    // parts of its row sum; then the four waves, through LDS.
    lsum = pair_sum(xor16_sum(lsum));
    __syncthreads();  // every wave is done with its V buffers
    float* mo = reinterpret_cast<float*>(&sm.v[0][0][0]);  // [wave][16 heads][HD]
    float* mml = mo + 4 * 16 * HD;                           // [wave][16 heads][2]
#pragma unroll
    for (int db = 0; db < T::NDB; ++db)
#pragma unroll
        for (int r = 0; r < 4; ++r) mo[(wave * 16 + l16) * HD + db * 16 + grp * 4 + r] = oacc[db][r];
    if (grp == 0) {
        mml[(wave * 16 + l16) * 2 + 0] = m;
        mml[(wave * 16 + l16) * 2 + 1] = lsum;
    }
    __syncthreads();
    for (int idx = tid; idx < R * HD; idx += kThreads) {
        const int h = idx / HD, d = idx % HD;
        float mx = -INFINITY;
#pragma unroll
        for (int w = 0; w < 4; ++w) mx = fmaxf(mx, mml[(w * 16 + h) * 2]);
        float num = 0.f, den = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const float mw = mml[(w * 16 + h) * 2];
            const float sc = mw == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw - mx);
            num += sc * mo[(w * 16 + h) * HD + d];
            den += sc * mml[(w * 16 + h) * 2 + 1];
        }
        const size_t slot = ((size_t)b * a.n_q_heads + g * R + h) * a.n_splits + split;
        a.ws_o[slot * HD + d] = num;
        if (d == 0) {
            a.ws_ml[slot * 2 + 0] = mx;
            a.ws_ml[slot * 2 + 1] = den;
        }
    }
}

// out[b][h] = sum_s w_s O_s / sum_s w_s l_s with w_s = exp2(m_s - max m);
// splits that saw no key carry m_s = -inf and weigh nothing.
template <int HD>
__global__ __launch_bounds__(HD) void combine_kernel(const DecodeArgs a) {
    const int bh = blockIdx.x;
    const int b = bh / a.n_q_heads, h = bh % a.n_q_heads;
    const int d = threadIdx.x;
    const size_t slot0 = (size_t)bh * a.n_splits;
    // the (max, sum) pairs and this dimension of every split's partial are
    // loaded together, four splits at a time, then merged in split order
    constexpr int C = 4;
    float mx = -INFINITY, num = 0.f, den = 0.f;
    auto load = [&](int s0, float2* ml, float* o) {
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const bool in = s0 + c < a.n_splits;
            ml[c] = in ? reinterpret_cast<const float2*>(a.ws_ml)[slot0 + s0 + c] : make_float2(-INFINITY, 0.f);
            o[c] = in ? a.ws_o[(slot0 + s0 + c) * HD + d] : 0.f;
        }
    };
    auto merge = [&](const float2* ml, const float* o) {
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const float w = ml[c].x == -INFINITY ? 0.f : exp2f(ml[c].x - mx);
            den += w * ml[c].y;
            num += w * o[c];
        }
    };
    if (a.n_splits <= C) {
        // the common case: every load in flight at once
        float2 ml[C];
        float o[C];
        load(0, ml, o);
#pragma unroll
        for (int c = 0; c < C; ++c) mx = fmaxf(mx, ml[c].x);
        merge(ml, o);
    } else {
        for (int s0 = 0; s0 < a.n_splits; s0 += C) {
            float2 ml[C];
            float o[C];
            load(s0, ml, o);
#pragma unroll
            for (int c = 0; c < C; ++c) mx = fmaxf(mx, ml[c].x);
        }
        for (int s0 = 0; s0 < a.n_splits; s0 += C) {
            float2 ml[C];
            float o[C];
            load(s0, ml, o);
            merge(ml, o);
        }
    }
    const int row = a.cu_q[b];
    if (row < 0 || row >= a.lse_rows) return;
    a.out[((size_t)row * a.n_q_heads + h) * HD + d] = f32_to_bf16_bits(num / den);
    if (a.lse && d == 0) a.lse[(size_t)h * a.lse_rows + row] = (mx + log2f(den)) * 0.69314718055994531f;
}

template <int HD>
hipError_t launch_dec(const DecodeArgs& a, hipStream_t s) {
    const long blocks = (long)a.n_req * a.n_kv_heads * a.n_splits;
    hipLaunchKernelGGL((decode_kernel<HD>), dim3((unsigned)blocks), dim3(kThreads), 0, s, a);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL((combine_kernel<HD>), dim3((unsigned)(a.n_req * a.n_q_heads)), dim3(HD), 0, s, a);
    return hipGetLastError();
}

}  // namespace

int decode_splits(int n_req, int n_kv_heads, int max_kv) {
    const long units = (long)n_req * n_kv_heads;
    long s = (1536 + units - 1) / units;       // about three rounds of two blocks per CU
    const long by_len = (max_kv + 511) / 512;  // and at least ~512 keys per block
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
    if (a.ratio < 1 || a.ratio > 16) return hipErrorInvalidValue;
    return a.head_dim == 128 ? launch_dec<128>(a, s) : launch_dec<64>(a, s);
}

}  // namespace rc
