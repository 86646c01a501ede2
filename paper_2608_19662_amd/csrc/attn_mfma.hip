// bf16 flash attention on gfx950 MFMA, shared by
//   - resource encoding: block-diagonal causal attention inside each packed
//     resource, with RoPE at resource-local positions applied to the query
//     tile on load (ReCache Sec. 3, "Resource-Wise Attention"; Fig. 2(a));
//   - conversation prefill: queries over the kept rows of the resources routed
//     to their (layer, KV group), then causal context (final ReCache mask,
//     Fig. 2; Sec. 3, "Structural Pruning" / "Semantic Pruning").
//
// Both are one "key stream" per (unit, KV group): a query with local index i
// sees stream keys p <= off + i.  Encode: unit = resource, stream = its rows,
// off = 0.  Prefill: unit = request, stream = [routed kept rows in request
// order] ++ [context rows], off = S_vis + Tc - Tq.
//
// Work decomposition.  A workgroup is 4 waves that share one KV group and
// 4 * P (query head, 32-row block) pairs of it (hpw heads x rbw row blocks,
// hpw the largest of 4, 2, 1 dividing the group size).  Each wave owns P pairs
// and computes, for each, the transposed products
//     S^T = K Q^T    (32x32x16 bf16 MFMA; A = K rows from LDS, B = Q^T in VGPRs)
//     O^T += V^T P^T (A = V^T from LDS, B = P^T straight from the S^T accumulators)
// Every A fragment read from LDS feeds the MFMAs of all P pairs.  P = 2 halves
// LDS traffic per flop but needs ~500 registers per lane, so only one wave
// fits per SIMD and the softmax of one wave can no longer hide behind another
// wave's MFMAs; on MI355X it measured slower than P = 1 at two waves per SIMD
// (encode 0.35 vs 0.47 PFLOP/s), so the launcher instantiates P = 1.  Each
// lane owns exactly one query row of a pair in both accumulators, so row max
// and row sum need one cross-lane step (lanes l and l^32) and the rescale of O
// is lane-local.  K / V tiles of 64 keys are staged through LDS, double buffered
// (global loads of tile t+1 are in flight while tile t is computed).  Both
// tiles are stored row-major with an XOR swizzle of their 16-byte chunks; the
// V^T operand is read with gfx950's LDS transpose reads, in the key order in
// which the S^T accumulator hands P^T to the second product.
//
// Tiles never cross a resource boundary in encode, and the reduction order
// depends only on local indices, so a resource's outputs are bit-identical
// wherever it is packed and whatever its neighbours are.
#include "common.hpp"
#include "kernels.hpp"

namespace rc {

namespace {

constexpr int kBK = 64;  // keys per tile
constexpr int kThreads = 256;

template <int HD, int P>
struct Tile {
    static constexpr int CPR = HD / 8;              // 16-byte chunks per row
    static constexpr int KPT = kBK * CPR / kThreads;  // keys per thread per tile (4 or 2)
    static constexpr int NT = HD / 16;              // MFMA k-steps over head_dim
    static constexpr int NDB = HD / 32;             // 32-wide blocks of head_dim
    static constexpr int STAGE = 2 * kBK * HD;      // bf16 elements per stage (K + V)
    static constexpr int ROPE = 128 * P * HD * 2;   // bf16-sized elements of a cos/sin table for 128 * P rows
};

constexpr int kMaxSeg = 1024;

template <int C>
struct StageTag {
    static constexpr int value = C;
};

template <int HD, bool ENCODE, int P>
struct Smem {
    // encode also stages a cos / sin table for up to 128 * P query rows here
    alignas(16) uint16_t kv[(ENCODE && Tile<HD, P>::ROPE > 2 * Tile<HD, P>::STAGE)
                                ? Tile<HD, P>::ROPE
                                : 2 * Tile<HD, P>::STAGE];
    int seg_start[ENCODE ? 1 : kMaxSeg + 1];
    int seg_row[ENCODE ? 1 : kMaxSeg];
    int scan[ENCODE ? 1 : kThreads];
};

template <int HD, bool ENCODE, int P>
__global__ __launch_bounds__(kThreads, P == 1 ? 2 : 1) void attn_mfma_kernel(const AttnArgs a) {
    using TL = Tile<HD, P>;
    constexpr int kPairs = P;
    __shared__ Smem<HD, ENCODE, P> sm;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, half = lane >> 5;

    // block -> (q tile [longest first], unit, head slice, group); the group
    // is the fastest index so that one group's blocks share an XCD's L2.
    int bid = blockIdx.x;
    const int g = bid % a.n_kv_heads;
    bid /= a.n_kv_heads;
    const int hq = bid % a.n_hq;
    bid /= a.n_hq;
    const int unit = bid % a.n_units;
    const int jt = a.n_qt - 1 - bid / a.n_units;

    int q_len, q_row0, off, stream, pos0 = 0;
    const uint16_t* kbase;
    const uint16_t* vbase;
    int n_seg = 0, s_vis = 0, ctx_row0 = 0, tc = 0;
    if constexpr (ENCODE) {
        const int o = a.cu_len[unit];
        q_len = a.cu_len[unit + 1] - o;
        q_row0 = o;
        off = 0;
        stream = q_len;
        pos0 = a.pos_base ? a.pos_base[unit] : 0;
        kbase = a.k + ((size_t)g * a.k_rows + o) * HD;
        vbase = a.v + ((size_t)g * a.k_rows + o) * HD;
    } else {
        q_row0 = a.cu_q[unit];
        q_len = a.cu_q[unit + 1] - q_row0;
        ctx_row0 = a.cu_ctx[unit];
        tc = a.cu_ctx[unit + 1] - ctx_row0;
        kbase = a.k + (size_t)g * a.k_rows * HD;
        vbase = a.v + (size_t)g * a.k_rows * HD;
    }
    const int wg_rows = 32 * a.rbw;
    const int q_first = jt * wg_rows;
    if (q_first >= q_len) return;
    const int q_last = min(q_first + wg_rows, q_len) - 1;

    if constexpr (!ENCODE) {
        // Visible segments of this (request, layer, group): kept rows of the
        // routed resources, request order.  Exclusive scan of their lengths.
        const size_t e = ((size_t)unit * a.n_layers + a.layer) * a.n_kv_heads + g;
        const int r0 = a.route_off[e];
        n_seg = min(a.route_off[e + 1] - r0, kMaxSeg);
        int part = 0;
        int lens[4];
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
        int run = sm.scan[tid] - part;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int s = tid * 4 + i;
            if (s < n_seg) sm.seg_start[s] = run;
            run += lens[i];
        }
        s_vis = sm.scan[kThreads - 1];
        if (tid == 0) sm.seg_start[n_seg] = s_vis;
        off = s_vis + tc - q_len;
        stream = s_vis + tc;
        __syncthreads();
    }
    const int n_tiles = (off + q_last) / kBK + 1;

    // The (head, row block) pairs of this wave.
    int head[kPairs], my_q[kPairs], my_q_c[kPairs];
    bool store[kPairs];
#pragma unroll
    for (int j = 0; j < kPairs; ++j) {
        const int u = wave * kPairs + j;
        head[j] = g * a.ratio + hq * a.hpw + u % a.hpw;
        my_q[j] = q_first + (u / a.hpw) * 32 + l32;
        // rows outside [0, lse_rows) of q / out are never touched
        my_q_c[j] = max(0, min(min(my_q[j], q_len - 1), (int)a.lse_rows - 1 - q_row0));
        store[j] = my_q[j] < q_len && q_row0 + my_q[j] < a.lse_rows;
    }

    // ---- K / V tiles in LDS, both row-major [64 keys][HD] with the 16-byte
    // chunks of each row XOR-swizzled by the key's low four bits, double
    // buffered.
    constexpr int ROWB = HD * 2;
    constexpr int TILEB = kBK * ROWB;
    constexpr int STAGEB = 2 * TILEB;  // K tile, then V tile
    char* lds = reinterpret_cast<char*>(sm.kv);
    // XOR mask of a row's chunk index: for 256-byte rows the two 2-bit halves
    // of row % 16 are swapped, which keeps the 16 rows of an A-operand read on
    // 16 distinct chunks and puts the four rows of one transpose-read lane
    // group on four distinct 4-chunk groups (both bank-conflict free, as
    // measured with the LDS conflict counter).
    auto swz = [](int row, int chunk) -> uint32_t {
        const int m = TL::CPR == 16 ? (((row & 3) << 2) | ((row >> 2) & 3)) : (row % TL::CPR);
        return (uint32_t)(row * ROWB + ((chunk ^ m) << 4));
    };

    // Staging: thread owns keys kq*KPT + [0, KPT) at chunk c (coalesced rows).
    const int c = tid % TL::CPR;
    const int kq = tid / TL::CPR;
    uint32_t st_off[TL::KPT];
#pragma unroll
    for (int j = 0; j < TL::KPT; ++j) st_off[j] = swz(kq * TL::KPT + j, c);
    // S^T operand A = K rows: key l32 (+32 for the second block), chunk 2t + half.
    uint32_t k_rd[TL::NT];
#pragma unroll
    for (int t = 0; t < TL::NT; ++t) k_rd[t] = swz(l32, 2 * t + half);
    // O^T operand A = V^T via transpose reads.  In a 16-lane group G, lane i
    // receives element i % 4 of the 8-byte pieces addressed by lanes 4k + i / 4
    // (k = 0..3); pointing lane 4k + q at row r0 + k, column c0 + 4q hands lane
    // i the column c0 + i of four consecutive rows.  Rows s*16 + w*8 + half*4
    // + [0, 4) are the keys that the P^T operand holds in slots w*4 + [0, 4).
    uint32_t v_rd[TL::NDB][2];
    {
        const int G = lane >> 4, i = lane & 15;
#pragma unroll
        for (int db = 0; db < TL::NDB; ++db)
#pragma unroll
            for (int w = 0; w < 2; ++w) {
                const int row = w * 8 + (G >> 1) * 4 + (i >> 2);
                const int col = db * 32 + (G & 1) * 16 + (i & 3) * 4;
                v_rd[db][w] = TILEB + swz(row, col >> 3) + (col & 7) * 2;
            }
    }

    u32x4 kreg[TL::KPT], vreg[TL::KPT];
    // Prefill streams visit segments in order, so each thread keeps the index
    // of the segment holding its current row and only ever moves it forward.
    int sidx = 0;
    auto load_tile = [&](int kt) {
        const int p0 = kt * kBK + kq * TL::KPT;
#pragma unroll
        for (int j = 0; j < TL::KPT; ++j) {
            const int p = min(p0 + j, stream - 1);
            const uint16_t* kp;
            const uint16_t* vp;
            if constexpr (ENCODE) {
                kp = kbase + (size_t)p * HD;
                vp = vbase + (size_t)p * HD;
            } else if (p < s_vis) {
                while (sidx + 1 < n_seg && sm.seg_start[sidx + 1] <= p) ++sidx;
                const size_t row = min((size_t)(sm.seg_row[sidx] + (p - sm.seg_start[sidx])),
                                       (size_t)a.k_rows - 1);
                kp = kbase + row * HD;
                vp = vbase + row * HD;
            } else {
                const size_t row = min((size_t)ctx_row0 + (p - s_vis), (size_t)a.c_rows - 1);
                kp = a.ck + ((size_t)g * a.c_rows + row) * HD;
                vp = a.cv + ((size_t)g * a.c_rows + row) * HD;
            }
            kreg[j] = *reinterpret_cast<const u32x4*>(kp + c * 8);
            vreg[j] = *reinterpret_cast<const u32x4*>(vp + c * 8);
        }
    };
    auto store_tile = [&](char* stage) {
#pragma unroll
        for (int j = 0; j < TL::KPT; ++j) {
            *reinterpret_cast<u32x4*>(stage + st_off[j]) = kreg[j];
            *reinterpret_cast<u32x4*>(stage + TILEB + st_off[j]) = vreg[j];
        }
    };

    // Issue the first tile's loads, then the query loads, so that their
    // latencies overlap (and overlap the RoPE table set-up in encode).
    load_tile(0);

    // ---- Q fragments (B operand of S^T = K Q^T): for pair j the lane holds
    // row my_q[j], elements d = t*16 + half*8 + [0,8) for t < NT.
    bf16x8 qf[kPairs][TL::NT];
    {
        u32x4 raw[kPairs][TL::NT];
#pragma unroll
        for (int j = 0; j < kPairs; ++j) {
            const uint16_t* qrow = a.q + ((size_t)(q_row0 + my_q_c[j]) * a.n_q_heads + head[j]) * HD;
#pragma unroll
            for (int t = 0; t < TL::NT; ++t)
                raw[j][t] = *reinterpret_cast<const u32x4*>(qrow + t * 16 + half * 8);
        }
        if constexpr (ENCODE) {
            // RoPE at the resource-local position.  cos / sin for the block's
            // rows are computed once into LDS (in the tile buffers, before the
            // first tile arrives): row r, frequency f sits in 16-byte chunk
            // (f / 2) ^ (r % 16) of the row, so the 16 rows read by a lane
            // group fall on distinct banks.  Pairs (f, f + HD/2) are
            // (t, t + NT/2) in this lane.
            constexpr int HALF = HD / 2;
            char* tab = reinterpret_cast<char*>(sm.kv);
            for (int idx = tid; idx < wg_rows * HALF; idx += kThreads) {
                const int r = idx / HALF, f = idx % HALF;
                float sn, cs;
                sincos_rev_fast(rope_revolutions(pos0 + min(q_first + r, q_len - 1), a.rope.rev[f]),
                                &sn, &cs);
                *reinterpret_cast<float2*>(tab + r * (HALF * 8) + (((f >> 1) ^ (r & 15)) << 4) +
                                           (f & 1) * 8) = make_float2(cs, sn);
            }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kPairs; ++j) {
                const int r = my_q[j] - q_first;
                const char* trow = tab + r * (HALF * 8);
#pragma unroll
                for (int t = 0; t < TL::NT / 2; ++t) {
                    uint32_t lo[4], hi[4];
#pragma unroll
                    for (int w = 0; w < 4; ++w) {
                        const int f = t * 16 + half * 8 + w * 2;  // even: one chunk holds f, f + 1
                        const f32x4 k = *reinterpret_cast<const f32x4*>(trow + (((f >> 1) ^ (r & 15)) << 4));
                        float y1[2], y2[2];
#pragma unroll
                        for (int h2 = 0; h2 < 2; ++h2) {
                            const float cs = k[2 * h2], sn = k[2 * h2 + 1];
                            const float x1 = bf16_bits_to_f32((raw[j][t][w] >> (16 * h2)) & 0xffffu);
                            const float x2 =
                                bf16_bits_to_f32((raw[j][t + TL::NT / 2][w] >> (16 * h2)) & 0xffffu);
                            y1[h2] = x1 * cs - x2 * sn;
                            y2[h2] = x2 * cs + x1 * sn;
                        }
                        lo[w] = pack_bf16x2(y1[0], y1[1]);
                        hi[w] = pack_bf16x2(y2[0], y2[1]);
                    }
                    raw[j][t] = u32x4{lo[0], lo[1], lo[2], lo[3]};
                    raw[j][t + TL::NT / 2] = u32x4{hi[0], hi[1], hi[2], hi[3]};
                }
            }
            __syncthreads();  // the table area is reused by the first tile
        }
#pragma unroll
        for (int j = 0; j < kPairs; ++j)
#pragma unroll
            for (int t = 0; t < TL::NT; ++t) qf[j][t] = __builtin_bit_cast(bf16x8, raw[j][t]);
    }
    store_tile(lds);
    __syncthreads();

    const float sl2 = a.scale_log2;
    const float lazy = 8.0f / sl2;
    const bf16x2 ones2 = __builtin_bit_cast(bf16x2, 0x3F803F80u);  // (1.0, 1.0) in bf16
    float m[kPairs], lsum[kPairs];
    int lim[kPairs];
    f32x16 oacc[kPairs][TL::NDB];
#pragma unroll
    for (int j = 0; j < kPairs; ++j) {
        m[j] = -INFINITY;  // running max of raw logits for this lane's row
        lsum[j] = 0.f;     // this lane's partial sum of the (bf16-rounded) weights
        lim[j] = off + my_q[j];  // keys p <= lim are visible to this lane's row
#pragma unroll
        for (int db = 0; db < TL::NDB; ++db) oacc[j][db] = f32x16{};
    }

    auto tile = [&](auto stage_tag, int kt) {
        constexpr int cur = decltype(stage_tag)::value;
        const char* st = lds + cur * STAGEB;
        if (kt + 1 < n_tiles) load_tile(kt + 1);

        f32x16 sacc[kPairs][2];
#pragma unroll
        for (int j = 0; j < kPairs; ++j) sacc[j][0] = sacc[j][1] = f32x16{};
#pragma unroll
        for (int t = 0; t < TL::NT; ++t) {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const bf16x8 av = *reinterpret_cast<const bf16x8*>(st + k_rd[t] + kb * 32 * ROWB);
#pragma unroll
                for (int j = 0; j < kPairs; ++j)
                    sacc[j][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qf[j][t], sacc[j][kb], 0, 0, 0);
            }
        }
        const bool diag = kt * kBK + kBK - 1 > off + q_first;
        bf16x8 pf[kPairs][4];
#pragma unroll
        for (int j = 0; j < kPairs; ++j) {
            // causal / stream-end mask, only on tiles that reach past the first row's limit
            if (diag) {
                const int rem = lim[j] - kt * kBK - half * 4;  // key offsets above rem are masked
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        if (kb * 32 + (r >> 2) * 8 + (r & 3) > rem) sacc[j][kb][r] = -INFINITY;
            }
            float mt = fmaxf(sacc[j][0][0], sacc[j][0][1]);
#pragma unroll
            for (int r = 2; r < 16; ++r) mt = fmaxf(mt, sacc[j][0][r]);
#pragma unroll
            for (int r = 0; r < 16; ++r) mt = fmaxf(mt, sacc[j][1][r]);
            mt = pair_max(mt);
            // Lazy rescale: weights are taken relative to m, which only moves
            // when a logit exceeds it by more than 8 / sl2 (weights stay <=
            // 2^8, far from overflow); O and the row sum share m, so the
            // result is exact.
            if (__builtin_amdgcn_ballot_w64(mt > m[j] + lazy)) {
                const float m_new = fmaxf(m[j], mt);
                const float alpha = __builtin_amdgcn_exp2f((m[j] - m_new) * sl2);  // 0 when m == -inf
                lsum[j] *= alpha;
#pragma unroll
                for (int db = 0; db < TL::NDB; ++db) oacc[j][db] *= alpha;
                m[j] = m_new;
            }
            const float msl = m[j] * sl2;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                uint32_t w[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float p0 = __builtin_amdgcn_exp2f(fmaf(sacc[j][s >> 1][8 * (s & 1) + 2 * i], sl2, -msl));
                    const float p1 = __builtin_amdgcn_exp2f(fmaf(sacc[j][s >> 1][8 * (s & 1) + 2 * i + 1], sl2, -msl));
                    w[i] = pack_bf16x2(p0, p1);
                    // row sum of the weights as rounded for the P V product, so
                    // the output is an exact weighted mean of the V rows it used
                    lsum[j] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[i]), ones2,
                                                              lsum[j], false);
                }
                pf[j][s] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
            }
        }
#pragma unroll
        for (int db = 0; db < TL::NDB; ++db) {
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
                const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_s16x4*)(st + v_rd[db][0] + s * 16 * ROWB));
                const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_s16x4*)(st + v_rd[db][1] + s * 16 * ROWB));
                const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
                const bf16x8 av = __builtin_bit_cast(bf16x8, u32x4{l2[0], l2[1], h2[0], h2[1]});
#pragma unroll
                for (int j = 0; j < kPairs; ++j)
                    oacc[j][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pf[j][s], oacc[j][db], 0, 0, 0);
            }
        }
        if (kt + 1 < n_tiles) store_tile(lds + (cur ^ 1) * STAGEB);
        __syncthreads();
    };
    for (int kt = 0; kt < n_tiles; kt += 2) {
        tile(StageTag<0>{}, kt);
        if (kt + 1 < n_tiles) tile(StageTag<1>{}, kt + 1);
    }

#pragma unroll
    for (int j = 0; j < kPairs; ++j) {
        const float l = pair_sum(lsum[j]);
        if (store[j]) {
            const float inv = 1.0f / l;
            uint16_t* orow = a.out + ((size_t)(q_row0 + my_q[j]) * a.n_q_heads + head[j]) * HD;
#pragma unroll
            for (int db = 0; db < TL::NDB; ++db)
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4) {
                    const int d = db * 32 + r4 * 8 + half * 4;
                    const uint2 w = make_uint2(pack_bf16x2(oacc[j][db][r4 * 4 + 0] * inv, oacc[j][db][r4 * 4 + 1] * inv),
                                               pack_bf16x2(oacc[j][db][r4 * 4 + 2] * inv, oacc[j][db][r4 * 4 + 3] * inv));
                    *reinterpret_cast<uint2*>(orow + d) = w;
                }
            if (a.lse && half == 0)
                a.lse[(size_t)head[j] * a.lse_rows + q_row0 + my_q[j]] =
                    m[j] * sl2 * 0.69314718055994531f + logf(l);
        }
    }
}

}  // namespace

hipError_t launch_attn_mfma(const AttnArgs& a, bool encode, int head_dim, hipStream_t stream) {
    const long blocks = (long)a.n_qt * a.n_units * a.n_hq * a.n_kv_heads;
    if (blocks <= 0) return hipSuccess;
    if (blocks > 0x7fffffffL) return hipErrorInvalidValue;
    if (a.hpw * a.rbw != 4) return hipErrorInvalidValue;  // one pair per wave
    dim3 grid((unsigned)blocks), block(kThreads);
    if (head_dim == 128) {
        if (encode) hipLaunchKernelGGL((attn_mfma_kernel<128, true, 1>), grid, block, 0, stream, a);
        else hipLaunchKernelGGL((attn_mfma_kernel<128, false, 1>), grid, block, 0, stream, a);
    } else {
        if (encode) hipLaunchKernelGGL((attn_mfma_kernel<64, true, 1>), grid, block, 0, stream, a);
        else hipLaunchKernelGGL((attn_mfma_kernel<64, false, 1>), grid, block, 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace rc
