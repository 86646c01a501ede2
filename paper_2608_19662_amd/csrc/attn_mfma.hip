// bf16 flash attention on gfx950 MFMA, shared by
//   - resource encoding: block-diagonal causal attention inside each packed
//     resource, with RoPE at resource-local positions applied to the query
//     tile on load (ReCache Sec. 3, "Resource-Wise Attention"; Fig. 2(a));
//   - conversation prefill: queries over the kept rows of the resources routed
//     to their (layer, KV group), then causal context (final ReCache mask,
//     Fig. 2; Sec. 3, "Structural Pruning" / "Semantic Pruning").
//
// Both are one "key stream" per (unit, KV group): a query with local index i
// sees stream keys p <= off + i.  Encode: unit = resource, stream = [shared
// prefix rows, fully visible (Sec. 3: resource tokens see the shared prefix
// and their own tokens)] ++ [its own rows], off = P.  Prefill: unit =
// request, stream = [routed kept rows in request order] ++ [context rows],
// off = S_vis + Tc - Tq.  Both are a list of segments followed by a causal
// part, and share one code path.
//
// Work decomposition.  A workgroup is NW waves (4 in encode, 8 in prefill)
// that share one KV group and NW (query head, 32-row block) pairs of it (hpw
// heads x rbw row blocks, hpw the largest power of two up to NW dividing the
// group size); each wave owns one pair and computes the transposed products
//     S^T = K Q^T    (32x32x16 bf16 MFMA; A = K rows from LDS, B = Q^T in VGPRs)
//     O^T += V^T P^T (A = V^T from LDS, B = P^T straight from the S^T accumulators)
// so that each lane owns exactly one query row in both accumulators: row max
// and row sum need one cross-lane step (lanes l and l^32) and the rescale of
// O is lane-local.
//
// Pipeline.  K / V tiles of 64 keys go from HBM straight into LDS with the
// gfx950 global-to-LDS loads (no staging registers), double buffered, with K
// one tile ahead of V: while tile t's softmax runs on the VALU, the MFMAs of
// S(t+1) are already issued, so one wave keeps its matrix pipe busy during
// its own exponentials.  In LDS both tiles are row-major with an XOR swizzle
// of their 16-byte chunks (applied on the global side of the copy, since the
// copy places lane i at byte 16 i); V^T is read with the LDS transpose reads,
// in the key order in which the S^T accumulator hands P^T to the second
// product.
//
// Softmax.  Weights are formed against a reference max per row, set by the
// first tile and moved only when a weight could grow past 2^16, so that the
// common tile needs no row max before its exponentials.
//
// Output.  The normalised rows go through LDS and leave as whole rows, four
// 256-byte rows per 16-byte store instruction.  The lane index is not held
// across the loop, so that the registers spilled around the last tiles stay
// few.
//
// Tiles never cross a resource boundary in encode, and the reduction order
// depends only on local indices, so a resource's outputs are bit-identical
// wherever it is packed and whatever its neighbours are.
#include <utility>

#include "common.hpp"
#include "kernels.hpp"

namespace rc {

namespace {

// f(integral_constant<int, i>) for i = 0 .. N-1, unrolled at compile time.
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

constexpr int kBK = 64;  // keys per tile
// A lane's sum of a tile's weights above this moves the reference max.
constexpr float kWeightCap = 65536.0f;  // 2^16
constexpr int kMaxSeg = 1024;
// Third dword of a gfx9 buffer resource for raw (unformatted) loads.
constexpr int kBufferFlags = 0x00020000;

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

template <int HD, int NW>
struct Tile {
    static constexpr int CPR = HD / 8;           // 16-byte chunks per row
    static constexpr int ROWB = HD * 2;          // bytes per row
    static constexpr int TILEB = kBK * ROWB;     // bytes per K or V tile
    static constexpr int STAGEB = 2 * TILEB;     // K tile, then V tile
    static constexpr int RPI = 64 / CPR;         // rows per 1 KB wave copy
    static constexpr int RPW = kBK / NW;         // rows of a tile each wave copies
    static constexpr int NJ = RPW / RPI;         // copies per wave per tile
    static constexpr int NT = HD / 16;           // MFMA k-steps over head_dim
    static constexpr int NDB = HD / 32;          // 32-wide blocks of head_dim
    static_assert(NJ >= 1 && RPW % RPI == 0, "each wave copies whole 1 KB runs");
    static_assert(NW * 32 * ROWB <= 2 * STAGEB, "the output staging fits the K / V stages");
    static_assert(NW <= 8, "at most eight waves stage their output rows");
};

// Small per-lane index sets live in vector registers rather than arrays, so
// that selecting between two of them never turns into a stack access.
template <int N>
using u32v = uint32_t __attribute__((ext_vector_type(N)));
template <int N>
using u64v = uint64_t __attribute__((ext_vector_type(N)));

template <int C>
struct StageTag {
    static constexpr int value = C;
};

// The K / V tiles of the two stages are four separate LDS arrays (declared
// in the kernel): the compiler can then tell that the copies in flight into
// one of them do not touch the tiles being read, and issues no wait for the
// copies before those reads.
template <bool ENCODE, int NW>
struct Smem {
    int seg_start[ENCODE ? 2 : kMaxSeg + 1];
    int seg_row[ENCODE ? 2 : kMaxSeg];
    int scan[NW];  // wave totals of the segment-length scan
};

// XOR mask of a row's chunk index: for 256-byte rows the two 2-bit halves of
// row % 16 are swapped, which keeps the 16 rows of an A-operand read on 16
// distinct chunks and puts the four rows of one transpose-read lane group on
// four distinct 4-chunk groups (both bank-conflict free, as measured with the
// LDS conflict counter).
template <int CPR>
__device__ __forceinline__ int chunk_mask(int row) {
    return CPR == 16 ? (((row & 3) << 2) | ((row >> 2) & 3)) : (row % CPR);
}

template <int HD>
__device__ __forceinline__ uint32_t swz(int row, int chunk) {
    constexpr int CPR = HD / 8;
    return (uint32_t)(row * HD * 2 + ((chunk ^ chunk_mask<CPR>(row)) << 4));
}

__device__ __forceinline__ void wait_vm0() {
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0), expcnt / lgkmcnt unconstrained
}

// Rows a block is responsible for but cannot compute (its route list is
// longer than the segment table, or they lie past the query rows the grid
// was sized for): NaN in out and lse, so that a caller's size error shows in
// the outputs instead of leaving rows unwritten or dropping resources.
// Rows [r_begin, r_end) of unit rows starting at q_row0, heads
// [head0, head0 + n_heads).
template <int HD, int NW>
__device__ __forceinline__ void poison_rows(const AttnArgs& a, int head0, int n_heads, int q_row0,
                                         int r_begin, int r_end) {
    constexpr int CPR = HD / 8;
    const u32x4 nan8 = {0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u};  // bf16 NaNs
    const long n = (long)max(r_end - r_begin, 0) * n_heads * CPR;
    for (long i = threadIdx.x; i < n; i += NW * 64) {
        const int c = (int)(i % CPR);
        const long rest = i / CPR;
        const int h = head0 + (int)(rest % n_heads);
        const long row = (long)q_row0 + r_begin + rest / n_heads;
        if (row < 0 || row >= a.lse_rows) continue;
        *reinterpret_cast<u32x4*>(a.out + ((size_t)row * a.n_q_heads + h) * HD + c * 8) = nan8;
        if (c == 0 && a.lse) a.lse[(size_t)h * a.lse_rows + row] = __builtin_nanf("");
    }
}

// NW waves per block, each owning one (query head, 32-row block) pair of the
// block's KV group; two waves per SIMD either way (two 4-wave blocks or one
// 8-wave block per CU).
template <int HD, bool ENCODE, int NW>
__global__ __launch_bounds__(NW * 64, 8 / NW) void attn_mfma_kernel(const AttnArgs a) {
    using TL = Tile<HD, NW>;
    constexpr int kThreads = NW * 64;
    constexpr int ROWB = TL::ROWB, TILEB = TL::TILEB, STAGEB = TL::STAGEB;
    __shared__ Smem<ENCODE, NW> sm;
    __shared__ __attribute__((aligned(16))) char k_st0[TILEB], k_st1[TILEB], v_st0[TILEB], v_st1[TILEB];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: a scalar
    const int l32 = lane & 31, half = lane >> 5;

    // block -> (unit, head slice, q tile [longest first], group).  The group
    // is the fastest index, so the blocks of one group land on one XCD, and
    // the q tiles of a (unit, group) come next, so the blocks that run side
    // by side on an XCD stream the same keys through its L2.
    int bid = blockIdx.x;
    int g = bid % a.n_kv_heads;
    bid /= a.n_kv_heads;
    const int jt = a.n_qt - 1 - bid % a.n_qt;
    bid /= a.n_qt;
    const int hq = bid % a.n_hq;
    int unit = bid / a.n_hq;
    if constexpr (!ENCODE) {
        if (a.plan) {
            // Prefill with a work order: grid position (unit, g) takes the
            // pair the plan dealt there (longest first, the pairs of one
            // position balanced across positions, so across the XCDs).
            const int n_pairs = a.n_units * a.n_kv_heads;
            int p = a.plan[(size_t)a.layer * n_pairs + unit * a.n_kv_heads + g];
            p = min(max(p, 0), n_pairs - 1);  // in bounds whatever the plan holds
            unit = p / a.n_kv_heads;
            g = p % a.n_kv_heads;
        } else {
            // Without one, the group is rotated by the request, so that an
            // XCD serves every group over the requests rather than one group
            // throughout; routes give the groups unequal work, and this
            // evens out the XCDs' shares.
            g = (g + unit) % a.n_kv_heads;
        }
        // either way the blocks of one (request, group) share one XCD
    }

    int q_len, q_row0, off, stream, pos0 = 0;
    int n_seg = 0, s_vis = 0, ctx_row0 = 0, tc = 0;
    if constexpr (ENCODE) {
        const int o = a.cu_len[unit];
        q_len = a.cu_len[unit + 1] - o;
        q_row0 = o;
        pos0 = a.pos_base ? a.pos_base[unit] : 0;
        // Keys: the shared prefix (one fully visible segment, rows [0, P) of
        // the prefix cache in k / v), then the resource's own rows (in ck / cv).
        s_vis = a.p_len;
        n_seg = s_vis > 0 ? 1 : 0;
        ctx_row0 = o;
        tc = q_len;
    } else {
        q_row0 = a.cu_q[unit];
        q_len = a.cu_q[unit + 1] - q_row0;
        ctx_row0 = a.cu_ctx[unit];
        tc = a.cu_ctx[unit + 1] - ctx_row0;
    }
    const int wg_rows = 32 * a.rbw;
    const int q_first = jt * wg_rows;
    // the grid covers query rows [0, n_qt * wg_rows) of every unit; the block
    // of the last tile answers for any rows beyond
    if (jt == a.n_qt - 1 && q_len > a.n_qt * wg_rows) {
        poison_rows<HD, NW>(a, g * a.ratio + hq * a.hpw, a.hpw, q_row0, q_first, q_len);
        return;
    }
    if (q_first >= q_len) return;
    const int q_last = min(q_first + wg_rows, q_len) - 1;

    if constexpr (!ENCODE) {
        // Visible segments of this (request, layer, group): kept rows of the
        // routed resources, request order.  Exclusive scan of their lengths.
        const size_t e = ((size_t)unit * a.n_layers + a.layer) * a.n_kv_heads + g;
        const int r0 = a.route_off[e];
        n_seg = a.route_off[e + 1] - r0;
        if (n_seg > kMaxSeg) {
            poison_rows<HD, NW>(a, g * a.ratio + hq * a.hpw, a.hpw, q_row0, q_first, q_last + 1);
            return;
        }
        constexpr int SPT = kMaxSeg / kThreads;  // segments per thread
        int part = 0;
        int lens[SPT];
#pragma unroll
        for (int i = 0; i < SPT; ++i) {
            const int s = tid * SPT + i;
            lens[i] = 0;
            if (s < n_seg) {
                const int r = a.route_res[r0 + s];
                const int k0 = a.cu_kept[r];
                lens[i] = a.cu_kept[r + 1] - k0;
                sm.seg_row[s] = a.res_off ? a.res_off[(size_t)r * a.n_kv_heads + g] : k0;
            }
            part += lens[i];
        }
        int run = block_exclusive_scan<NW>(part, sm.scan, &s_vis);
#pragma unroll
        for (int i = 0; i < SPT; ++i) {
            const int s = tid * SPT + i;
            if (s < n_seg) sm.seg_start[s] = run;
            run += lens[i];
        }
        if (tid == 0) sm.seg_start[n_seg] = s_vis;
        __syncthreads();
    }
    off = s_vis + tc - q_len;
    stream = s_vis + tc;
    const int n_tiles = (off + q_last) / kBK + 1;

    const int head = g * a.ratio + hq * a.hpw + (wave % a.hpw);
    const int my_q = q_first + (wave / a.hpw) * 32 + l32;
    // rows outside [0, lse_rows) of q / out are never touched
    const int my_q_c = max(0, min(min(my_q, q_len - 1), (int)a.lse_rows - 1 - q_row0));

    // ---- HBM -> LDS copies.  Copy j of a wave moves rows wave*RPW + j*RPI +
    // [0, RPI) of a tile; lane i lands at byte 16 i of that run, i.e. row
    // rj = wave*RPW + j*RPI + i / CPR, physical chunk i % CPR, which holds
    // logical chunk (i % CPR) ^ mask(rj) of the key's row.
    // For 256-byte rows, rj % 4 = (i / 16) % 4 and (rj / 4) % 4 = (wave*RPW/4
    // + j) % 4, which is ((wave*RPW/4) % 4) ^ j: RPW is 16 or 8, so that term
    // is 0 or 2 and j < NJ <= 2 adds without a carry.  For 128-byte rows
    // rj % 8 = i / 8 whatever the wave and j (RPW and RPI are multiples of 8).
    static_assert(TL::CPR != 16 || (TL::RPW % 8 == 0 && TL::NJ <= 2) || TL::RPW % 16 == 0,
                  "copy j's chunk mask is copy 0's xor j");
    const int cp_lane_row = lane / TL::CPR;
    const int cp_chunk0 = (lane % TL::CPR) ^ chunk_mask<TL::CPR>(wave * TL::RPW + cp_lane_row);
    auto cp_chunk = [&](int j) { return TL::CPR == 16 ? (cp_chunk0 ^ j) : cp_chunk0; };
    // Where one tile comes from.  Every copy is a buffer load into LDS from
    // one of four planes: the group's segment rows (K and V; the shared
    // prefix in encode) and its causal rows (K and V; the resource's own rows
    // in encode), each addressed through a buffer resource.  Buffer loads are
    // bounds-checked (reads past a plane return zeros) and leave the
    // compiler's LDS wait counting exact, which the flat-address form of the
    // LDS copy does not.
    //
    // The stream is walked as "runs" of stream positions whose rows are
    // consecutive in one plane (one segment, or the whole causal part).  The
    // wave keeps the current run's end, the byte offset of stream position 0
    // in the run's plane (modulo 2^32) and the run's two resources, so a tile
    // inside the run costs a compare and an add: each copy takes the tile's
    // offset in a scalar register plus a per-lane constant.  Only a tile that
    // crosses the end of a run, or of the stream, takes per-lane offsets and
    // a flag per key for the plane it is in (one exec-masked load per plane).
    auto plane_k = [&](bool causal) {
        return causal ? __builtin_amdgcn_make_buffer_rsrc((void*)(a.ck + (size_t)g * a.c_rows * HD), (short)0,
                                                          (int)(a.c_rows * ROWB), kBufferFlags)
                      : __builtin_amdgcn_make_buffer_rsrc((void*)(a.k + (size_t)g * a.k_gstride * HD), (short)0,
                                                          (int)(a.k_rows * ROWB), kBufferFlags);
    };
    auto plane_v = [&](bool causal) {
        return causal ? __builtin_amdgcn_make_buffer_rsrc((void*)(a.cv + (size_t)g * a.c_rows * HD), (short)0,
                                                          (int)(a.c_rows * ROWB), kBufferFlags)
                      : __builtin_amdgcn_make_buffer_rsrc((void*)(a.v + (size_t)g * a.k_gstride * HD), (short)0,
                                                          (int)(a.k_rows * ROWB), kBufferFlags);
    };
    u32v<TL::NJ> lane_off;  // this lane's byte offset within a run of 64 rows
#pragma unroll
    for (int j = 0; j < TL::NJ; ++j)
        lane_off[j] = ((uint32_t)(wave * TL::RPW + j * TL::RPI + cp_lane_row) * HD + cp_chunk(j) * 8) * 2;
    // the current run (wave-uniform)
    int run_hi = 0;           // first stream position past the run (0: no run yet)
    bool run_causal = true;   // the run's plane: causal rows, or segment rows
    uint32_t run_off0 = 0;    // byte offset of stream position 0 in the run's plane, mod 2^32
    __amdgpu_buffer_rsrc_t run_k = plane_k(true), run_v = plane_v(true);
    // the tile being set up (wave-uniform, except the per-lane straddle data)
    bool t_fast = false;
    uint32_t t_off = 0;
    u32v<TL::NJ> voff = {};
    uint32_t in_ctx = 0;
    // Streams visit segments in order.  The wave keeps the segment of the
    // current run (u_*), each lane the segment of its current key for
    // straddling tiles (sidx, ...); both only move forward.
    int u_sidx = 0, u_hi = 0, u_dl = 0;
    int sidx = 0, seg_hi = 0, seg_dl = 0;
    if (n_seg > 0) {
        if constexpr (ENCODE) {
            u_hi = s_vis;  // the prefix: stream keys [0, P) are its rows [0, P)
        } else {
            u_hi = __builtin_amdgcn_readfirstlane(sm.seg_start[1]);
            u_dl = __builtin_amdgcn_readfirstlane(sm.seg_row[0]);
        }
        seg_hi = u_hi;
        seg_dl = u_dl;
    }
    auto key_ptrs = [&](int kt) {
        const int p0 = kt * kBK;
        if (p0 + kBK > run_hi) {
            // leave the current run: find the one containing p0
            if (p0 < s_vis) {
                while (p0 >= u_hi && u_sidx + 1 < n_seg) {
                    ++u_sidx;
                    u_hi = __builtin_amdgcn_readfirstlane(sm.seg_start[u_sidx + 1]);
                    u_dl = __builtin_amdgcn_readfirstlane(sm.seg_row[u_sidx]) -
                           __builtin_amdgcn_readfirstlane(sm.seg_start[u_sidx]);
                }
                if (run_causal) {  // entering the segment plane
                    run_causal = false;
                    run_k = plane_k(false);
                    run_v = plane_v(false);
                }
                run_hi = u_hi;
                run_off0 = (uint32_t)u_dl * ROWB;
            } else {
                run_hi = stream;  // (run_k / run_v start on the causal plane)
                if (!run_causal) {  // entering the causal plane
                    run_causal = true;
                    run_k = plane_k(true);
                    run_v = plane_v(true);
                }
                run_off0 = (uint32_t)(ctx_row0 - s_vis) * ROWB;
            }
        }
        t_fast = p0 + kBK <= run_hi;
        t_off = run_off0 + (uint32_t)p0 * ROWB;
        if (!t_fast) {
            static_for<TL::NJ>([&](auto jc) {
                constexpr int j = decltype(jc)::value;
                const int p = min(p0 + wave * TL::RPW + j * TL::RPI + cp_lane_row, stream - 1);
                uint32_t row;
                if (p < s_vis) {
                    while (p >= seg_hi && sidx + 1 < n_seg) {
                        ++sidx;
                        seg_hi = sm.seg_start[sidx + 1];
                        seg_dl = sm.seg_row[sidx] - sm.seg_start[sidx];
                    }
                    row = (uint32_t)(seg_dl + p);
                    in_ctx &= ~(1u << j);
                } else {
                    row = (uint32_t)(ctx_row0 + (p - s_vis));
                    in_ctx |= 1u << j;
                }
                voff[j] = row * ROWB + cp_chunk(j) * 16;
            });
        }
    };
    // (the offsets are passed as int, the builtin's parameter type: handed an
    // unsigned vector element, the host pass drops the kernel's launch stub)
    auto copy = [&](bool is_v, char* buf) {
        char* dst = buf + wave * TL::RPW * ROWB;
        if (t_fast) {
            const __amdgpu_buffer_rsrc_t r = is_v ? run_v : run_k;
#pragma unroll
            for (int j = 0; j < TL::NJ; ++j)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(dst + j * TL::RPI * ROWB), 16,
                                                         (int)lane_off[j], (int)t_off, 0, 0);
        } else {
            const __amdgpu_buffer_rsrc_t rs = is_v ? plane_v(false) : plane_k(false);
            const __amdgpu_buffer_rsrc_t rc = is_v ? plane_v(true) : plane_k(true);
#pragma unroll
            for (int j = 0; j < TL::NJ; ++j) {
                // The rows of one copy lie in one plane except where the
                // segments end and the causal rows begin (once per stream):
                // choose the resource on a wave-uniform test, and only that
                // rare mixed copy picks it per lane.
                const bool c = (in_ctx >> j) & 1;
                const uint64_t m = __builtin_amdgcn_ballot_w64(c);
                lds_void* d = (lds_void*)(dst + j * TL::RPI * ROWB);
                if (m == 0) {
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, d, 16, (int)voff[j], 0, 0, 0);
                } else if (m == __builtin_amdgcn_read_exec()) {
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, d, 16, (int)voff[j], 0, 0, 0);
                } else if (c) {
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, d, 16, (int)voff[j], 0, 0, 0);
                } else {
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, d, 16, (int)voff[j], 0, 0, 0);
                }
            }
        }
    };

    // Query rows first (they are needed first, for the RoPE), then the
    // prologue copies: K(0), V(0) into stage 0, K(1) into stage 1.  The
    // sources of tile 1 are kept for V(1) in the first loop iteration.
    u32x4 qraw[TL::NT];
    {
        const uint16_t* qrow = a.q + ((size_t)(q_row0 + my_q_c) * a.n_q_heads + head) * HD;
#pragma unroll
        for (int t = 0; t < TL::NT; ++t)
            qraw[t] = *reinterpret_cast<const u32x4*>(qrow + t * 16 + half * 8);
    }
    key_ptrs(0);
    copy(false, k_st0);
    copy(true, v_st0);
    if (n_tiles > 1) {
        key_ptrs(1);
        copy(false, k_st1);
    }

    // ---- Q fragment (B operand of S^T = K Q^T): lane holds row my_q, elements
    // d = t*16 + half*8 + [0,8) for t < NT.
    bf16x8 qf[TL::NT];
    {
        u32x4* raw = qraw;
        if constexpr (ENCODE) {
            // RoPE at the resource-local position; the pairs (f, f + HD/2) are
            // (t, t + NT/2) in this lane.  For blocks of 32 rows (4 heads) the
            // cos / sin of the block's rows are computed once into LDS, in the
            // V buffer of stage 1, which no copy touches before the loop: row
            // r, frequency f sits in 16-byte chunk (f / 2) ^ (r % 16) of the
            // row, so the 16 rows read by a lane group fall on distinct banks.
            // Larger blocks compute their lane's 32 frequencies directly.
            constexpr int HALF = HD / 2;
            const char* tab = v_st1;
            const bool use_tab = wg_rows <= 32;
            const int r = my_q - q_first;
            if (use_tab) {
                char* wtab = v_st1;
                for (int idx = tid; idx < wg_rows * HALF; idx += kThreads) {
                    const int rr = idx / HALF, f = idx % HALF;
                    float sn, cs;
                    sincos_rev_fast(rope_revolutions(pos0 + min(q_first + rr, q_len - 1), a.rope.rev[f]),
                                    &sn, &cs);
                    *reinterpret_cast<float2*>(wtab + rr * (HALF * 8) + (((f >> 1) ^ (rr & 15)) << 4) +
                                               (f & 1) * 8) = make_float2(cs, sn);
                }
                __syncthreads();
            }
            const int pos = pos0 + my_q_c;
#pragma unroll
            for (int t = 0; t < TL::NT / 2; ++t) {
                uint32_t lo[4], hi[4];
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const int f = t * 16 + half * 8 + w * 2;  // even: one chunk holds f, f + 1
                    float cs2[2], sn2[2];
                    if (use_tab) {
                        const f32x4 k = *reinterpret_cast<const f32x4*>(
                            tab + r * (HALF * 8) + (((f >> 1) ^ (r & 15)) << 4));
                        cs2[0] = k[0], sn2[0] = k[1], cs2[1] = k[2], sn2[1] = k[3];
                    } else {
#pragma unroll
                        for (int h2 = 0; h2 < 2; ++h2)
                            sincos_rev_fast(rope_revolutions(pos, a.rope.rev[f + h2]), &sn2[h2], &cs2[h2]);
                    }
                    float y1[2], y2[2];
#pragma unroll
                    for (int h2 = 0; h2 < 2; ++h2) {
                        const float x1 = bf16_bits_to_f32((raw[t][w] >> (16 * h2)) & 0xffffu);
                        const float x2 =
                            bf16_bits_to_f32((raw[t + TL::NT / 2][w] >> (16 * h2)) & 0xffffu);
                        // the rounding of the key rotation, written out
                        y1[h2] = fmaf(x1, cs2[h2], -(x2 * sn2[h2]));
                        y2[h2] = fmaf(x2, cs2[h2], x1 * sn2[h2]);
                    }
                    lo[w] = pack_bf16x2(y1[0], y1[1]);
                    hi[w] = pack_bf16x2(y2[0], y2[1]);
                }
                raw[t] = u32x4{lo[0], lo[1], lo[2], lo[3]};
                raw[t + TL::NT / 2] = u32x4{hi[0], hi[1], hi[2], hi[3]};
            }
        }
#pragma unroll
        for (int t = 0; t < TL::NT; ++t) qf[t] = __builtin_bit_cast(bf16x8, raw[t]);
    }

    // LDS read offsets.  S^T operand A = K rows: key l32 (+32 for the second
    // block), chunk 2t + half.
    // Chunk 2t + half of row l32 sits at k_rd0 ^ (t << 5): the mask only
    // permutes chunk bits, and t moves bits 1..3 of the chunk.
    const uint32_t k_rd0 = swz<HD>(l32, half);
    // O^T operand A = V^T via transpose reads.  In a 16-lane group G, lane i
    // receives element i % 4 of the 8-byte pieces addressed by lanes 4k + i / 4
    // (k = 0..3); pointing lane 4k + q at row r0 + k, column c0 + 4q hands lane
    // i the column c0 + i of four consecutive rows.  Rows s*16 + w*8 + half*4
    // + [0, 4) are the keys that the P^T operand holds in slots w*4 + [0, 4).
    // (db, w) = (0, 0) is computed; db moves chunk bits 2..3 and w moves the
    // row by 8 and, through the mask, chunk bit 1 (256-byte rows) or the row
    // by 8 only (128-byte rows, whose mask is row % 8).
    uint32_t v_rd0;
    {
        const int G = lane >> 4, i = lane & 15;
        const int row = (G >> 1) * 4 + (i >> 2);
        const int col = (G & 1) * 16 + (i & 3) * 4;
        v_rd0 = swz<HD>(row, col >> 3) + (col & 7) * 2;
    }
    auto v_rd = [&](int db, int w) -> uint32_t {
        return v_rd0 ^ (uint32_t)(db << 6) ^ (uint32_t)(w * (8 * ROWB + (TL::CPR == 16 ? 32 : 0)));
    };

    f32x16 sacc[2][2];  // S^T of two consecutive tiles, [tile & 1][key block]
    auto qk = [&](f32x16* acc, const char* st) {
        acc[0] = acc[1] = f32x16{};
#pragma unroll
        for (int t = 0; t < TL::NT; ++t)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const bf16x8 av = *reinterpret_cast<const bf16x8*>(st + (k_rd0 ^ (t << 5)) + kb * 32 * ROWB);
                acc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qf[t], acc[kb], 0, 0, 0);
            }
    };

    wait_vm0();
    __syncthreads();  // K(0), V(0), K(1) in LDS; RoPE table reads done
    qk(sacc[0], k_st0);
    __syncthreads();  // every wave has read K(0) before K(2) is copied over it

    const float sl2 = a.scale_log2;
    const bf16x2 ones2 = __builtin_bit_cast(bf16x2, 0x3F803F80u);  // (1.0, 1.0) in bf16
    float m = -INFINITY;   // reference max of raw logits for this lane's row (set by the first tile)
    float lsum = 0.f;      // this lane's partial sum of the (bf16-rounded) weights
    // keys p <= off + my_q are visible to this lane's row; this lane's S^T
    // entries of a tile start at key offset half * 4
    const int lim4 = off + my_q - half * 4;
    f32x16 oacc[TL::NDB];
#pragma unroll
    for (int db = 0; db < TL::NDB; ++db) oacc[db] = f32x16{};

    // One tile t: V(t + 1) and K(t + 2) copies start, tile t's softmax runs
    // beside the MFMAs of S(t + 1), then O += V(t)^T P(t)^T.
    auto tile = [&](auto stage_tag, auto next_tag, int kt) {
        constexpr int cur = decltype(stage_tag)::value;
        constexpr bool NEXT = decltype(next_tag)::value != 0;
        if constexpr (NEXT) copy(true, cur ? v_st0 : v_st1);
        if (kt + 2 < n_tiles) {
            key_ptrs(kt + 2);
            copy(false, cur ? k_st1 : k_st0);
        }
        f32x16* sc = sacc[cur];
        // causal / stream-end mask, only on tiles that reach past the first row's limit
        if (kt * kBK + kBK - 1 > off + q_first) {
            const int rem = lim4 - kt * kBK;  // key offsets above rem are masked
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (kb * 32 + (r >> 2) * 8 + (r & 3) > rem) sc[kb][r] = -INFINITY;
        }
        auto row_max = [&]() {
            float mt = fmaxf(sc[0][0], sc[0][1]);
#pragma unroll
            for (int r = 2; r < 16; ++r) mt = fmaxf(mt, sc[0][r]);
#pragma unroll
            for (int r = 0; r < 16; ++r) mt = fmaxf(mt, sc[1][r]);
            return pair_max(mt);
        };
        // the first tile sets the reference m (O and the row sum are still 0)
        if (kt == 0) m = row_max();
        // S(t + 1) on the matrix pipe while the weights of tile t are formed.
        if constexpr (NEXT) qk(sacc[cur ^ 1], cur ? k_st0 : k_st1);
        // Weights relative to the reference m as it stands (no max of the
        // tile first), with this lane's sum of them as rounded for the P V
        // product, so that the output is an exact weighted mean of the V rows
        // it used.
        bf16x8 pf[4];
        float tsum;
        auto weights = [&]() {
            const float msl = m * sl2;
            tsum = 0.f;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                uint32_t w[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float p0 = __builtin_amdgcn_exp2f(fmaf(sc[s >> 1][8 * (s & 1) + 2 * i], sl2, -msl));
                    const float p1 = __builtin_amdgcn_exp2f(fmaf(sc[s >> 1][8 * (s & 1) + 2 * i + 1], sl2, -msl));
                    w[i] = pack_bf16x2(p0, p1);
                    tsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[i]), ones2, tsum, false);
                }
                pf[s] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
            }
        };
        weights();
        if constexpr (NEXT) {
            // Interleave: K reads two MFMAs ahead, then each MFMA of S(t + 1)
            // followed by an equal share of the ~96 VALU instructions that
            // form tile t's weights, so the matrix pipe and the VALU overlap
            // within this wave.
            constexpr int NM = 2 * TL::NT, VPM = 96 / NM;
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
            for (int i = 0; i < NM; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, VPM, 0);
                if (i + 2 < NM) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        // The reference m stays until a weight could exceed 2^16, which
        // shows as a lane's sum of them above that (or not finite, for a
        // logit more than 128 / sl2 above m).  Then m becomes the larger of
        // m and the tile's row max, O and the row sum are rescaled by the
        // change, and the tile's weights are formed again (each at most 1
        // now).  O and the row sum always share m, so the result is exact
        // whatever m is.
        if (__builtin_expect(__builtin_amdgcn_ballot_w64(!(tsum <= kWeightCap)) != 0, 0)) {
            const float m_new = fmaxf(m, row_max());
            const float alpha = __builtin_amdgcn_exp2f((m - m_new) * sl2);
            lsum *= alpha;
#pragma unroll
            for (int db = 0; db < TL::NDB; ++db) oacc[db] *= alpha;
            m = m_new;
            weights();
        }
        lsum += tsum;
        const char* st = cur ? v_st1 : v_st0;
#pragma unroll
        for (int db = 0; db < TL::NDB; ++db) {
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_s16x4*)(st + v_rd(db, 0) + s * 16 * ROWB));
                const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_s16x4*)(st + v_rd(db, 1) + s * 16 * ROWB));
                const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
                const bf16x8 av = __builtin_bit_cast(bf16x8, u32x4{l2[0], l2[1], h2[0], h2[1]});
                oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pf[s], oacc[db], 0, 0, 0);
            }
        }
        {
            // transpose reads run four MFMAs ahead of their product
            constexpr int NM = 4 * TL::NDB;
            __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
            for (int i = 0; i < NM; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                if (i + 4 < NM) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            }
        }
        if constexpr (NEXT) {
            wait_vm0();
            __syncthreads();  // V(t + 1), K(t + 2) in LDS; stage cur free again
        }
    };
    int kt = 0;
    for (; kt + 2 < n_tiles; kt += 2) {
        tile(StageTag<0>{}, StageTag<1>{}, kt);
        tile(StageTag<1>{}, StageTag<1>{}, kt + 1);
    }
    if (kt + 1 < n_tiles) {
        tile(StageTag<0>{}, StageTag<1>{}, kt);
        tile(StageTag<1>{}, StageTag<0>{}, kt + 1);
    } else {
        tile(StageTag<0>{}, StageTag<0>{}, kt);
    }

    const float l = pair_sum(lsum);
    // Output through LDS: each wave writes its 32 normalised rows there
    // (16-byte chunks swizzled by row), then stores whole rows with 16-byte
    // stores, so every store instruction fills complete lines.
    __syncthreads();  // every wave is done with the K / V stages
    {
        // lane-derived values again, from the lane counter rather than kept
        // in registers across the loop
        const int ln = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
        const int row = ln & 31, hf = ln >> 5;  // this lane's row, and which half of it
        constexpr int CPR = TL::CPR;
        // two waves' 32 rows per K / V tile array
        static_assert(TILEB == 2 * 32 * ROWB, "two waves stage their rows in one tile array");
        const int wb = wave >> 1;
        char* ob = (wb == 0 ? k_st0 : wb == 1 ? v_st0 : wb == 2 ? k_st1 : v_st1) + (wave & 1) * 32 * ROWB;
        const float inv = 1.0f / l;
#pragma unroll
        for (int db = 0; db < TL::NDB; ++db)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const int c = db * 4 + r4;  // 16-byte chunk of the row
                const uint2 w = make_uint2(pack_bf16x2(oacc[db][r4 * 4 + 0] * inv, oacc[db][r4 * 4 + 1] * inv),
                                           pack_bf16x2(oacc[db][r4 * 4 + 2] * inv, oacc[db][r4 * 4 + 3] * inv));
                *reinterpret_cast<uint2*>(ob + row * ROWB + ((c ^ (row % CPR)) << 4) + hf * 8) = w;
            }
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
        __builtin_amdgcn_wave_barrier();
        constexpr int RPS = 64 / CPR;  // rows per store instruction
        const int q_base = q_first + (wave / a.hpw) * 32;
#pragma unroll
        for (int it = 0; it < 32 / RPS; ++it) {
            const int r = it * RPS + ln / CPR, c = ln % CPR;
            const u32x4 v = *reinterpret_cast<const u32x4*>(ob + r * ROWB + ((c ^ (r % CPR)) << 4));
            const int q = q_base + r;
            if (q < q_len && q_row0 + q < a.lse_rows)
                *reinterpret_cast<u32x4*>(a.out + ((size_t)(q_row0 + q) * a.n_q_heads + head) * HD + c * 8) = v;
        }
        const int q = q_base + row;
        if (a.lse && hf == 0 && q < q_len && q_row0 + q < a.lse_rows)
            a.lse[(size_t)head * a.lse_rows + q_row0 + q] = m * sl2 * 0.69314718055994531f + logf(l);
    }
}

}  // namespace

namespace {

// Waves per block of each mode: encode's blocks are short (a few tiles per
// resource), so two 4-wave blocks per CU overlap one block's prologue with
// the other's loop; prefill streams long key lists, where one 8-wave block
// per CU copies each K / V tile once for twice the query rows.
constexpr int kEncodeWaves = 4;
constexpr int kAttendWaves = 8;

// A block covers NW (query head, 32-row block) pairs of one KV group: hpw
// heads x rbw row blocks, hpw the largest power of two up to NW dividing the
// group size, so every head of the group is covered exactly once.
template <int NW>
int block_rows(int ratio) {
    int h = NW;
    while (ratio % h) h >>= 1;
    return 32 * (NW / h);
}

template <int NW>
void set_tiling(AttnArgs& b) {
    int h = NW;
    while (b.ratio % h) h >>= 1;
    b.hpw = h;
    b.rbw = NW / h;
    b.n_hq = b.ratio / h;
    b.n_qt = (b.max_rows + 32 * b.rbw - 1) / (32 * b.rbw);
}

template <int HD, bool ENCODE, int NW>
hipError_t launch(const AttnArgs& a, hipStream_t stream) {
    AttnArgs b = a;
    set_tiling<NW>(b);
    const long blocks = (long)b.n_qt * b.n_units * b.n_hq * b.n_kv_heads;
    if (blocks <= 0) return hipSuccess;
    if (blocks > 0x7fffffffL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((attn_mfma_kernel<HD, ENCODE, NW>), dim3((unsigned)blocks), dim3(NW * 64), 0,
                       stream, b);
    return hipGetLastError();
}

}  // namespace

int attend_block_rows(int ratio) { return ratio >= 1 ? block_rows<kAttendWaves>(ratio) : 0; }

hipError_t launch_attn_mfma(const AttnArgs& a, bool encode, int head_dim, hipStream_t stream) {
    if (a.ratio < 1 || a.max_rows < 1) return hipErrorInvalidValue;
    if (head_dim == 128)
        return encode ? launch<128, true, kEncodeWaves>(a, stream)
                      : launch<128, false, kAttendWaves>(a, stream);
    return encode ? launch<64, true, kEncodeWaves>(a, stream)
                  : launch<64, false, kAttendWaves>(a, stream);
}

}  // namespace rc
