// Argument blocks and launchers of the gfx950 kernels.  The C-ABI layer
// (api.hip) validates every scalar before it fills these and launches.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "common.hpp"

namespace rc {

// bf16 MFMA flash attention (encode or conversation prefill).
struct AttnArgs {
    // decomposition: blocks = n_qt * n_units * n_hq * n_kv_heads; the
    // launcher fills hpw, rbw, n_hq and n_qt from ratio and max_rows
    int n_q_heads, n_kv_heads, ratio;
    int hpw;      // query heads per block (largest power of two <= waves dividing ratio)
    int rbw;      // 32-row blocks per block (waves / hpw: one (head, row block) pair per wave)
    int n_hq;     // blocks per group along heads (ratio / hpw)
    int n_units;  // resources (encode) or requests (prefill)
    int n_qt;     // query tiles per unit (ceil(max_rows / (32 * rbw)))
    float scale_log2;  // softmax_scale * log2(e)
    const uint16_t* q;
    uint16_t* out;
    float* lse;
    long lse_rows;      // rows of q / out / lse (total_T or total_q); bounds every row index
    // Segments (encode: the shared prefix cache, rows [0, p_len); prefill:
    // kept resource rows) and the causal part (encode: the resources' rotated
    // K / V caches; prefill: conversation context), all [n_kv_heads][rows][d].
    const uint16_t* k;
    const uint16_t* v;
    long k_rows;        // rows of one KV head's part of k / v (all rows with res_off)
    long k_gstride;     // rows between KV heads in k / v (0 with res_off)
    const uint16_t* ck;
    const uint16_t* cv;
    long c_rows;        // rows per KV head in ck / cv
    // encode
    const int32_t* cu_len;
    const int32_t* pos_base;
    int p_len;          // shared prefix rows (0: none)
    RopeRev rope;
    // prefill
    const int32_t* cu_q;
    const int32_t* cu_ctx;
    int layer, n_layers;
    const int32_t* route_off;
    const int32_t* route_res;
    const int32_t* cu_kept;
    const int32_t* res_off;  // route-compacted store rows [n_res * Hkv], or NULL
    int max_rows;            // query rows of the longest unit (the grid covers no more)
    const int32_t* plan;     // prefill: work order of the (request, group) pairs
                             // [n_layers][n_units * n_kv_heads], or NULL
};
hipError_t launch_attn_mfma(const AttnArgs& a, bool encode, int head_dim, hipStream_t stream);
// Query rows of one prefill block (32 per row block) for a group size.
int attend_block_rows(int ratio);

// fp32 reference-precision attention (encode or conversation attend).
struct AttnF32Args {
    int n_q_heads, n_kv_heads, ratio, head_dim;
    int n_units, max_rows;  // grid: max_rows x n_units x n_q_heads waves
    float scale;
    const float* q;
    float* out;
    float* lse;
    long lse_rows;
    const float* k;
    const float* v;
    long k_rows;
    long k_gstride;
    const float* ck;
    const float* cv;
    long c_rows;
    const int32_t* cu_len;
    const int32_t* pos_base;
    int p_len;  // encode: shared prefix rows in k / v; own rows in ck / cv
    RopeRev rope;
    const int32_t* cu_q;
    const int32_t* cu_ctx;
    int layer, n_layers;
    const int32_t* route_off;
    const int32_t* route_res;
    const int32_t* cu_kept;
    const int32_t* res_off;
};
hipError_t launch_attn_f32(const AttnF32Args& a, bool encode, hipStream_t stream);

// RoPE + cache write / in-place RoPE.
struct RopeArgs {
    int T, n_heads, head_dim, dtype;  // dtype: 0 f32, 1 bf16
    const int32_t* pos;               // explicit positions [T], or NULL with cu_len
    const int32_t* cu_len;            // resource-local positions from packing offsets
    const int32_t* pos_base;
    int n_res;
    RopeRev rope;
    const void* x;  // source [T][H][d]
    void* y;        // rotated destination: in place ([T][H][d]) or cache ([H][rows][d])
    const void* v;  // optional value copy source [T][H][d]
    void* v_dst;    // value cache [H][rows][d]
    long cache_rows;
    int row0;
    int to_cache;  // 1: write head-major caches at row0 + t
};
hipError_t launch_rope(const RopeArgs& a, hipStream_t stream);

// Kept-row gather.
hipError_t launch_prune_gather(int elem_bytes, int n_res, const int32_t* cu_len,
                               const int32_t* cu_kept, const int32_t* kept_idx, long total_T,
                               long total_kept, int n_kv_heads, int head_dim, const void* k_cache,
                               const void* v_cache, void* k_kept, void* v_kept, hipStream_t s);

// Route-compacted store: row tables for every layer, then one layer's rows.
hipError_t launch_store_offsets(int n_res, int n_layers, int n_kv_heads, const uint8_t* mask,
                                const int32_t* cu_kept, int32_t* store_off, hipStream_t s);
hipError_t launch_store_routes(int elem_bytes, int layer, int n_res, const int32_t* cu_len,
                               const int32_t* cu_kept, const int32_t* kept_idx, long total_T,
                               long total_kept, int n_kv_heads, int head_dim,
                               const int32_t* store_off, long store_rows, const void* k_cache,
                               const void* v_cache, void* k_store, void* v_store, hipStream_t s);

// Route CSR build.
hipError_t launch_build_routes(int n_req, const int32_t* req_res_off, const int32_t* req_res,
                               int n_res, int n_layers, int n_kv_heads, const uint8_t* mask,
                               const int32_t* cu_kept, int32_t* route_off, int32_t* route_res,
                               int32_t* route_tokens, hipStream_t s);

// Split-KV decode (one query per request) and its LSE merge.
struct DecodeArgs {
    int n_req, n_q_heads, n_kv_heads, ratio, head_dim, n_splits;
    float scale_log2;
    const uint16_t* q;
    uint16_t* out;
    float* lse;
    long lse_rows;
    const uint16_t* rk;
    const uint16_t* rv;
    long r_rows;     // rows of one KV head's part of rk / rv (all rows with res_off)
    long r_gstride;  // rows between KV heads in rk / rv (0 with res_off)
    const uint16_t* ck;
    const uint16_t* cv;
    long c_rows;
    const int32_t* cu_q;
    const int32_t* cu_ctx;
    int layer, n_layers;
    const int32_t* route_off;
    const int32_t* route_res;
    const int32_t* cu_kept;
    const int32_t* res_off;  // route-compacted store rows [n_res * Hkv], or NULL
    float* ws_o;   // [n_req][Hq][n_splits][head_dim]
    float* ws_ml;  // [n_req][Hq][n_splits][2]  (max in log2 units, sum)
    const int32_t* plan;  // work order of the (request, group) pairs, or NULL
};
hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream);
size_t decode_workspace_bytes(int n_req, int n_q_heads, int head_dim, int n_splits);
int decode_splits(int n_req, int n_kv_heads, int max_kv);

// Work order of the attend kernels (plan.hip): per layer, the pairs
// b * n_kv_heads + g sorted by their work, longest first, dealt in snake order
// over the n_kv_heads grid positions.
constexpr int kMaxPlanPairs = 8192;  // n_req * n_kv_heads per plan (sorted in LDS)
constexpr int kPlanBlockCost = 3;    // fixed cost of a block, in 64-key tiles
struct PlanArgs {
    int n_req, n_layers, n_kv_heads;
    int wg_rows;  // query rows per prefill block (attend_block_rows)
    const int32_t* cu_q;
    const int32_t* cu_ctx;
    const int32_t* route_tokens;  // [n_req][n_layers][n_kv_heads]
    int32_t* plan;                // [n_layers][n_req * n_kv_heads]
};
hipError_t launch_attend_plan(const PlanArgs& a, hipStream_t stream);

}  // namespace rc
