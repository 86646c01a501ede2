/*
 * recache.h -- C ABI of the MI355X (gfx950) resource-wise attention library.
 *
 * ReCache (arXiv 2608.19662) encodes each retrieved resource (a tool or skill
 * schema) as an independent KV block and lets conversation tokens read those
 * blocks only through selected (layer, KV group) routes and only at retained
 * token positions.  This library implements that data path on one GPU:
 *
 *   recache_rope_q / recache_rope_kv   RoPE at explicit positions; K/V cache write
 *   recache_encode_resources           block-diagonal causal encode (Sec. 3,
 *                                      "Resource-Wise Attention"; Fig. 2(a))
 *   recache_encode_attention           its attention half, on built caches
 *   recache_prune_gather               kept-token compaction (Sec. 3,
 *                                      "Semantic Pruning"; Fig. 2(c))
 *   recache_build_routes               per (request, layer, KV group) visible
 *                                      resource lists (Sec. 3, "Structural
 *                                      Pruning"; Fig. 2(b))
 *   recache_route_store_offsets /      a resource store holding only visible
 *   recache_store_routes               routes at kept positions (both pruning
 *                                      stages; the memory it saves)
 *   recache_attend_cached              conversation queries over routed, kept
 *                                      resource rows plus causal context (final
 *                                      ReCache mask, Fig. 2)
 *   recache_select_routes              [host] Omega* = L* x G* from contribution
 *                                      scores, with sparsity and coverage
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers are DEVICE pointers unless a parameter is marked [host].  The
 *   caller owns every buffer; the library allocates no device memory, keeps no
 *   pointer after returning and holds no state besides a thread-local error
 *   string.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *   device work is enqueued on it; nothing synchronises.
 * - Scalar arguments are validated on the host before any launch.  On a
 *   non-zero return no kernel has been launched and no output was written
 *   (except RECACHE_EHIP, which reports a launch failure).
 *   recache_last_error() returns the text for the last non-OK status of the
 *   calling thread.
 * - Device index arrays (offsets, kept lists, route lists, store tables) are
 *   trusted by the kernels: pass them through recache_check_offsets /
 *   recache_check_kept on a host copy when they come from an untrusted source.
 *   Kernels clamp every row address of Q, K, V, O and the caches to the extents
 *   given as scalars, so bad row indices give wrong numbers, not accesses
 *   outside those buffers.  The index arrays must agree with each other (route
 *   lists and store tables as recache_build_routes and
 *   recache_route_store_offsets write them), since one is read at positions
 *   another names.
 * - Element types: RECACHE_F32 (float) or RECACHE_BF16 (bfloat16); all
 *   floating tensors of one call share the dtype.  bf16 math accumulates in
 *   fp32; outputs are rounded to nearest even.  head_dim is 64 or 128.
 * - The bf16 encode and prefill kernels address each KV plane (one KV head's
 *   rows of a cache or of the context, a layer's route-compacted store)
 *   through 32-bit byte offsets: a plane of 4 GiB or more (16.7M rows at
 *   head_dim 128) is RECACHE_EUNSUPPORTED.
 * - Layouts: token-major tensors are [rows][heads][head_dim]; KV caches are
 *   head-major [kv_heads][cache_rows][head_dim], so the rows of one resource
 *   (or one request's context) for one KV group are contiguous.  GQA: query
 *   head h reads KV head h / (n_q_heads / n_kv_heads).
 * - RoPE pairs element i with element i + head_dim/2 ("rotate half"), with
 *   theta_i = rope_base^(-2i/head_dim); angles are reduced in fp64.
 * - softmax_scale <= 0 selects 1/sqrt(head_dim).  LSE outputs are natural-log
 *   sum-exp of the scaled logits, fp32, [n_q_heads][rows].
 */
#ifndef RECACHE_H
#define RECACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum recache_status {
    RECACHE_OK = 0,
    RECACHE_EINVAL = -1,       /* bad argument: null pointer, bad size, Tq > Tc, ... */
    RECACHE_EUNSUPPORTED = -2, /* valid but not implemented: head_dim, dtype, GQA ratio */
    RECACHE_EWORKSPACE = -3,   /* workspace missing or smaller than required */
    RECACHE_EHIP = -4          /* a HIP call failed (launch error, bad device pointer) */
};

enum recache_dtype { RECACHE_F32 = 0, RECACHE_BF16 = 1 };

/* Library version: major * 10000 + minor * 100 + patch. */
int recache_version(void);

/* Text of the last non-OK status returned on this thread ("" if none). */
const char* recache_last_error(void);

/*
 * RoPE in place on x[T][n_heads][head_dim] at positions pos[T] (device int32).
 * Used for conversation queries, whose positions continue the original
 * sequence (Sec. 3, "Resource-Wise Attention": the surrounding context keeps
 * its positional encodings).
 */
int recache_rope_q(int dtype, int T, int n_heads, int head_dim, double rope_base,
                   const int32_t* pos, void* x, void* stream);

/*
 * Rotate k[T][n_kv_heads][head_dim] at pos[T] and write it to
 * k_cache[g][row0 + t][:]; copy v[T][n_kv_heads][head_dim] to
 * v_cache[g][row0 + t][:].  Caches are [n_kv_heads][cache_rows][head_dim];
 * requires 0 <= row0 and row0 + T <= cache_rows.  This is the cache
 * construction step of Sec. 3, "Resource-Wise Attention": each resource's
 * keys are rotated at local indices assigned while its cache is built
 * (pos = j for token j), and the surrounding context keeps its original
 * positions (pass them in pos).  Used to append conversation K/V and, inside
 * recache_encode_resources, resource K/V at resource-local positions.
 * Errors: RECACHE_EINVAL for T < 0, rows outside the cache, a null pointer or
 * rope_base <= 1; RECACHE_EUNSUPPORTED for dtype / head_dim.
 */
int recache_rope_kv(int dtype, int T, int n_kv_heads, int head_dim, double rope_base,
                    const int32_t* pos, const void* k, const void* v,
                    void* k_cache, void* v_cache, int cache_rows, int row0, void* stream);

/*
 * One layer of resource encoding (Sec. 3, "Resource-Wise Attention";
 * Fig. 2(a)).  n_res resources are packed in order: resource r owns rows
 * [cu_len[r], cu_len[r+1]) (device int32, cu_len[0] = 0, every length >= 1,
 * cu_len[n_res] = total_T, every length <= max_len: see
 * recache_check_encode_lengths; a resource longer than max_len gets NaN rows
 * instead of outputs).  Token j of resource r
 * gets position pos_base[r] + j (pos_base device int32 [n_res], or NULL for
 * 0: resource-local positions, pos(t_ij) = j).
 *
 * Optional shared prefix (the instruction every resource is encoded after,
 * Sec. 3: resource tokens attend the shared prefix and their own tokens):
 * prefix_len rows of an already rotated cache, prefix_k/prefix_v
 * [n_kv_heads][prefix_len][head_dim] (device; NULL when prefix_len is 0).
 * With a prefix, pos_base[r] = prefix_len places every resource right after
 * it; pos_base[r] = prefix_len + (tokens before r) gives the original global
 * positions ("Block").
 *
 * Query row t of resource r, head h, attends every prefix row and keys u in
 * [cu_len[r], t] of KV head h / (Hq / Hkv): no attention crosses resources,
 * so each resource's outputs and cache rows do not depend on its neighbours
 * or on its packing offset (bit-exact on the GPU).
 *
 *   q[total_T][n_q_heads][head_dim], k/v[total_T][n_kv_heads][head_dim]: inputs
 *   out[total_T][n_q_heads][head_dim]: attention output
 *   k_cache/v_cache[n_kv_heads][total_T][head_dim]: rotated K and plain V,
 *       the resource KV blocks to keep for reuse
 *   lse[n_q_heads][total_T] (fp32) or NULL
 * Errors: RECACHE_EINVAL also for prefix_len < 0 or a missing prefix pointer.
 */
int recache_encode_resources(int dtype, int n_res, const int32_t* cu_len, int total_T,
                             int max_len, int n_q_heads, int n_kv_heads, int head_dim,
                             double rope_base, const int32_t* pos_base, int prefix_len,
                             const void* prefix_k, const void* prefix_v, float softmax_scale,
                             const void* q, const void* k, const void* v, void* out,
                             void* k_cache, void* v_cache, float* lse, void* stream);

/*
 * The attention half of recache_encode_resources on caches that already hold
 * the rotated keys and the values of the packed resources
 * (k_cache/v_cache[n_kv_heads][total_T][head_dim], e.g. written by
 * recache_rope_kv at positions pos_base[r] + j).  Queries are rotated on the
 * fly at the same positions.  Same arguments and outputs otherwise;
 * recache_encode_resources = recache_rope_kv + this call.
 */
int recache_encode_attention(int dtype, int n_res, const int32_t* cu_len, int total_T,
                             int max_len, int n_q_heads, int n_kv_heads, int head_dim,
                             double rope_base, const int32_t* pos_base, int prefix_len,
                             const void* prefix_k, const void* prefix_v, float softmax_scale,
                             const void* q, const void* k_cache, const void* v_cache, void* out,
                             float* lse, void* stream);

/*
 * Semantic-pruning gather, one layer (Sec. 3, "Semantic Pruning"): resource r
 * keeps local token indices kept_idx[cu_kept[r] .. cu_kept[r+1]) (device
 * int32, strictly ascending, inside [0, D_r), at least one per resource;
 * cu_kept[n_res] = total_kept).  Kept rows are copied bit for bit, so they
 * keep the rotation they got at construction:
 *   k_kept[g][cu_kept[r] + j] = k_cache[g][cu_len[r] + kept_idx[cu_kept[r] + j]]
 * and the same for v.  Caches are [n_kv_heads][total_T][head_dim], outputs
 * [n_kv_heads][total_kept][head_dim].
 */
int recache_prune_gather(int dtype, int n_res, const int32_t* cu_len, const int32_t* cu_kept,
                         const int32_t* kept_idx, int total_T, int total_kept, int n_kv_heads,
                         int head_dim, const void* k_cache, const void* v_cache, void* k_kept,
                         void* v_kept, void* stream);

/*
 * Structural-pruning routes for every (request, layer, KV group) (Sec. 3,
 * "Structural Pruning"): route_mask[r][l][g] (device uint8, non-zero = the
 * route (l, g) of resource r is in Omega and exposes its states) generalises
 * the paper's Omega* = L* x G* to a per-resource mask.  Request b lists
 * resources req_res[req_res_off[b] .. req_res_off[b+1]) (device int32,
 * request order, ids in [0, n_res); req_res_off[n_req] = total_req_res).
 *
 * For entry e = (b * n_layers + l) * n_kv_heads + g the outputs are
 *   route_res[route_off[e] .. route_off[e+1]): the listed resources of b whose
 *       bit (l, g) is set, in request order;
 *   route_tokens[e]: the sum of their kept lengths, cu_kept[r+1] - cu_kept[r].
 * route_off has n_req * n_layers * n_kv_heads + 1 entries (route_off[0] = 0);
 * route_res needs room for total_req_res * n_layers * n_kv_heads ids.
 * Results are exact and deterministic.
 */
int recache_build_routes(int n_req, const int32_t* req_res_off, const int32_t* req_res,
                         int total_req_res, int n_res, int n_layers, int n_kv_heads,
                         const uint8_t* route_mask, const int32_t* cu_kept, int32_t* route_off,
                         int32_t* route_res, int32_t* route_tokens, void* stream);

/*
 * Row tables of a route-compacted resource store (Sec. 3: after structural
 * and semantic pruning a resource is read only through its visible routes
 * and only at kept positions, so only those rows need memory; the memory
 * column of the results tables counts this saving).  Layer l of the store
 * holds, for every resource r and KV group g with route_mask[r][l][g] set,
 * the kept rows of r for head g, resource-major: routes (r, g) in increasing
 * r, then g.  Output, device int32, n_layers rows of n_res * n_kv_heads + 1:
 *   store_off[l][r * n_kv_heads + g]: first store row of route (r, g) (an
 *       invisible route holds no rows and gets the row where it would start)
 *   store_off[l][n_res * n_kv_heads]: rows stored for layer l.
 * A route holds cu_kept[r+1] - cu_kept[r] rows.  total_kept = cu_kept[n_res];
 * n_kv_heads * total_kept must be below 2^31.  Exact and deterministic.
 */
int recache_route_store_offsets(int n_res, int n_layers, int n_kv_heads, int total_kept,
                                const uint8_t* route_mask, const int32_t* cu_kept,
                                int32_t* store_off, void* stream);

/*
 * Fill layer `layer` of a route-compacted store straight from that layer's
 * constructed head-major caches (semantic-pruning gather and route
 * compaction in one pass; Sec. 3, "Semantic Pruning" and "Structural
 * Pruning"):
 *   k_store[store_off[l][r * Hkv + g] + j] =
 *       k_cache[g][cu_len[r] + kept_idx[cu_kept[r] + j]],  j < kept rows of r,
 * for every visible route (r, g), and the same for v; rows are copied bit
 * for bit.  store_off is the full table of recache_route_store_offsets;
 * store_rows = store_off[layer][n_res * n_kv_heads] (read it back to size the
 * store); k_store / v_store are [store_rows][head_dim].  kept lists follow
 * recache_prune_gather's rules.
 */
int recache_store_routes(int dtype, int layer, int n_layers, int n_res, const int32_t* cu_len,
                         const int32_t* cu_kept, const int32_t* kept_idx, int total_T,
                         int total_kept, int n_kv_heads, int head_dim, const int32_t* store_off,
                         int store_rows, const void* k_cache, const void* v_cache, void* k_store,
                         void* v_store, void* stream);

/*
 * Workspace bytes that recache_attend_cached needs for these sizes (0 when
 * max_q > 1: the prefill kernels use none).  Library convention, not a
 * passage of the paper: decode (Fig. 2's final mask with one query per
 * request) splits each (request, group) key stream into chunks whose partial
 * outputs and log-sum-exps are merged afterwards; the workspace holds those
 * partials, fp32, n_req * n_q_heads * splits * (head_dim + 2) values.
 * max_kv is an upper bound on the keys a (request, group) can see in one layer
 * (route tokens + context), used only to choose the split count; 0 means
 * "use max_ctx".  Returns 0 for invalid sizes.  Pure host arithmetic.
 */
size_t recache_attend_workspace_bytes(int n_req, int max_q, int max_ctx, int max_kv,
                                      int n_q_heads, int n_kv_heads, int head_dim);

/*
 * Conversation tokens over cached resources, one layer (final ReCache mask,
 * Fig. 2; Sec. 3, "Structural Pruning" and "Semantic Pruning").
 *
 * Request b has Tq_b = cu_q[b+1] - cu_q[b] queries and Tc_b = cu_ctx[b+1] -
 * cu_ctx[b] context rows, 1 <= Tq_b <= Tc_b <= max_ctx, Tq_b <= max_q,
 * cu_q[n_req] = total_q; its queries are the last Tq_b context tokens.  For query i of request b, head
 * h and group g = h / (Hq / Hkv), the visible keys are, in this order:
 *   1. every kept row of every resource in route_res[route_off[e] ..
 *      route_off[e+1]) with e = (b * n_layers + layer) * n_kv_heads + g
 *      (rows res_k[g][cu_kept[r] .. cu_kept[r+1]), or with a store table
 *      rows res_k[res_off[r * n_kv_heads + g] + j], j < cu_kept[r+1] -
 *      cu_kept[r]) -- M_resource routes; an empty list is an M_context route;
 *   2. context rows ctx_k[g][cu_ctx[b] + c] for c = 0 .. Tc_b - Tq_b + i
 *      (causal, bottom-right aligned; with Tq = 1 the new token sees all).
 *
 *   q[total_q][n_q_heads][head_dim]: rotated queries
 *   ctx_k/ctx_v[n_kv_heads][ctx_rows][head_dim]: rotated context K, context V
 *   res_k/res_v: this layer's resource rows, in one of two layouts:
 *       res_off == NULL: [n_kv_heads][res_rows][head_dim] compacted kept rows
 *           (output of recache_prune_gather, or unpruned caches with
 *           cu_kept = cu_len);
 *       res_off != NULL: a route-compacted store [res_rows][head_dim]
 *           (recache_store_routes), res_off = this layer's row of
 *           recache_route_store_offsets' table, res_rows its stored rows.
 *   route_off/route_res/route_tokens: output of recache_build_routes
 *   out[total_q][n_q_heads][head_dim]; lse[n_q_heads][total_q] or NULL
 *   max_route_len: upper bound on the resources of any route list (at most
 *       1024), i.e. on resources per request (check the request lists with
 *       recache_check_requests); a route list longer than 1024 makes the
 *       kernels write NaN for that (request, group) instead of truncating it
 *   Tq_b must also not exceed max_q: the prefill grid is sized by it, and
 *       rows past it are written as NaN; with max_q = 1 every request must
 *       have exactly one query (decode writes NaN for one that has more)
 *   plan: NULL, or the work order that recache_attend_plan built for this
 *       batch (the same n_req, n_kv_heads and n_q_heads); used by the bf16
 *       kernels (prefill and decode), ignored by fp32.  It only changes
 *       which grid position computes which (request, group): the results
 *       are bit-identical with and without it.  A plan of another batch
 *       leaves every access in bounds but computes some pairs twice and
 *       others not at all.
 *   workspace: device scratch of recache_attend_workspace_bytes(...) bytes
 *       (may be NULL when that is 0); contents need no initialisation.
 */
int recache_attend_cached(int dtype, int layer, int n_layers, int n_req, const int32_t* cu_q,
                          const int32_t* cu_ctx, int total_q, int max_q, int max_ctx, int max_kv,
                          int max_route_len, int n_q_heads, int n_kv_heads, int head_dim,
                          float softmax_scale, const void* q, const void* ctx_k,
                          const void* ctx_v, int ctx_rows, const void* res_k, const void* res_v,
                          int res_rows, const int32_t* cu_kept, const int32_t* res_off,
                          const int32_t* route_off, const int32_t* route_res,
                          const int32_t* route_tokens, const int32_t* plan, void* out,
                          float* lse, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Work order of recache_attend_cached's kernels for every layer of a batch.
 * A schedule, not a passage of the paper: routed resources (Sec. 3,
 * "Structural Pruning") give the (request, KV group) pairs key streams of
 * unequal length, and a grid that takes them in request order ends on a
 * tail of long streams (decode) or loads some XCDs more than others
 * (prefill).  For each layer l the pairs p = b * n_kv_heads + g are sorted
 * by their work (longest first; the work counts the 64-key tiles of every
 * query tile of the prefill kernel, plus a fixed cost per tile, from Tq_b,
 * Tc_b and route_tokens), and the sorted pairs are dealt row by row to the
 * n_kv_heads grid positions, alternating direction.
 *   cu_q/cu_ctx[n_req + 1], route_tokens[n_req][n_layers][n_kv_heads]: as
 *       for recache_attend_cached (route_tokens from recache_build_routes)
 *   plan[n_layers][n_req * n_kv_heads] int32 (device), of
 *       recache_attend_plan_bytes(...) bytes: written, a permutation of
 *       0 .. n_req * n_kv_heads - 1 per layer.
 * Build it once per batch, after recache_build_routes; in decode it stays a
 * valid order as the contexts grow (only its balance ages).
 * Errors: RECACHE_EINVAL for bad sizes or null pointers;
 * RECACHE_EUNSUPPORTED when n_req * n_kv_heads exceeds 8192 (pass plan =
 * NULL to recache_attend_cached then).
 */
size_t recache_attend_plan_bytes(int n_req, int n_layers, int n_kv_heads);
int recache_attend_plan(int n_layers, int n_req, int n_q_heads, int n_kv_heads,
                        const int32_t* cu_q, const int32_t* cu_ctx,
                        const int32_t* route_tokens, int32_t* plan, void* stream);

/*
 * recache_attend_cached for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  The same arguments and the same results (the same kernels)
 * without workspace / workspace_bytes: decode keeps its split partials in a
 * static device array of the library, RECACHE_NOALLOC_SCRATCH_BYTES (32 MiB)
 * per GPU, held by every GPU the library runs on until the process ends.  No
 * call allocates (no hipMalloc, no library routine that does).  The first
 * call on a device looks the array's address up with that device current
 * (the caller's stream must belong to the current device; make that first
 * call outside any stream capture).
 * The caller still owns and passes every input and output.  Nothing in the
 * array needs to start at zero: decode writes every partial its merge reads.
 * Every call on one GPU shares that GPU's array and it keeps the last call's
 * contents, so calls that overlap on one GPU (several streams, several host
 * threads) race: serialise them.
 * Errors: those of recache_attend_cached, and RECACHE_EWORKSPACE when
 * recache_attend_workspace_bytes(...) for these sizes exceeds
 * RECACHE_NOALLOC_SCRATCH_BYTES (decode with n_req * n_q_heads * splits *
 * (head_dim + 2) fp32 partials; about 65K partial slots at head_dim 128),
 * checked before any HIP call; RECACHE_EHIP if the address lookup fails.
 */
#define RECACHE_NOALLOC_SCRATCH_BYTES (32 * 1024 * 1024)
int recache_attend_cached_noalloc(int dtype, int layer, int n_layers, int n_req,
                                  const int32_t* cu_q, const int32_t* cu_ctx, int total_q,
                                  int max_q, int max_ctx, int max_kv, int max_route_len,
                                  int n_q_heads, int n_kv_heads, int head_dim, float softmax_scale,
                                  const void* q, const void* ctx_k, const void* ctx_v,
                                  int ctx_rows, const void* res_k, const void* res_v, int res_rows,
                                  const int32_t* cu_kept, const int32_t* res_off,
                                  const int32_t* route_off, const int32_t* route_res,
                                  const int32_t* route_tokens, const int32_t* plan, void* out,
                                  float* lse, void* stream);

/*
 * [host] Structural budget selection (Sec. 3, "Structural Pruning").  From
 * each layer's and each KV head group's leave-one-in contribution s_i (the
 * drop in invocation loss when only that unit sees resource states), the
 * contribution weights are w_i = max(s_i, 0) / sum_j max(s_j, 0); L* is the
 * k_layers layers and G* the k_groups groups of largest weight (equal weights:
 * lower index first), and the route set is Omega* = L* x G*.
 *   route_mask[n_layers][n_groups]: 1 on Omega*, else 0 (the same for every
 *       resource: copy it into recache_build_routes' [n_res][L][G] mask)
 *   w_layer[n_layers], w_group[n_groups]: the contribution weights
 *   rho = 1 - k_layers k_groups / (n_layers n_groups), the structural sparsity
 *   cc_layer, cc_group: summed weight of the retained layers / groups (the
 *       contribution coverage, as a fraction)
 * Errors: RECACHE_EINVAL for counts < 1, a budget outside [0, n], a null
 * pointer, a non-finite contribution, or no positive contribution in a kind.
 */
int recache_select_routes(int n_layers, int n_groups, const double* s_layer, const double* s_group,
                          int k_layers, int k_groups, uint8_t* route_mask, double* w_layer,
                          double* w_group, double* rho, double* cc_layer, double* cc_group);

/*
 * [host] Validators for host copies of index arrays.  The device kernels trust
 * the index arrays they are given (library convention: validation is a host
 * step, so a kernel never waits on an error check), and these functions state
 * the preconditions the problem statement of Sec. 3 puts on them: X is a
 * sequence of resources R_i of D_i >= 1 tokens packed in order, each request
 * lists the resources it retrieved, and a semantically pruned resource keeps
 * a non-empty subsequence of its own tokens ("Semantic Pruning").  Each
 * returns RECACHE_OK or RECACHE_EINVAL (recache_last_error() names the first
 * bad entry); none touches device memory.
 *   recache_check_offsets: cu[0] = 0, cu non-decreasing (strictly increasing
 *       when strict != 0), cu[n] = total.
 *   recache_check_kept: for each resource, kept indices strictly ascending,
 *       inside [0, D_r), at least one, and cu_kept consistent.
 *   recache_check_encode_lengths: the packing offsets of an encode call
 *       (strictly increasing from 0 to total_T) with every resource at most
 *       max_len tokens long.  The encode grid is sized by max_len; a longer
 *       resource would reach past it (the kernels then write NaN into that
 *       resource's rows rather than leave them unwritten).
 *   recache_check_requests: the request lists of recache_build_routes
 *       (req_res_off from 0, non-decreasing, req_res_off[n_req] =
 *       total_req_res; every id in [0, n_res)) with no request listing more
 *       than max_route_len resources, and max_route_len <= 1024, the longest
 *       route list the attention kernels take (a longer list makes them write
 *       NaN outputs for that route rather than drop resources).
 */
int recache_check_offsets(const int32_t* cu, int n, int total, int strict);
int recache_check_kept(const int32_t* cu_len, const int32_t* cu_kept, const int32_t* kept_idx,
                       int n_res);
int recache_check_encode_lengths(const int32_t* cu_len, int n_res, int total_T, int max_len);
int recache_check_requests(const int32_t* req_res_off, const int32_t* req_res, int n_req,
                           int total_req_res, int n_res, int max_route_len);

#ifdef __cplusplus
}
#endif

#endif /* RECACHE_H */
