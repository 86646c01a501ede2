// C ABI of the library (declared and documented in include/recache.h).
//
// Every entry point validates its scalar arguments on the host and returns an
// error code before launching anything; then it fills the kernel argument
// block and enqueues the kernels on the caller's stream.  No device memory is
// allocated here and nothing synchronises.
#include <math.h>
#include <stdint.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "recache.h"
#include "kernels.hpp"

using namespace rc;

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int ok() {
    g_err[0] = '\0';
    return RECACHE_OK;
}

int hip_status(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(RECACHE_EHIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

#define REQUIRE(cond, code, ...)                        \
    do {                                                \
        if (!(cond)) return fail((code), __VA_ARGS__);  \
    } while (0)

int check_dtype_dim(int dtype, int head_dim) {
    REQUIRE(dtype == RECACHE_F32 || dtype == RECACHE_BF16, RECACHE_EUNSUPPORTED,
            "dtype %d is not RECACHE_F32 or RECACHE_BF16", dtype);
    REQUIRE(head_dim == 64 || head_dim == 128, RECACHE_EUNSUPPORTED,
            "head_dim %d is not 64 or 128", head_dim);
    return RECACHE_OK;
}

int check_heads(int dtype, int n_q_heads, int n_kv_heads) {
    REQUIRE(n_q_heads > 0 && n_kv_heads > 0, RECACHE_EINVAL, "head counts must be positive (%d, %d)",
            n_q_heads, n_kv_heads);
    REQUIRE(n_q_heads % n_kv_heads == 0, RECACHE_EINVAL,
            "n_q_heads %d is not a multiple of n_kv_heads %d", n_q_heads, n_kv_heads);
    const int r = n_q_heads / n_kv_heads;
    if (dtype == RECACHE_BF16)
        REQUIRE(r >= 1 && r <= 8, RECACHE_EUNSUPPORTED,
                "bf16 kernels take 1 to 8 query heads per KV head, not %d", r);
    return RECACHE_OK;
}

int check_base(double rope_base) {
    REQUIRE(isfinite(rope_base) && rope_base > 1.0, RECACHE_EINVAL, "rope_base %g must be > 1",
            rope_base);
    return RECACHE_OK;
}

// theta_i / (2 pi), theta_i = base^(-2i/d), in fp64.
RopeRev make_rope(double base, int head_dim) {
    RopeRev r;
    memset(&r, 0, sizeof r);
    for (int i = 0; i < head_dim / 2; ++i)
        r.rev[i] = pow(base, -2.0 * (double)i / (double)head_dim) / 6.283185307179586476925286766559;
    return r;
}

float resolve_scale(float s, int head_dim) { return s > 0.f ? s : 1.0f / sqrtf((float)head_dim); }

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// The bf16 attention kernels read every KV plane (one KV head's rows of a
// cache, a layer's route-compacted store, the context) through 32-bit byte
// offsets: each must stay below 4 GiB.
int check_planes(long rows_a, long rows_b, int head_dim) {
    const long limit = 1L << 32, row_bytes = 2L * head_dim;
    REQUIRE(rows_a * row_bytes < limit && rows_b * row_bytes < limit, RECACHE_EUNSUPPORTED,
            "a KV plane of %ld or %ld rows of %ld bytes reaches 4 GiB", rows_a, rows_b, row_bytes);
    return RECACHE_OK;
}

}  // namespace

extern "C" {

int recache_version(void) { return 100; }

const char* recache_last_error(void) { return g_err; }

int recache_rope_q(int dtype, int T, int n_heads, int head_dim, double rope_base,
                   const int32_t* pos, void* x, void* stream) {
    int rc_ = check_dtype_dim(dtype, head_dim);
    if (rc_) return rc_;
    if ((rc_ = check_base(rope_base))) return rc_;
    REQUIRE(T >= 0 && n_heads > 0, RECACHE_EINVAL, "bad sizes T=%d n_heads=%d", T, n_heads);
    if (T == 0) return ok();
    REQUIRE(pos && x, RECACHE_EINVAL, "pos and x must be non-null");
    RopeArgs a{};
    a.T = T;
    a.n_heads = n_heads;
    a.head_dim = head_dim;
    a.dtype = dtype;
    a.pos = pos;
    a.rope = make_rope(rope_base, head_dim);
    a.x = x;
    a.y = x;
    return hip_status(launch_rope(a, as_stream(stream)), "recache_rope_q launch");
}

int recache_rope_kv(int dtype, int T, int n_kv_heads, int head_dim, double rope_base,
                    const int32_t* pos, const void* k, const void* v, void* k_cache,
                    void* v_cache, int cache_rows, int row0, void* stream) {
    int rc_ = check_dtype_dim(dtype, head_dim);
    if (rc_) return rc_;
    if ((rc_ = check_base(rope_base))) return rc_;
    REQUIRE(T >= 0 && n_kv_heads > 0, RECACHE_EINVAL, "bad sizes T=%d n_kv_heads=%d", T, n_kv_heads);
    REQUIRE(row0 >= 0 && cache_rows >= 0 && (long)row0 + T <= cache_rows, RECACHE_EINVAL,
            "rows [%d, %ld) do not fit a cache of %d rows", row0, (long)row0 + T, cache_rows);
    if (T == 0) return ok();
    REQUIRE(pos && k && v && k_cache && v_cache, RECACHE_EINVAL, "null pointer argument");
    RopeArgs a{};
    a.T = T;
    a.n_heads = n_kv_heads;
    a.head_dim = head_dim;
    a.dtype = dtype;
    a.pos = pos;
    a.rope = make_rope(rope_base, head_dim);
    a.x = k;
    a.y = k_cache;
    a.v = v;
    a.v_dst = v_cache;
    a.cache_rows = cache_rows;
    a.row0 = row0;
    a.to_cache = 1;
    return hip_status(launch_rope(a, as_stream(stream)), "recache_rope_kv launch");
}

namespace {

int check_encode(int dtype, int n_res, const int32_t* cu_len, int total_T, int max_len,
                 int n_q_heads, int n_kv_heads, int head_dim, double rope_base, float softmax_scale,
                 int prefix_len, const void* prefix_k, const void* prefix_v) {
    int rc_ = check_dtype_dim(dtype, head_dim);
    if (rc_) return rc_;
    if ((rc_ = check_heads(dtype, n_q_heads, n_kv_heads))) return rc_;
    if ((rc_ = check_base(rope_base))) return rc_;
    REQUIRE(n_res >= 1, RECACHE_EINVAL, "n_res %d must be >= 1", n_res);
    REQUIRE(total_T >= n_res, RECACHE_EINVAL, "total_T %d < n_res %d (every resource needs a token)",
            total_T, n_res);
    REQUIRE(max_len >= 1 && max_len <= total_T, RECACHE_EINVAL, "max_len %d outside [1, %d]",
            max_len, total_T);
    REQUIRE(cu_len, RECACHE_EINVAL, "null pointer argument");
    REQUIRE(!(isnan(softmax_scale) || isinf(softmax_scale)), RECACHE_EINVAL, "softmax_scale not finite");
    REQUIRE(prefix_len >= 0, RECACHE_EINVAL, "prefix_len %d must be >= 0", prefix_len);
    REQUIRE(prefix_len == 0 || (prefix_k && prefix_v), RECACHE_EINVAL,
            "prefix_len %d needs prefix_k and prefix_v", prefix_len);
    if (dtype == RECACHE_BF16)
        if ((rc_ = check_planes(total_T, prefix_len, head_dim))) return rc_;
    return RECACHE_OK;
}

hipError_t encode_attention_launch(int dtype, int n_res, const int32_t* cu_len, int total_T,
                                   int max_len, int n_q_heads, int n_kv_heads, int head_dim,
                                   const RopeRev& rope, const int32_t* pos_base, int prefix_len,
                                   const void* prefix_k, const void* prefix_v,
                                   float softmax_scale, const void* q, const void* k_cache,
                                   const void* v_cache, void* out, float* lse, hipStream_t s) {
    const float scale = resolve_scale(softmax_scale, head_dim);
    const int ratio = n_q_heads / n_kv_heads;
    if (dtype == RECACHE_BF16) {
        AttnArgs a{};
        a.n_q_heads = n_q_heads;
        a.n_kv_heads = n_kv_heads;
        a.ratio = ratio;
        a.max_rows = max_len;
        a.n_units = n_res;
        a.scale_log2 = scale * 1.4426950408889634f;
        a.q = static_cast<const uint16_t*>(q);
        a.out = static_cast<uint16_t*>(out);
        a.lse = lse;
        a.lse_rows = total_T;
        // segments: the shared prefix; causal part: the resources' own rows
        a.k = static_cast<const uint16_t*>(prefix_k);
        a.v = static_cast<const uint16_t*>(prefix_v);
        a.k_rows = prefix_len;
        a.k_gstride = prefix_len;
        a.ck = static_cast<const uint16_t*>(k_cache);
        a.cv = static_cast<const uint16_t*>(v_cache);
        a.c_rows = total_T;
        a.p_len = prefix_len;
        a.cu_len = cu_len;
        a.pos_base = pos_base;
        a.rope = rope;
        return launch_attn_mfma(a, true, head_dim, s);
    }
    AttnF32Args a{};
    a.n_q_heads = n_q_heads;
    a.n_kv_heads = n_kv_heads;
    a.ratio = ratio;
    a.head_dim = head_dim;
    a.n_units = n_res;
    a.max_rows = max_len;
    a.scale = scale;
    a.q = static_cast<const float*>(q);
    a.out = static_cast<float*>(out);
    a.lse = lse;
    a.lse_rows = total_T;
    a.k = static_cast<const float*>(prefix_k);
    a.v = static_cast<const float*>(prefix_v);
    a.k_rows = prefix_len;
    a.k_gstride = prefix_len;
    a.ck = static_cast<const float*>(k_cache);
    a.cv = static_cast<const float*>(v_cache);
    a.c_rows = total_T;
    a.p_len = prefix_len;
    a.cu_len = cu_len;
    a.pos_base = pos_base;
    a.rope = rope;
    return launch_attn_f32(a, true, s);
}

}  // namespace

int recache_encode_resources(int dtype, int n_res, const int32_t* cu_len, int total_T,
                             int max_len, int n_q_heads, int n_kv_heads, int head_dim,
                             double rope_base, const int32_t* pos_base, int prefix_len,
                             const void* prefix_k, const void* prefix_v, float softmax_scale,
                             const void* q, const void* k, const void* v, void* out,
                             void* k_cache, void* v_cache, float* lse, void* stream) {
    int rc_ = check_encode(dtype, n_res, cu_len, total_T, max_len, n_q_heads, n_kv_heads, head_dim,
                           rope_base, softmax_scale, prefix_len, prefix_k, prefix_v);
    if (rc_) return rc_;
    REQUIRE(q && k && v && out && k_cache && v_cache, RECACHE_EINVAL, "null pointer argument");
    const hipStream_t s = as_stream(stream);
    (void)hipGetLastError();  // clear a stale error so the status below is ours

    RopeArgs ra{};
    ra.T = total_T;
    ra.n_heads = n_kv_heads;
    ra.head_dim = head_dim;
    ra.dtype = dtype;
    ra.cu_len = cu_len;
    ra.pos_base = pos_base;
    ra.n_res = n_res;
    ra.rope = make_rope(rope_base, head_dim);
    ra.x = k;
    ra.y = k_cache;
    ra.v = v;
    ra.v_dst = v_cache;
    ra.cache_rows = total_T;
    ra.row0 = 0;
    ra.to_cache = 1;
    hipError_t e = launch_rope(ra, s);
    if (e != hipSuccess) return hip_status(e, "encode: rope/cache launch");
    e = encode_attention_launch(dtype, n_res, cu_len, total_T, max_len, n_q_heads, n_kv_heads,
                                head_dim, ra.rope, pos_base, prefix_len, prefix_k, prefix_v,
                                softmax_scale, q, k_cache, v_cache, out, lse, s);
    return hip_status(e, "encode: attention launch");
}

int recache_encode_attention(int dtype, int n_res, const int32_t* cu_len, int total_T,
                             int max_len, int n_q_heads, int n_kv_heads, int head_dim,
                             double rope_base, const int32_t* pos_base, int prefix_len,
                             const void* prefix_k, const void* prefix_v, float softmax_scale,
                             const void* q, const void* k_cache, const void* v_cache, void* out,
                             float* lse, void* stream) {
    int rc_ = check_encode(dtype, n_res, cu_len, total_T, max_len, n_q_heads, n_kv_heads, head_dim,
                           rope_base, softmax_scale, prefix_len, prefix_k, prefix_v);
    if (rc_) return rc_;
    REQUIRE(q && k_cache && v_cache && out, RECACHE_EINVAL, "null pointer argument");
    (void)hipGetLastError();
    return hip_status(encode_attention_launch(dtype, n_res, cu_len, total_T, max_len, n_q_heads,
                                              n_kv_heads, head_dim, make_rope(rope_base, head_dim),
                                              pos_base, prefix_len, prefix_k, prefix_v,
                                              softmax_scale, q, k_cache, v_cache, out, lse,
                                              as_stream(stream)),
                      "encode attention launch");
}

int recache_prune_gather(int dtype, int n_res, const int32_t* cu_len, const int32_t* cu_kept,
                         const int32_t* kept_idx, int total_T, int total_kept, int n_kv_heads,
                         int head_dim, const void* k_cache, const void* v_cache, void* k_kept,
                         void* v_kept, void* stream) {
    int rc_ = check_dtype_dim(dtype, head_dim);
    if (rc_) return rc_;
    REQUIRE(n_res >= 1 && n_kv_heads >= 1, RECACHE_EINVAL, "n_res %d / n_kv_heads %d must be >= 1",
            n_res, n_kv_heads);
    REQUIRE(total_T >= n_res, RECACHE_EINVAL, "total_T %d < n_res %d", total_T, n_res);
    REQUIRE(total_kept >= n_res && total_kept <= total_T, RECACHE_EINVAL,
            "total_kept %d outside [n_res, total_T] = [%d, %d]", total_kept, n_res, total_T);
    REQUIRE(cu_len && cu_kept && kept_idx && k_cache && v_cache && k_kept && v_kept, RECACHE_EINVAL,
            "null pointer argument");
    (void)hipGetLastError();
    const int es = dtype == RECACHE_F32 ? 4 : 2;
    return hip_status(launch_prune_gather(es, n_res, cu_len, cu_kept, kept_idx, total_T, total_kept,
                                          n_kv_heads, head_dim, k_cache, v_cache, k_kept, v_kept,
                                          as_stream(stream)),
                      "recache_prune_gather launch");
}

int recache_build_routes(int n_req, const int32_t* req_res_off, const int32_t* req_res,
                         int total_req_res, int n_res, int n_layers, int n_kv_heads,
                         const uint8_t* route_mask, const int32_t* cu_kept, int32_t* route_off,
                         int32_t* route_res, int32_t* route_tokens, void* stream) {
    REQUIRE(n_req >= 1 && n_res >= 1 && n_layers >= 1 && n_kv_heads >= 1, RECACHE_EINVAL,
            "n_req %d, n_res %d, n_layers %d, n_kv_heads %d must be >= 1", n_req, n_res, n_layers,
            n_kv_heads);
    REQUIRE(total_req_res >= 0, RECACHE_EINVAL, "total_req_res %d < 0", total_req_res);
    REQUIRE((long long)total_req_res * n_layers * n_kv_heads <= 0x7fffffffLL &&
                (long long)n_req * n_layers * n_kv_heads < 0x7fffffffLL,
            RECACHE_EINVAL, "route CSR would overflow int32");
    REQUIRE(req_res_off && req_res && route_mask && cu_kept && route_off && route_res && route_tokens,
            RECACHE_EINVAL, "null pointer argument");
    (void)hipGetLastError();
    return hip_status(launch_build_routes(n_req, req_res_off, req_res, n_res, n_layers, n_kv_heads,
                                          route_mask, cu_kept, route_off, route_res, route_tokens,
                                          as_stream(stream)),
                      "recache_build_routes launch");
}

int recache_route_store_offsets(int n_res, int n_layers, int n_kv_heads, int total_kept,
                                const uint8_t* route_mask, const int32_t* cu_kept,
                                int32_t* store_off, void* stream) {
    REQUIRE(n_res >= 1 && n_layers >= 1 && n_kv_heads >= 1, RECACHE_EINVAL,
            "n_res %d, n_layers %d, n_kv_heads %d must be >= 1", n_res, n_layers, n_kv_heads);
    REQUIRE(total_kept >= n_res, RECACHE_EINVAL, "total_kept %d < n_res %d", total_kept, n_res);
    REQUIRE((long long)n_kv_heads * total_kept < 0x7fffffffLL &&
                (long long)n_layers * ((long long)n_res * n_kv_heads + 1) <= 0x7fffffffLL,
            RECACHE_EINVAL, "store tables would overflow int32");
    REQUIRE(route_mask && cu_kept && store_off, RECACHE_EINVAL, "null pointer argument");
    (void)hipGetLastError();
    return hip_status(launch_store_offsets(n_res, n_layers, n_kv_heads, route_mask, cu_kept,
                                           store_off, as_stream(stream)),
                      "recache_route_store_offsets launch");
}

int recache_store_routes(int dtype, int layer, int n_layers, int n_res, const int32_t* cu_len,
                         const int32_t* cu_kept, const int32_t* kept_idx, int total_T,
                         int total_kept, int n_kv_heads, int head_dim, const int32_t* store_off,
                         int store_rows, const void* k_cache, const void* v_cache, void* k_store,
                         void* v_store, void* stream) {
    int rc_ = check_dtype_dim(dtype, head_dim);
    if (rc_) return rc_;
    REQUIRE(n_res >= 1 && n_kv_heads >= 1, RECACHE_EINVAL, "n_res %d / n_kv_heads %d must be >= 1",
            n_res, n_kv_heads);
    REQUIRE(n_layers >= 1 && layer >= 0 && layer < n_layers, RECACHE_EINVAL,
            "layer %d outside [0, %d)", layer, n_layers);
    REQUIRE(total_T >= n_res, RECACHE_EINVAL, "total_T %d < n_res %d", total_T, n_res);
    REQUIRE(total_kept >= n_res && total_kept <= total_T, RECACHE_EINVAL,
            "total_kept %d outside [n_res, total_T] = [%d, %d]", total_kept, n_res, total_T);
    REQUIRE(store_rows >= 0 && (long long)store_rows <= (long long)n_kv_heads * total_kept,
            RECACHE_EINVAL, "store_rows %d outside [0, n_kv_heads * total_kept]", store_rows);
    REQUIRE(cu_len && cu_kept && kept_idx && store_off && k_cache && v_cache &&
                (store_rows == 0 || (k_store && v_store)),
            RECACHE_EINVAL, "null pointer argument");
    (void)hipGetLastError();
    const int es = dtype == RECACHE_F32 ? 4 : 2;
    return hip_status(launch_store_routes(es, layer, n_res, cu_len, cu_kept, kept_idx, total_T,
                                          total_kept, n_kv_heads, head_dim, store_off, store_rows,
                                          k_cache, v_cache, k_store, v_store, as_stream(stream)),
                      "recache_store_routes launch");
}

size_t recache_attend_workspace_bytes(int n_req, int max_q, int max_ctx, int max_kv,
                                      int n_q_heads, int n_kv_heads, int head_dim) {
    if (n_req <= 0 || max_q != 1 || n_q_heads <= 0 || n_kv_heads <= 0 || head_dim <= 0) return 0;
    const int kv = max_kv > 0 ? max_kv : max_ctx;
    return decode_workspace_bytes(n_req, n_q_heads, head_dim, decode_splits(n_req, n_kv_heads, kv));
}

}  // extern "C"

namespace {

// Scalar and pointer checks of an attend call (everything but the
// workspace); no HIP call.
int check_attend(int dtype, int layer, int n_layers, int n_req, const int32_t* cu_q,
                 const int32_t* cu_ctx, int total_q, int max_q, int max_ctx, int max_route_len,
                 int n_q_heads, int n_kv_heads, int head_dim, float softmax_scale, const void* q,
                 const void* ctx_k, const void* ctx_v, int ctx_rows, const void* res_k,
                 const void* res_v, int res_rows, const int32_t* cu_kept, const int32_t* res_off,
                 const int32_t* route_off, const int32_t* route_res, const int32_t* route_tokens,
                 const void* out) {
    int rc_ = check_dtype_dim(dtype, head_dim);
    if (rc_) return rc_;
    if ((rc_ = check_heads(dtype, n_q_heads, n_kv_heads))) return rc_;
    REQUIRE(n_layers >= 1 && layer >= 0 && layer < n_layers, RECACHE_EINVAL,
            "layer %d outside [0, %d)", layer, n_layers);
    REQUIRE(n_req >= 1, RECACHE_EINVAL, "n_req %d must be >= 1", n_req);
    REQUIRE(max_q >= 1 && max_ctx >= max_q, RECACHE_EINVAL,
            "need 1 <= max_q <= max_ctx (queries are the last context tokens), got %d, %d", max_q,
            max_ctx);
    REQUIRE(total_q >= n_req && (long)total_q <= (long)n_req * max_q, RECACHE_EINVAL,
            "total_q %d outside [n_req, n_req * max_q] = [%d, %ld]", total_q, n_req,
            (long)n_req * max_q);
    REQUIRE(max_route_len >= 0 && max_route_len <= 1024, RECACHE_EUNSUPPORTED,
            "max_route_len %d outside [0, 1024]", max_route_len);
    // a route-compacted store may hold no rows for a layer outside every route
    REQUIRE(ctx_rows >= 1 && res_rows >= (res_off ? 0 : 1), RECACHE_EINVAL,
            "ctx_rows %d / res_rows %d too small", ctx_rows, res_rows);
    REQUIRE(cu_q && cu_ctx && q && ctx_k && ctx_v && ((res_k && res_v) || res_rows == 0) &&
                cu_kept && route_off && route_res && route_tokens && out,
            RECACHE_EINVAL, "null pointer argument");
    REQUIRE(!(isnan(softmax_scale) || isinf(softmax_scale)), RECACHE_EINVAL, "softmax_scale not finite");
    if (dtype == RECACHE_BF16 && max_q > 1)
        if ((rc_ = check_planes(res_rows, ctx_rows, head_dim))) return rc_;
    return RECACHE_OK;
}

}  // namespace

extern "C" {

int recache_attend_cached(int dtype, int layer, int n_layers, int n_req, const int32_t* cu_q,
                          const int32_t* cu_ctx, int total_q, int max_q, int max_ctx, int max_kv,
                          int max_route_len, int n_q_heads, int n_kv_heads, int head_dim,
                          float softmax_scale, const void* q, const void* ctx_k,
                          const void* ctx_v, int ctx_rows, const void* res_k, const void* res_v,
                          int res_rows, const int32_t* cu_kept, const int32_t* res_off,
                          const int32_t* route_off, const int32_t* route_res,
                          const int32_t* route_tokens, const int32_t* plan, void* out,
                          float* lse, void* workspace, size_t workspace_bytes, void* stream) {
    REQUIRE(((uintptr_t)plan & 3) == 0, RECACHE_EINVAL, "plan is not 4-byte aligned");
    int rc_ = check_attend(dtype, layer, n_layers, n_req, cu_q, cu_ctx, total_q, max_q, max_ctx,
                           max_route_len, n_q_heads, n_kv_heads, head_dim, softmax_scale, q, ctx_k,
                           ctx_v, ctx_rows, res_k, res_v, res_rows, cu_kept, res_off, route_off,
                           route_res, route_tokens, out);
    if (rc_) return rc_;
    const float scale = resolve_scale(softmax_scale, head_dim);
    const int ratio = n_q_heads / n_kv_heads;
    const hipStream_t s = as_stream(stream);
    (void)hipGetLastError();

    if (dtype == RECACHE_F32) {
        AttnF32Args a{};
        a.n_q_heads = n_q_heads;
        a.n_kv_heads = n_kv_heads;
        a.ratio = ratio;
        a.head_dim = head_dim;
        a.n_units = n_req;
        a.max_rows = max_q;
        a.scale = scale;
        a.q = static_cast<const float*>(q);
        a.out = static_cast<float*>(out);
        a.lse = lse;
        a.k = static_cast<const float*>(res_k);
        a.v = static_cast<const float*>(res_v);
        a.k_rows = res_rows;
        a.k_gstride = res_off ? 0 : res_rows;
        a.res_off = res_off;
        a.cu_q = cu_q;
        a.cu_ctx = cu_ctx;
        a.ck = static_cast<const float*>(ctx_k);
        a.cv = static_cast<const float*>(ctx_v);
        a.c_rows = ctx_rows;
        a.layer = layer;
        a.n_layers = n_layers;
        a.route_off = route_off;
        a.route_res = route_res;
        a.cu_kept = cu_kept;
        a.lse_rows = total_q;
        return hip_status(launch_attn_f32(a, false, s), "attend (fp32) launch");
    }
    if (max_q == 1) {
        const int kv = max_kv > 0 ? max_kv : max_ctx;
        const int n_splits = decode_splits(n_req, n_kv_heads, kv);
        const size_t need = decode_workspace_bytes(n_req, n_q_heads, head_dim, n_splits);
        REQUIRE(workspace && workspace_bytes >= need, RECACHE_EWORKSPACE,
                "decode needs a %zu-byte workspace, got %zu", need, workspace ? workspace_bytes : 0);
        DecodeArgs a{};
        a.n_req = n_req;
        a.n_q_heads = n_q_heads;
        a.n_kv_heads = n_kv_heads;
        a.ratio = ratio;
        a.head_dim = head_dim;
        a.n_splits = n_splits;
        a.scale_log2 = scale * 1.4426950408889634f;
        a.q = static_cast<const uint16_t*>(q);
        a.out = static_cast<uint16_t*>(out);
        a.lse = lse;
        a.lse_rows = total_q;
        a.rk = static_cast<const uint16_t*>(res_k);
        a.rv = static_cast<const uint16_t*>(res_v);
        a.r_rows = res_rows;
        a.r_gstride = res_off ? 0 : res_rows;
        a.res_off = res_off;
        a.ck = static_cast<const uint16_t*>(ctx_k);
        a.cv = static_cast<const uint16_t*>(ctx_v);
        a.c_rows = ctx_rows;
        a.cu_q = cu_q;
        a.cu_ctx = cu_ctx;
        a.layer = layer;
        a.n_layers = n_layers;
        a.route_off = route_off;
        a.route_res = route_res;
        a.cu_kept = cu_kept;
        a.ws_o = static_cast<float*>(workspace);
        a.ws_ml = a.ws_o + (size_t)n_req * n_q_heads * n_splits * head_dim;
        a.plan = plan;
        return hip_status(launch_decode(a, s), "attend (decode) launch");
    }
    AttnArgs a{};
    a.n_q_heads = n_q_heads;
    a.n_kv_heads = n_kv_heads;
    a.ratio = ratio;
    a.max_rows = max_q;
    a.n_units = n_req;
    a.scale_log2 = scale * 1.4426950408889634f;
    a.q = static_cast<const uint16_t*>(q);
    a.out = static_cast<uint16_t*>(out);
    a.lse = lse;
    a.lse_rows = total_q;
    a.k = static_cast<const uint16_t*>(res_k);
    a.v = static_cast<const uint16_t*>(res_v);
    a.k_rows = res_rows;
    a.k_gstride = res_off ? 0 : res_rows;
    a.res_off = res_off;
    a.cu_q = cu_q;
    a.cu_ctx = cu_ctx;
    a.ck = static_cast<const uint16_t*>(ctx_k);
    a.cv = static_cast<const uint16_t*>(ctx_v);
    a.c_rows = ctx_rows;
    a.layer = layer;
    a.n_layers = n_layers;
    a.route_off = route_off;
    a.route_res = route_res;
    a.cu_kept = cu_kept;
    a.plan = plan;
    return hip_status(launch_attn_mfma(a, false, head_dim, s), "attend (prefill) launch");
}

size_t recache_attend_plan_bytes(int n_req, int n_layers, int n_kv_heads) {
    if (n_req < 1 || n_layers < 1 || n_kv_heads < 1) return 0;
    return (size_t)n_layers * n_req * n_kv_heads * sizeof(int32_t);
}

int recache_attend_plan(int n_layers, int n_req, int n_q_heads, int n_kv_heads,
                        const int32_t* cu_q, const int32_t* cu_ctx, const int32_t* route_tokens,
                        int32_t* plan, void* stream) {
    REQUIRE(n_layers >= 1 && n_req >= 1 && n_kv_heads >= 1 && n_q_heads >= n_kv_heads &&
                n_q_heads % n_kv_heads == 0,
            RECACHE_EINVAL, "n_layers %d, n_req %d, n_q_heads %d, n_kv_heads %d", n_layers, n_req,
            n_q_heads, n_kv_heads);
    REQUIRE((long long)n_req * n_kv_heads <= kMaxPlanPairs, RECACHE_EUNSUPPORTED,
            "n_req * n_kv_heads = %lld pairs, more than the %d one plan sorts",
            (long long)n_req * n_kv_heads, kMaxPlanPairs);
    REQUIRE((long long)n_req * n_layers * n_kv_heads < 0x7fffffffLL, RECACHE_EINVAL,
            "plan would overflow int32 indexing");
    REQUIRE(cu_q && cu_ctx && route_tokens && plan, RECACHE_EINVAL, "null pointer argument");
    REQUIRE(((uintptr_t)plan & 3) == 0, RECACHE_EINVAL, "plan is not 4-byte aligned");
    PlanArgs a{};
    a.n_req = n_req;
    a.n_layers = n_layers;
    a.n_kv_heads = n_kv_heads;
    a.wg_rows = attend_block_rows(n_q_heads / n_kv_heads);
    a.cu_q = cu_q;
    a.cu_ctx = cu_ctx;
    a.route_tokens = route_tokens;
    a.plan = plan;
    (void)hipGetLastError();
    return hip_status(launch_attend_plan(a, as_stream(stream)), "recache_attend_plan launch");
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Attend without a caller workspace: decode's split partials go to a
// library-owned static device array (for callers that cannot allocate).

namespace {

// One copy per GPU the library runs on, each held until the process ends.
// In host code its name is only a stand-in: kernels get the device address
// that hipGetSymbolAddress returns for the current device (scratch_ptr).
static __device__ __align__(256) char scratch[RECACHE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's copy of `scratch`, looked up with
// that device current on the first call there and kept for later calls.
int scratch_ptr(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(RECACHE_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
    REQUIRE(dev >= 0 && dev < kMaxDevices, RECACHE_EUNSUPPORTED, "device %d: at most %d devices",
            dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(RECACHE_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                        hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return RECACHE_OK;
}

}  // namespace

extern "C" {

int recache_attend_cached_noalloc(int dtype, int layer, int n_layers, int n_req,
                                  const int32_t* cu_q, const int32_t* cu_ctx, int total_q,
                                  int max_q, int max_ctx, int max_kv, int max_route_len,
                                  int n_q_heads, int n_kv_heads, int head_dim, float softmax_scale,
                                  const void* q, const void* ctx_k, const void* ctx_v,
                                  int ctx_rows, const void* res_k, const void* res_v, int res_rows,
                                  const int32_t* cu_kept, const int32_t* res_off,
                                  const int32_t* route_off, const int32_t* route_res,
                                  const int32_t* route_tokens, const int32_t* plan, void* out,
                                  float* lse, void* stream) {
    REQUIRE(((uintptr_t)plan & 3) == 0, RECACHE_EINVAL, "plan is not 4-byte aligned");
    int rc_ = check_attend(dtype, layer, n_layers, n_req, cu_q, cu_ctx, total_q, max_q, max_ctx,
                           max_route_len, n_q_heads, n_kv_heads, head_dim, softmax_scale, q, ctx_k,
                           ctx_v, ctx_rows, res_k, res_v, res_rows, cu_kept, res_off, route_off,
                           route_res, route_tokens, out);
    if (rc_) return rc_;
    // the same workspace rule as recache_attend_cached: only bf16 decode uses one
    const size_t need = dtype == RECACHE_BF16
                            ? recache_attend_workspace_bytes(n_req, max_q, max_ctx, max_kv,
                                                             n_q_heads, n_kv_heads, head_dim)
                            : 0;
    REQUIRE(need <= (size_t)RECACHE_NOALLOC_SCRATCH_BYTES, RECACHE_EWORKSPACE,
            "decode needs %zu bytes of split partials, more than the %zu-byte static scratch of "
            "the allocation-free entry point (use recache_attend_cached with a workspace)",
            need, (size_t)RECACHE_NOALLOC_SCRATCH_BYTES);
    void* ws = nullptr;
    if ((rc_ = scratch_ptr(&ws))) return rc_;
    return recache_attend_cached(dtype, layer, n_layers, n_req, cu_q, cu_ctx, total_q, max_q,
                                 max_ctx, max_kv, max_route_len, n_q_heads, n_kv_heads, head_dim,
                                 softmax_scale, q, ctx_k, ctx_v, ctx_rows, res_k, res_v, res_rows,
                                 cu_kept, res_off, route_off, route_res, route_tokens, plan, out,
                                 lse, ws, (size_t)RECACHE_NOALLOC_SCRATCH_BYTES, stream);
}

int recache_check_offsets(const int32_t* cu, int n, int total, int strict) {
    REQUIRE(cu && n >= 0, RECACHE_EINVAL, "null offsets or negative count");
    REQUIRE(cu[0] == 0, RECACHE_EINVAL, "offsets[0] = %d, not 0", cu[0]);
    for (int i = 0; i < n; ++i) {
        const bool good = strict ? cu[i + 1] > cu[i] : cu[i + 1] >= cu[i];
        REQUIRE(good, RECACHE_EINVAL, "offsets[%d] = %d after offsets[%d] = %d", i + 1, cu[i + 1], i,
                cu[i]);
    }
    REQUIRE(cu[n] == total, RECACHE_EINVAL, "offsets[%d] = %d, expected total %d", n, cu[n], total);
    return ok();
}

int recache_check_kept(const int32_t* cu_len, const int32_t* cu_kept, const int32_t* kept_idx,
                       int n_res) {
    REQUIRE(cu_len && cu_kept && kept_idx && n_res >= 1, RECACHE_EINVAL, "null pointer or n_res < 1");
    REQUIRE(cu_len[0] == 0 && cu_kept[0] == 0, RECACHE_EINVAL, "offsets must start at 0");
    for (int r = 0; r < n_res; ++r) {
        const int len = cu_len[r + 1] - cu_len[r];
        const int a = cu_kept[r], b = cu_kept[r + 1];
        REQUIRE(len >= 1, RECACHE_EINVAL, "resource %d has length %d", r, len);
        REQUIRE(b > a && b - a <= len, RECACHE_EINVAL, "resource %d keeps %d of %d tokens", r, b - a, len);
        for (int j = a; j < b; ++j) {
            REQUIRE(kept_idx[j] >= 0 && kept_idx[j] < len, RECACHE_EINVAL,
                    "kept_idx[%d] = %d outside [0, %d) of resource %d", j, kept_idx[j], len, r);
            REQUIRE(j == a || kept_idx[j] > kept_idx[j - 1], RECACHE_EINVAL,
                    "kept_idx[%d] = %d not above kept_idx[%d] = %d (resource %d)", j, kept_idx[j],
                    j - 1, kept_idx[j - 1], r);
        }
    }
    return ok();
}

int recache_check_encode_lengths(const int32_t* cu_len, int n_res, int total_T, int max_len) {
    REQUIRE(cu_len && n_res >= 1, RECACHE_EINVAL, "null offsets or n_res < 1");
    int rc_ = recache_check_offsets(cu_len, n_res, total_T, 1);
    if (rc_) return rc_;
    for (int r = 0; r < n_res; ++r)
        REQUIRE(cu_len[r + 1] - cu_len[r] <= max_len, RECACHE_EINVAL,
                "resource %d has %d tokens, more than max_len %d", r, cu_len[r + 1] - cu_len[r],
                max_len);
    return ok();
}

int recache_check_requests(const int32_t* req_res_off, const int32_t* req_res, int n_req,
                           int total_req_res, int n_res, int max_route_len) {
    REQUIRE(req_res_off && n_req >= 1 && n_res >= 1, RECACHE_EINVAL,
            "null request offsets, n_req < 1 or n_res < 1");
    REQUIRE(total_req_res == 0 || req_res, RECACHE_EINVAL, "null request lists");
    REQUIRE(max_route_len >= 0 && max_route_len <= 1024, RECACHE_EINVAL,
            "max_route_len %d outside [0, 1024]", max_route_len);
    int rc_ = recache_check_offsets(req_res_off, n_req, total_req_res, 0);
    if (rc_) return rc_;
    for (int b = 0; b < n_req; ++b)
        REQUIRE(req_res_off[b + 1] - req_res_off[b] <= max_route_len, RECACHE_EINVAL,
                "request %d lists %d resources, more than max_route_len %d", b,
                req_res_off[b + 1] - req_res_off[b], max_route_len);
    for (int j = 0; j < total_req_res; ++j)
        REQUIRE(req_res[j] >= 0 && req_res[j] < n_res, RECACHE_EINVAL,
                "req_res[%d] = %d outside [0, %d)", j, req_res[j], n_res);
    return ok();
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Structural budget selection (Sec. 3, "Structural Pruning"; rho and CC from
// the structural budget analysis).  Host code.

namespace {

// w_i = max(s_i, 0) / sum_j max(s_j, 0); false if no s_i is positive or one is
// not finite.
bool contribution_weights(const double* s, int n, double* w) {
    double total = 0.0;
    for (int i = 0; i < n; ++i) {
        if (!isfinite(s[i])) return false;
        if (s[i] > 0.0) total += s[i];
    }
    if (!(total > 0.0)) return false;
    for (int i = 0; i < n; ++i) w[i] = s[i] > 0.0 ? s[i] / total : 0.0;
    return true;
}

// Units ranked by decreasing weight, equal weights by increasing index; keep[i]
// is set for the first k.  Returns the kept weight.
double keep_top(const double* w, int n, int k, std::vector<uint8_t>& keep) {
    std::vector<int> order(n);
    for (int i = 0; i < n; ++i) order[i] = i;
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return w[a] > w[b]; });
    keep.assign(n, 0);
    double cc = 0.0;
    for (int r = 0; r < k; ++r) {
        keep[order[r]] = 1;
        cc += w[order[r]];
    }
    return cc;
}

}  // namespace

int recache_select_routes(int n_layers, int n_groups, const double* s_layer, const double* s_group,
                          int k_layers, int k_groups, uint8_t* route_mask, double* w_layer,
                          double* w_group, double* rho, double* cc_layer, double* cc_group) {
    REQUIRE(n_layers >= 1 && n_groups >= 1, RECACHE_EINVAL, "n_layers %d / n_groups %d must be >= 1",
            n_layers, n_groups);
    REQUIRE(k_layers >= 0 && k_layers <= n_layers && k_groups >= 0 && k_groups <= n_groups,
            RECACHE_EINVAL, "budget %d x %d outside [0, %d] x [0, %d]", k_layers, k_groups, n_layers,
            n_groups);
    REQUIRE(s_layer && s_group && route_mask && w_layer && w_group && rho && cc_layer && cc_group,
            RECACHE_EINVAL, "null pointer argument");
    // weights into local buffers first: no output is written on an error
    std::vector<double> wl(n_layers), wg(n_groups);
    REQUIRE(contribution_weights(s_layer, n_layers, wl.data()) &&
                contribution_weights(s_group, n_groups, wg.data()),
            RECACHE_EINVAL, "contributions must be finite, with a positive one among layers and groups");
    std::vector<uint8_t> keep_l, keep_g;
    *cc_layer = keep_top(wl.data(), n_layers, k_layers, keep_l);
    *cc_group = keep_top(wg.data(), n_groups, k_groups, keep_g);
    std::copy(wl.begin(), wl.end(), w_layer);
    std::copy(wg.begin(), wg.end(), w_group);
    for (int l = 0; l < n_layers; ++l)
        for (int g = 0; g < n_groups; ++g) route_mask[(size_t)l * n_groups + g] = keep_l[l] & keep_g[g];
    *rho = 1.0 - (double)k_layers * k_groups / ((double)n_layers * n_groups);
    return ok();
}
