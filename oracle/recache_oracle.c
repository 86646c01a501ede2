/*
 * recache_oracle.c -- plain fp64 CPU oracle for ReCache resource-wise attention.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the correctness reference that the
 * GPU library is checked against.  Only the test suite, the smoke check and
 * the CPU-baseline leg of the benchmark may load it.  It shares no code,
 * header, table or helper with the HIP library, and it never calls it.
 *
 * Everything here is the plain definition, written out:
 *   - every input element is widened exactly to double (fp32 -> double, or
 *     bf16 bit pattern -> float -> double; fp64 inputs are taken as they are)
 *     at the point of use;
 *   - RoPE angles, cos and sin are evaluated in double with the host libm;
 *   - softmax is two-pass (max, then sum of exponentials) over the visible
 *     keys in ascending key order, with no tiling and no online rescaling.
 *
 * Paper sections followed (ReCache, arXiv 2608.19662):
 *   oracle_rope        -- RoPE with resource-local positions (Sec. 3,
 *                         "Resource-Wise Attention": pos(t_ij) = j).
 *   oracle_encode      -- block-diagonal causal attention inside each resource
 *                         (Sec. 3 "Resource-Wise Attention", Fig. 2(a)).
 *   oracle_prune       -- semantic pruning, keeping a subsequence of each
 *                         resource's cached states (Sec. 3 "Semantic Pruning").
 *   oracle_routes      -- structural pruning: per (layer, KV group) visibility
 *                         of resource states (Sec. 3 "Structural Pruning",
 *                         M_resource vs M_context; Fig. 2(b)).
 *   oracle_attend      -- conversation queries under the final ReCache mask
 *                         (Fig. 2 caption; Sec. 3 "Semantic Pruning", last
 *                         paragraph).
 *   oracle_store_offsets, oracle_store_routes
 *                      -- a resource store that holds state only for the
 *                         visible routes (both pruning stages of Sec. 3; the
 *                         memory column of the efficiency table counts it).
 *
 * Readings where the paper is silent (all listed in the design notes):
 *   RoPE pairs element i with element i + d/2 ("rotate half"); positions are
 *   0-based; the softmax scale is passed in (1/sqrt(d) by default); masked
 *   keys are removed from the softmax normaliser; a query of request b with
 *   local index i sees context rows 0 .. Tc_b - Tq_b + i (bottom-right causal
 *   alignment); visible resources enter the key stream in request order;
 *   kept rows keep the rotation they received at construction.
 *
 * Parity pins: every function here is pinned by the CPU tests against
 * independent facts (a brute-force dense N x N mask built from the Fig. 2
 * definition, PyTorch's scaled_dot_product_attention in fp64 for the special
 * cases that reduce to textbook causal attention, closed forms such as Q = 0
 * giving the mean of the visible V rows, RoPE identities, composition and
 * order invariance, and exact index comparisons).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_F32 0
#define ORACLE_BF16 1
#define ORACLE_F64 2

/* Threads the OpenMP loops below use. */
int oracle_threads(void) { return omp_get_max_threads(); }

/* Exact widening of one stored element to double. */
static double widen(const void* base, int dtype, size_t i) {
    if (dtype == ORACLE_F64) return ((const double*)base)[i];
    if (dtype == ORACLE_F32) return (double)((const float*)base)[i];
    uint32_t bits = (uint32_t)((const uint16_t*)base)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static size_t elem_size(int dtype) {
    return dtype == ORACLE_F64 ? 8 : dtype == ORACLE_F32 ? 4 : 2;
}

/* Round to nearest, ties to even, to the precision of a storage dtype: fp64
 * unchanged, fp32 via the C conversion (round-to-nearest-even), bf16 to 8
 * significant bits.  Rotated queries and keys are held at the workload's
 * storage precision, as a backbone running in that precision holds them (the
 * key cache is stored in it); everything after that is fp64. */
static double round_to(double x, int dtype) {
    if (dtype == ORACLE_F64 || x == 0.0 || !isfinite(x)) return x;
    if (dtype == ORACLE_F32) return (double)(float)x;
    int e;
    double m = frexp(x, &e);          /* x = m 2^e, 0.5 <= |m| < 1 */
    return ldexp(rint(ldexp(m, 8)), e - 8);  /* 8 significant bits, ties to even */
}

double oracle_round(double x, int dtype) { return round_to(x, dtype); }

/* ------------------------------------------------------------------------ */
/* RoPE (half-split).  For i in [0, d/2): theta_i = base^(-2i/d),
 * y_i       = x_i cos(p theta_i) - x_{i+d/2} sin(p theta_i)
 * y_{i+d/2} = x_{i+d/2} cos(p theta_i) + x_i sin(p theta_i).              */
void oracle_rope_vec(const double* x, double* y, int d, double base, double pos) {
    int half = d / 2;
    for (int i = 0; i < half; ++i) {
        double theta = pow(base, -2.0 * (double)i / (double)d);
        double c = cos(pos * theta), s = sin(pos * theta);
        double a = x[i], b = x[i + half];
        y[i] = a * c - b * s;
        y[i + half] = b * c + a * s;
    }
}

/* Rotate x[T][H][d] (stored dtype) at positions pos[T]; y[T][H][d] double,
 * each value rounded to the precision of rot_dtype. */
int oracle_rope(int dtype, int T, int H, int d, double base, const int32_t* pos,
                const void* x, double* y, int rot_dtype) {
    if (T < 0 || H <= 0 || d <= 0 || d > 512 || (d % 2) || !pos || (T && (!x || !y))) return -1;
#pragma omp parallel for schedule(static)
    for (long th = 0; th < (long)T * H; ++th) {
        long t = th / H;
        double xv[512];
        for (int e = 0; e < d; ++e) xv[e] = widen(x, dtype, (size_t)th * d + e);
        double* yr = y + (size_t)th * d;
        oracle_rope_vec(xv, yr, d, base, (double)pos[t]);
        for (int e = 0; e < d; ++e) yr[e] = round_to(yr[e], rot_dtype);
    }
    return 0;
}

/* Two-pass softmax-weighted average over n keys whose logits are z[0..n).
 * Writes out[0..d) = sum_u w_u V_u / sum_u w_u and returns the natural-log
 * sum-exp of the logits.  vrow(u) gives the u-th visible V row (double). */
typedef const double* (*vrow_fn)(void* ctx, int u, double* scratch);

static double softmax_average(const double* z, int n, int d, vrow_fn vrow, void* ctx,
                              double* out, double* scratch) {
    double m = -INFINITY;
    for (int u = 0; u < n; ++u) if (z[u] > m) m = z[u];
    double denom = 0.0;
    for (int e = 0; e < d; ++e) out[e] = 0.0;
    for (int u = 0; u < n; ++u) {
        double w = exp(z[u] - m);
        denom += w;
        const double* vr = vrow(ctx, u, scratch);
        for (int e = 0; e < d; ++e) out[e] += w * vr[e];
    }
    for (int e = 0; e < d; ++e) out[e] /= denom;
    return m + log(denom);
}

/* ------------------------------------------------------------------------ */
/* Resource encoding, one layer (Sec. 3 "Resource-Wise Attention").
 *
 * Resources are packed in order: resource r owns rows [cu_len[r], cu_len[r+1])
 * of q[T][Hq][d], k[T][Hkv][d], v[T][Hkv][d].  Token j of resource r sits at
 * position pos_base[r] + j (pos_base == NULL means 0: resource-local).
 * Query row t of resource r, head h, attends every row of the shared prefix
 * (if any) and keys u in [cu_len[r], t] of KV head h / (Hq / Hkv), with
 * logits scale * <RoPE(q_t), RoPE(k_u)>.  The shared prefix is the part of
 * the input every resource is encoded after (Sec. 3: resource tokens attend
 * the shared prefix and their local resource tokens); it is given as its
 * already rotated cache, prefix_k / prefix_v [Hkv][prefix_len][d] in the
 * input dtype, used as stored.
 *
 * Rotated queries and keys are rounded to the precision of rot_dtype (the
 * workload's storage dtype; fp64 keeps them exact).
 *
 * Outputs (double): out[T][Hq][d]; k_cache[Hkv][T][d] holds the rotated keys
 * and v_cache[Hkv][T][d] the values (head-major); lse[Hq][T] (optional)
 * holds the natural-log sum-exp of the scaled logits.                      */
struct enc_vctx {
    const double* vc; int T, d, g, row0;
    const void* pv; int p_len, dtype;
};
static const double* enc_vrow(void* c, int u, double* scratch) {
    struct enc_vctx* x = (struct enc_vctx*)c;
    if (u < x->p_len) {  /* prefix row u */
        for (int e = 0; e < x->d; ++e)
            scratch[e] = widen(x->pv, x->dtype, ((size_t)x->g * x->p_len + u) * x->d + e);
        return scratch;
    }
    return x->vc + ((size_t)x->g * x->T + x->row0 + (u - x->p_len)) * x->d;
}

int oracle_encode(int dtype, int n_res, const int32_t* cu_len, int Hq, int Hkv, int d,
                  double base, const int32_t* pos_base, double scale,
                  const void* q, const void* k, const void* v,
                  int prefix_len, const void* prefix_k, const void* prefix_v,
                  double* out, double* k_cache, double* v_cache, double* lse, int rot_dtype) {
    if (n_res <= 0 || !cu_len || Hq <= 0 || Hkv <= 0 || Hq % Hkv || d <= 0 || d > 512 ||
        (d % 2) || !q || !k || !v || !out || !k_cache || !v_cache)
        return -1;
    if (prefix_len < 0 || (prefix_len > 0 && (!prefix_k || !prefix_v))) return -1;
    if (cu_len[0] != 0) return -1;
    int max_len = 0;
    for (int r = 0; r < n_res; ++r) {
        int len = cu_len[r + 1] - cu_len[r];
        if (len <= 0) return -1;
        if (len > max_len) max_len = len;
    }
    const int T = cu_len[n_res];
    const int ratio = Hq / Hkv;

    /* Rotated key cache and plain value cache, head-major. */
#pragma omp parallel for schedule(static)
    for (long gt = 0; gt < (long)Hkv * T; ++gt) {
        int g = (int)(gt / T), t = (int)(gt % T);
        int r = 0;
        while (cu_len[r + 1] <= t) ++r;
        double p = (double)((pos_base ? pos_base[r] : 0) + (t - cu_len[r]));
        double xv[512];
        for (int e = 0; e < d; ++e) xv[e] = widen(k, dtype, ((size_t)t * Hkv + g) * d + e);
        double* kr = k_cache + ((size_t)g * T + t) * d;
        oracle_rope_vec(xv, kr, d, base, p);
        for (int e = 0; e < d; ++e) kr[e] = round_to(kr[e], rot_dtype);
        for (int e = 0; e < d; ++e)
            v_cache[((size_t)g * T + t) * d + e] = widen(v, dtype, ((size_t)t * Hkv + g) * d + e);
    }

#pragma omp parallel
    {
        double* z = (double*)malloc(sizeof(double) * ((size_t)prefix_len + max_len));
        double qv[512], qr[512], kv[512], vs[512];
#pragma omp for schedule(dynamic, 16)
        for (long th = 0; th < (long)T * Hq; ++th) {
            int t = (int)(th / Hq), h = (int)(th % Hq), g = h / ratio;
            int r = 0;
            while (cu_len[r + 1] <= t) ++r;
            int o = cu_len[r], j = t - o;
            double p = (double)((pos_base ? pos_base[r] : 0) + j);
            for (int e = 0; e < d; ++e) qv[e] = widen(q, dtype, ((size_t)t * Hq + h) * d + e);
            oracle_rope_vec(qv, qr, d, base, p);
            for (int e = 0; e < d; ++e) qr[e] = round_to(qr[e], rot_dtype);
            /* keys: the prefix rows, then rows o .. o + j of the resource */
            for (int u = 0; u < prefix_len; ++u) {
                for (int e = 0; e < d; ++e)
                    kv[e] = widen(prefix_k, dtype, ((size_t)g * prefix_len + u) * d + e);
                double dot = 0.0;
                for (int e = 0; e < d; ++e) dot += qr[e] * kv[e];
                z[u] = scale * dot;
            }
            for (int u = 0; u <= j; ++u) {
                const double* kr = k_cache + ((size_t)g * T + o + u) * d;
                double dot = 0.0;
                for (int e = 0; e < d; ++e) dot += qr[e] * kr[e];
                z[prefix_len + u] = scale * dot;
            }
            struct enc_vctx c = {v_cache, T, d, g, o, prefix_v, prefix_len, dtype};
            double l = softmax_average(z, prefix_len + j + 1, d, enc_vrow, &c,
                                       out + (size_t)th * d, vs);
            if (lse) lse[(size_t)h * T + t] = l;
        }
        free(z);
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Kept-list validation (Sec. 3 "Semantic Pruning": the retained subsequence
 * of R_i, with length at most D_i).  Indices are resource-local, strictly
 * ascending, inside [0, D_i), and every resource keeps at least one row.  */
int oracle_check_kept(int n_res, const int32_t* cu_len, const int32_t* cu_kept,
                      const int32_t* kept_idx) {
    if (n_res <= 0 || !cu_len || !cu_kept || !kept_idx) return -1;
    if (cu_kept[0] != 0 || cu_len[0] != 0) return -1;
    for (int r = 0; r < n_res; ++r) {
        int len = cu_len[r + 1] - cu_len[r];
        int a = cu_kept[r], b = cu_kept[r + 1];
        if (len <= 0 || b <= a || b - a > len) return -1;
        for (int j = a; j < b; ++j) {
            if (kept_idx[j] < 0 || kept_idx[j] >= len) return -1;
            if (j > a && kept_idx[j] <= kept_idx[j - 1]) return -1;
        }
    }
    return 0;
}

/* Semantic-pruning gather: k_kept[g][cu_kept[r] + j] = k_cache[g][cu_len[r] +
 * kept_idx[cu_kept[r] + j]], the same for v.  Stored elements are copied
 * byte for byte (the kept states are the constructed states, unchanged).   */
int oracle_prune(int dtype, int n_res, const int32_t* cu_len, const int32_t* cu_kept,
                 const int32_t* kept_idx, int Hkv, int d, const void* k_cache,
                 const void* v_cache, void* k_kept, void* v_kept) {
    if (oracle_check_kept(n_res, cu_len, cu_kept, kept_idx)) return -1;
    if (Hkv <= 0 || d <= 0 || !k_cache || !v_cache || !k_kept || !v_kept) return -1;
    const size_t es = elem_size(dtype), row = es * (size_t)d;
    const int T = cu_len[n_res], K = cu_kept[n_res];
    for (int g = 0; g < Hkv; ++g)
        for (int r = 0; r < n_res; ++r)
            for (int j = cu_kept[r]; j < cu_kept[r + 1]; ++j) {
                size_t src = ((size_t)g * T + cu_len[r] + kept_idx[j]) * row;
                size_t dst = ((size_t)g * K + j) * row;
                memcpy((char*)k_kept + dst, (const char*)k_cache + src, row);
                memcpy((char*)v_kept + dst, (const char*)v_cache + src, row);
            }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Structural pruning routes (Sec. 3 "Structural Pruning").  For request b,
 * layer l and KV group g, the visible resources are those of b's list, in
 * request order, whose route bit mask[r][l][g] is set (route in Omega ->
 * M_resource; otherwise M_context, i.e. no resource state).  Entry
 * e = (b * L + l) * G + g of the CSR gets the list and its total kept rows. */
int oracle_routes(int n_req, const int32_t* req_res_off, const int32_t* req_res, int n_res,
                  int L, int G, const uint8_t* mask, const int32_t* cu_kept,
                  int32_t* route_off, int32_t* route_res, int32_t* route_tokens) {
    if (n_req <= 0 || !req_res_off || !req_res || n_res <= 0 || L <= 0 || G <= 0 || !mask ||
        !cu_kept || !route_off || !route_res || !route_tokens)
        return -1;
    int32_t n = 0;
    route_off[0] = 0;
    for (int b = 0; b < n_req; ++b)
        for (int l = 0; l < L; ++l)
            for (int g = 0; g < G; ++g) {
                int32_t tokens = 0;
                for (int j = req_res_off[b]; j < req_res_off[b + 1]; ++j) {
                    int r = req_res[j];
                    if (r < 0 || r >= n_res) return -1;
                    if (mask[((size_t)r * L + l) * G + g]) {
                        route_res[n++] = r;
                        tokens += cu_kept[r + 1] - cu_kept[r];
                    }
                }
                size_t e = ((size_t)b * L + l) * G + g;
                route_tokens[e] = tokens;
                route_off[e + 1] = n;
            }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Conversation queries over cached resources, one layer (Fig. 2, final mask).
 *
 * q[sum Tq][Hq][d] holds rotated queries; request b owns rows
 * [cu_q[b], cu_q[b+1]).  ctx_k / ctx_v are head-major [Hkv][ctx_stride][d]
 * rotated context keys and values; request b owns rows [cu_ctx[b],
 * cu_ctx[b+1]).  res_k / res_v are head-major [Hkv][res_stride][d] resource
 * rows; resource r owns rows [cu_rows[r], cu_rows[r+1]).  If kept_idx is
 * given, the visible rows of resource r are cu_rows[r] + kept_idx[cu_kept[r]
 * + j] (semantic pruning applied by definition); otherwise every row of the
 * resource is visible (rows already compacted, or no pruning).  If store_off
 * is given (this layer's table from oracle_store_offsets), res_k / res_v are
 * a route-compacted store [rows][d] instead, and the rows of resource r for
 * group g are store_off[r * Hkv + g] + [0, cu_rows[r+1] - cu_rows[r]).
 *
 * For query i of request b (0-based within the request), head h and group
 * g = h / (Hq / Hkv), the keys are: every visible row of every resource of
 * b's list (request order) whose route bit mask[r][layer][g] is set, then
 * context rows 0 .. Tc_b - Tq_b + i.  rows_b / rows_i select which queries
 * to evaluate (n_rows of them); out[n_rows][Hq][d], lse[n_rows][Hq].       */
struct att_vctx {
    const void* res_v; const void* ctx_v; int dtype, d;
    const int64_t* key_row; /* >=0: res row index into res_v; <0: -(ctx row)-1 */
    int g; long res_stride, ctx_stride;
};
static const double* att_vrow(void* c, int u, double* scratch) {
    struct att_vctx* x = (struct att_vctx*)c;
    int64_t kr = x->key_row[u];
    const void* src = kr >= 0 ? x->res_v : x->ctx_v;
    size_t row = kr >= 0 ? (size_t)kr : (size_t)(-kr - 1);
    long stride = kr >= 0 ? x->res_stride : x->ctx_stride;
    size_t off = ((size_t)x->g * stride + row) * x->d;
    for (int e = 0; e < x->d; ++e) scratch[e] = widen(src, x->dtype, off + e);
    return scratch;
}

int oracle_attend(int dtype, int n_req, const int32_t* cu_q, const int32_t* cu_ctx,
                  int Hq, int Hkv, int d, double scale,
                  const void* q, const void* ctx_k, const void* ctx_v, long ctx_stride,
                  int n_res, const int32_t* cu_rows, long res_stride,
                  const void* res_k, const void* res_v,
                  const int32_t* cu_kept, const int32_t* kept_idx,
                  const int32_t* req_res_off, const int32_t* req_res,
                  int n_layers, int layer, const uint8_t* mask, const int32_t* store_off,
                  int n_rows, const int32_t* rows_b, const int32_t* rows_i,
                  double* out, double* lse) {
    if (n_req <= 0 || !cu_q || !cu_ctx || Hq <= 0 || Hkv <= 0 || Hq % Hkv || d <= 0 ||
        d > 512 || !q || !ctx_k || !ctx_v || n_res <= 0 || !cu_rows || !req_res_off ||
        !req_res || n_layers <= 0 || layer < 0 || layer >= n_layers || !mask || n_rows < 0 ||
        (n_rows && (!rows_b || !rows_i || !out)))
        return -1;
    if (kept_idx && oracle_check_kept(n_res, cu_rows, cu_kept, kept_idx)) return -1;
    if (store_off && kept_idx) return -1;
    /* A route-compacted store has no per-head planes: rows are absolute. */
    if (store_off) res_stride = 0;
    const int ratio = Hq / Hkv;
    long max_keys = 0;
    for (int b = 0; b < n_req; ++b) {
        int Tq = cu_q[b + 1] - cu_q[b], Tc = cu_ctx[b + 1] - cu_ctx[b];
        if (Tq < 0 || Tq > Tc) return -1;
        long nk = Tc;
        for (int j = req_res_off[b]; j < req_res_off[b + 1]; ++j) {
            int r = req_res[j];
            if (r < 0 || r >= n_res) return -1;
            nk += cu_rows[r + 1] - cu_rows[r];
        }
        if (nk > max_keys) max_keys = nk;
    }
    for (int s = 0; s < n_rows; ++s) {
        int b = rows_b[s];
        if (b < 0 || b >= n_req || rows_i[s] < 0 || rows_i[s] >= cu_q[b + 1] - cu_q[b]) return -1;
    }

#pragma omp parallel
    {
        double* z = (double*)malloc(sizeof(double) * (size_t)(max_keys + 1));
        int64_t* key_row = (int64_t*)malloc(sizeof(int64_t) * (size_t)(max_keys + 1));
        double qv[512], scratch[512];
#pragma omp for schedule(dynamic, 4)
        for (long sh = 0; sh < (long)n_rows * Hq; ++sh) {
            int s = (int)(sh / Hq), h = (int)(sh % Hq), g = h / ratio;
            int b = rows_b[s], i = rows_i[s];
            int Tq = cu_q[b + 1] - cu_q[b], Tc = cu_ctx[b + 1] - cu_ctx[b];
            for (int e = 0; e < d; ++e) qv[e] = widen(q, dtype, ((size_t)(cu_q[b] + i) * Hq + h) * d + e);
            /* Key stream: visible (kept) rows of routed resources, then causal context. */
            int n = 0;
            for (int j = req_res_off[b]; j < req_res_off[b + 1]; ++j) {
                int r = req_res[j];
                if (!mask[((size_t)r * n_layers + layer) * Hkv + g]) continue;
                if (store_off) {
                    for (int t = 0; t < cu_rows[r + 1] - cu_rows[r]; ++t)
                        key_row[n++] = (int64_t)store_off[(size_t)r * Hkv + g] + t;
                } else if (kept_idx) {
                    for (int t = cu_kept[r]; t < cu_kept[r + 1]; ++t)
                        key_row[n++] = (int64_t)cu_rows[r] + kept_idx[t];
                } else {
                    for (int t = cu_rows[r]; t < cu_rows[r + 1]; ++t) key_row[n++] = t;
                }
            }
            int last_ctx = Tc - Tq + i;
            for (int c = 0; c <= last_ctx; ++c) key_row[n++] = -(int64_t)(cu_ctx[b] + c) - 1;
            for (int u = 0; u < n; ++u) {
                int64_t kr = key_row[u];
                const void* src = kr >= 0 ? res_k : ctx_k;
                size_t row = kr >= 0 ? (size_t)kr : (size_t)(-kr - 1);
                long stride = kr >= 0 ? res_stride : ctx_stride;
                size_t off = ((size_t)g * stride + row) * d;
                double dot = 0.0;
                for (int e = 0; e < d; ++e) dot += qv[e] * widen(src, dtype, off + e);
                z[u] = scale * dot;
            }
            struct att_vctx c = {res_v, ctx_v, dtype, d, key_row, g, res_stride, ctx_stride};
            double l = softmax_average(z, n, d, att_vrow, &c, out + (size_t)sh * d, scratch);
            if (lse) lse[sh] = l;
        }
        free(z);
        free(key_row);
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Route-compacted resource store.  After both pruning stages of Sec. 3 a
 * resource's state is read only through the visible routes of Omega and only
 * at its kept positions, so only those rows need storage: for layer l, every
 * (resource r, KV group g) with mask[r][l][g] set holds the kept rows of r
 * for head g, in kept order.  Routes are laid out resource-major, (r, g) in
 * increasing r and then g, one table per layer:
 *   store_off[l][r * G + g]  first row of route (r, g) (for an invisible route
 *                            the row where it would start; it holds no rows),
 *   store_off[l][n_res * G]  rows stored for layer l.
 * The rows of a route are the kept count of r, cu_kept[r+1] - cu_kept[r].   */
int oracle_store_offsets(int n_res, int L, int G, const uint8_t* mask, const int32_t* cu_kept,
                         int32_t* store_off) {
    if (n_res <= 0 || L <= 0 || G <= 0 || !mask || !cu_kept || !store_off) return -1;
    const size_t stride = (size_t)n_res * G + 1;
    for (int l = 0; l < L; ++l) {
        int64_t run = 0;
        for (int r = 0; r < n_res; ++r)
            for (int g = 0; g < G; ++g) {
                store_off[l * stride + (size_t)r * G + g] = (int32_t)run;
                if (mask[((size_t)r * L + l) * G + g]) run += cu_kept[r + 1] - cu_kept[r];
                if (run > INT32_MAX) return -1;
            }
        store_off[l * stride + (size_t)n_res * G] = (int32_t)run;
    }
    return 0;
}

/* Fill layer `layer` of the store straight from the constructed head-major
 * caches [Hkv][T][d]: routes in (r, g) order, each appending the rows
 * cu_len[r] + kept_idx[cu_kept[r] .. cu_kept[r+1]) of head g, copied byte for
 * byte, into stores of cap_rows rows.  Returns the number of rows written
 * (the store's layer size), or -1 (bad input, or more than cap_rows rows).  */
long oracle_store_routes(int dtype, int n_res, const int32_t* cu_len, const int32_t* cu_kept,
                         const int32_t* kept_idx, int Hkv, int d, int L, int layer,
                         const uint8_t* mask, const void* k_cache, const void* v_cache,
                         void* k_store, void* v_store, long cap_rows) {
    if (oracle_check_kept(n_res, cu_len, cu_kept, kept_idx)) return -1;
    if (Hkv <= 0 || d <= 0 || L <= 0 || layer < 0 || layer >= L || !mask || !k_cache ||
        !v_cache || !k_store || !v_store)
        return -1;
    const size_t row = elem_size(dtype) * (size_t)d;
    const int T = cu_len[n_res];
    long n = 0;
    for (int r = 0; r < n_res; ++r)
        for (int g = 0; g < Hkv; ++g) {
            if (!mask[((size_t)r * L + layer) * Hkv + g]) continue;
            for (int j = cu_kept[r]; j < cu_kept[r + 1]; ++j, ++n) {
                if (n >= cap_rows) return -1;
                const size_t from = ((size_t)g * T + cu_len[r] + kept_idx[j]) * row;
                memcpy((char*)k_store + (size_t)n * row, (const char*)k_cache + from, row);
                memcpy((char*)v_store + (size_t)n * row, (const char*)v_cache + from, row);
            }
        }
    return n;
}
