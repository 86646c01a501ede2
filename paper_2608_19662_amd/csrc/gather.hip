// Index work of the method, all integer and exact:
//   - kept-row gather (ReCache Sec. 3, "Semantic Pruning"): the retained
//     subsequence of every resource, copied bit for bit into a compacted,
//     head-major buffer;
//   - route lists (Sec. 3, "Structural Pruning"): for every (request, layer,
//     KV group), the request's resources whose route is in Omega, in request
//     order, as a CSR with a per-entry kept-token total;
//   - a route-compacted store (both pruning stages): per layer, only the
//     visible (resource, group) routes hold rows, resource-major, each with
//     the kept rows of its resource.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace rc {

namespace {

// Blocks per (resource r, KV head g): n_parts of them share the kept rows of
// r for head g (contiguous, equal shares), which go to rows g * total_kept +
// cu_kept[r] + j of the compacted caches.  Each thread moves U 16-byte
// chunks per step, all loads issued before the stores; source rows are
// clamped into the caches.
__global__ __launch_bounds__(256) void prune_gather_kernel(
    int chunks_per_row, int n_kv_heads, int n_parts, const int32_t* __restrict__ cu_len,
    const int32_t* __restrict__ cu_kept, const int32_t* __restrict__ kept_idx, long total_T,
    long total_kept, const u32x4* __restrict__ kc, const u32x4* __restrict__ vc,
    u32x4* __restrict__ ko, u32x4* __restrict__ vo) {
    constexpr int U = 8;
    const int part = blockIdx.x % n_parts, rg = blockIdx.x / n_parts;
    const int r = rg / n_kv_heads, g = rg % n_kv_heads;
    const long r0 = cu_kept[r];
    const long r1 = min((long)cu_kept[r + 1], total_kept);
    if (r0 < 0 || r1 <= r0) return;
    // this block's share of the resource's kept rows
    const long k0 = r0 + (r1 - r0) * part / n_parts;
    const long k1 = r0 + (r1 - r0) * (part + 1) / n_parts;
    if (k1 <= k0) return;
    const long beg = cu_len[r];
    const int sh = __builtin_ctz(chunks_per_row);  // a power of two
    const long n = (k1 - k0) * chunks_per_row;
    const size_t src_base = (size_t)g * total_T;
    const size_t dst_base = ((size_t)g * total_kept + k0) * chunks_per_row;
    for (long c0 = threadIdx.x; c0 < n; c0 += 256 * U) {
        u32x4 kx[U], vx[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const long c = min(c0 + u * 256, n - 1);
            const long j = c >> sh;
            const int e = (int)(c & (chunks_per_row - 1));
            long src = beg + kept_idx[k0 + j];
            src = src < 0 ? 0 : (src >= total_T ? total_T - 1 : src);
            const size_t si = (src_base + src) * chunks_per_row + e;
            kx[u] = kc[si];
            vx[u] = vc[si];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const long c = c0 + u * 256;
            if (c < n) {
                ko[dst_base + c] = kx[u];
                vo[dst_base + c] = vx[u];
            }
        }
    }
}

// Entry e = (b * L + l) * G + g: count the visible resources and their kept rows.
__global__ __launch_bounds__(256) void route_count_kernel(
    int n_req, int L, int G, int n_res, const int32_t* __restrict__ req_res_off,
    const int32_t* __restrict__ req_res, const uint8_t* __restrict__ mask,
    const int32_t* __restrict__ cu_kept, int32_t* __restrict__ route_off,
    int32_t* __restrict__ route_tokens) {
    const long e = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= (long)n_req * L * G) return;
    const int g = (int)(e % G);
    const int l = (int)((e / G) % L);
    const int b = (int)(e / ((long)G * L));
    int cnt = 0, tok = 0;
#pragma unroll 4
    for (int j = req_res_off[b]; j < req_res_off[b + 1]; ++j) {
        const int r = req_res[j];
        if (r < 0 || r >= n_res) continue;
        if (mask[((size_t)r * L + l) * G + g]) {
            ++cnt;
            tok += cu_kept[r + 1] - cu_kept[r];
        }
    }
    route_off[e + 1] = cnt;
    route_tokens[e] = tok;
}

// In-place inclusive scan of route_off[1..E] by one block; route_off[0] = 0.
// The entries go through in chunks of 4096 consecutive ones, four per thread
// (coalesced loads and stores), with a block-wide scan of the thread sums per
// chunk and the chunk totals carried on.
__global__ __launch_bounds__(1024) void route_scan_kernel(long E, int32_t* __restrict__ route_off) {
    constexpr int V = 4;
    __shared__ int wave_tot[2][16];  // alternate buffers: one barrier per chunk suffices
    const int tid = threadIdx.x;
    int carry = 0, k = 0;
    for (long base = 1; base <= E; base += 1024L * V, k ^= 1) {
        const long i0 = base + (long)tid * V;
        int v[V], s = 0;
#pragma unroll
        for (int j = 0; j < V; ++j) {
            v[j] = i0 + j <= E ? route_off[i0 + j] : 0;
            s += v[j];
        }
        int total;
        int run = carry + block_exclusive_scan<16>(s, wave_tot[k], &total);
#pragma unroll
        for (int j = 0; j < V; ++j) {
            run += v[j];
            if (i0 + j <= E) route_off[i0 + j] = run;
        }
        carry += total;
    }
    if (tid == 0) route_off[0] = 0;
}

__global__ __launch_bounds__(256) void route_fill_kernel(
    int n_req, int L, int G, int n_res, const int32_t* __restrict__ req_res_off,
    const int32_t* __restrict__ req_res, const uint8_t* __restrict__ mask,
    const int32_t* __restrict__ route_off, int32_t* __restrict__ route_res) {
    const long e = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= (long)n_req * L * G) return;
    const int g = (int)(e % G);
    const int l = (int)((e / G) % L);
    const int b = (int)(e / ((long)G * L));
    int w = route_off[e];
#pragma unroll 4
    for (int j = req_res_off[b]; j < req_res_off[b + 1]; ++j) {
        const int r = req_res[j];
        if (r < 0 || r >= n_res) continue;
        if (mask[((size_t)r * L + l) * G + g]) route_res[w++] = r;
    }
}

// One block per layer: exclusive scan over routes i = r * G + g of
// mask[r][l][g] * kept_r, written to the layer's row of the table, plus the
// layer's total.  The routes go through in chunks of 4096 consecutive ones,
// four per thread, with a block-wide scan of the thread sums per chunk and
// the chunk totals carried on.
__global__ __launch_bounds__(1024) void store_offsets_kernel(
    int n_res, int L, int G, const uint8_t* __restrict__ mask,
    const int32_t* __restrict__ cu_kept, int32_t* __restrict__ store_off) {
    constexpr int V = 4;
    __shared__ int wave_tot[2][16];  // alternate buffers: one barrier per chunk suffices
    const int l = blockIdx.x, tid = threadIdx.x;
    const long n = (long)n_res * G;
    int32_t* off = store_off + (size_t)l * (n + 1);
    auto rows = [&](long i) {
        const int r = (int)(i / G), g = (int)(i % G);
        return mask[((size_t)r * L + l) * G + g] ? cu_kept[r + 1] - cu_kept[r] : 0;
    };
    int carry = 0, k = 0;
    for (long base = 0; base < n; base += 1024L * V, k ^= 1) {
        const long i0 = base + (long)tid * V;
        int v[V], s = 0;
#pragma unroll
        for (int j = 0; j < V; ++j) {
            v[j] = i0 + j < n ? rows(i0 + j) : 0;
            s += v[j];
        }
        int total;
        int run = carry + block_exclusive_scan<16>(s, wave_tot[k], &total);
#pragma unroll
        for (int j = 0; j < V; ++j) {
            if (i0 + j < n) off[i0 + j] = run;
            run += v[j];
        }
        carry += total;
    }
    if (tid == 0) off[n] = carry;
}

// One block per route i = r * G + g of the layer: a visible route copies
// the kept rows of r for head g to store rows off[i] .. off[i + 1]; an
// invisible route (no rows) exits at once.  Each thread moves U 16-byte
// chunks per step, all loads issued before the stores.
__global__ __launch_bounds__(256) void store_routes_kernel(
    int chunks_per_row, int G, const int32_t* __restrict__ off,
    const int32_t* __restrict__ cu_len, const int32_t* __restrict__ cu_kept,
    const int32_t* __restrict__ kept_idx, long total_T, long total_kept, long store_rows,
    const u32x4* __restrict__ kc, const u32x4* __restrict__ vc, u32x4* __restrict__ ko,
    u32x4* __restrict__ vo) {
    constexpr int U = 8;
    const int i = blockIdx.x;
    const int o0 = off[i];
    const int n_rows = off[i + 1] - o0;
    if (n_rows <= 0 || o0 < 0) return;
    const int r = i / G, g = i % G;
    const long k0 = cu_kept[r];
    const long row0 = (long)g * total_T;
    const long beg = cu_len[r];
    // rows past the end of the store (an inconsistent table) are not written
    const long n = min((long)n_rows, store_rows - o0) * chunks_per_row;
    for (long c0 = threadIdx.x; c0 < n; c0 += 256 * U) {
        u32x4 kx[U], vx[U];
        size_t dst[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const long c = min(c0 + u * 256, n - 1);
            const int sh = __builtin_ctz(chunks_per_row);  // a power of two
            const long j = c >> sh;
            const int e = (int)(c & (chunks_per_row - 1));
            const long kj = min(k0 + j, total_kept - 1);
            long src = beg + kept_idx[kj];
            src = src < 0 ? 0 : (src >= total_T ? total_T - 1 : src);
            const size_t s = (size_t)(row0 + src) * chunks_per_row + e;
            kx[u] = kc[s];
            vx[u] = vc[s];
            dst[u] = (size_t)(o0 + j) * chunks_per_row + e;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (c0 + u * 256 < n) {
                ko[dst[u]] = kx[u];
                vo[dst[u]] = vx[u];
            }
        }
    }
}

}  // namespace

hipError_t launch_store_offsets(int n_res, int n_layers, int n_kv_heads, const uint8_t* mask,
                                const int32_t* cu_kept, int32_t* store_off, hipStream_t s) {
    hipLaunchKernelGGL(store_offsets_kernel, dim3(n_layers), dim3(1024), 0, s, n_res, n_layers,
                       n_kv_heads, mask, cu_kept, store_off);
    return hipGetLastError();
}

hipError_t launch_store_routes(int elem_bytes, int layer, int n_res, const int32_t* cu_len,
                               const int32_t* cu_kept, const int32_t* kept_idx, long total_T,
                               long total_kept, int n_kv_heads, int head_dim,
                               const int32_t* store_off, long store_rows, const void* k_cache,
                               const void* v_cache, void* k_store, void* v_store, hipStream_t s) {
    if (store_rows == 0) return hipSuccess;
    const int cpr = head_dim * elem_bytes / 16;
    const long n_routes = (long)n_res * n_kv_heads;
    if (n_routes > 0x7fffffffL) return hipErrorInvalidValue;
    hipLaunchKernelGGL(store_routes_kernel, dim3((unsigned)n_routes), dim3(256), 0, s, cpr,
                       n_kv_heads, store_off + (size_t)layer * (n_routes + 1), cu_len, cu_kept,
                       kept_idx, total_T, total_kept, store_rows, static_cast<const u32x4*>(k_cache),
                       static_cast<const u32x4*>(v_cache), static_cast<u32x4*>(k_store),
                       static_cast<u32x4*>(v_store));
    return hipGetLastError();
}

hipError_t launch_prune_gather(int elem_bytes, int n_res, const int32_t* cu_len,
                               const int32_t* cu_kept, const int32_t* kept_idx, long total_T,
                               long total_kept, int n_kv_heads, int head_dim, const void* k_cache,
                               const void* v_cache, void* k_kept, void* v_kept, hipStream_t s) {
    const int cpr = head_dim * elem_bytes / 16;
    const long rg = (long)n_res * n_kv_heads;
    if (rg == 0) return hipSuccess;
    // about 2048 blocks (eight per CU) whatever the resource count
    const int parts = (int)std::min(16L, std::max(1L, (2048 + rg - 1) / rg));
    const long blocks = rg * parts;
    if (blocks > 0x7fffffffL) return hipErrorInvalidValue;
    hipLaunchKernelGGL(prune_gather_kernel, dim3((unsigned)blocks), dim3(256), 0, s, cpr, n_kv_heads, parts,
                       cu_len, cu_kept, kept_idx, total_T, total_kept,
                       static_cast<const u32x4*>(k_cache), static_cast<const u32x4*>(v_cache),
                       static_cast<u32x4*>(k_kept), static_cast<u32x4*>(v_kept));
    return hipGetLastError();
}

hipError_t launch_build_routes(int n_req, const int32_t* req_res_off, const int32_t* req_res,
                               int n_res, int n_layers, int n_kv_heads, const uint8_t* mask,
                               const int32_t* cu_kept, int32_t* route_off, int32_t* route_res,
                               int32_t* route_tokens, hipStream_t s) {
    const long E = (long)n_req * n_layers * n_kv_heads;
    const unsigned blocks = (unsigned)((E + 255) / 256);
    hipLaunchKernelGGL(route_count_kernel, dim3(blocks), dim3(256), 0, s, n_req, n_layers,
                       n_kv_heads, n_res, req_res_off, req_res, mask, cu_kept, route_off,
                       route_tokens);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(route_scan_kernel, dim3(1), dim3(1024), 0, s, E, route_off);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(route_fill_kernel, dim3(blocks), dim3(256), 0, s, n_req, n_layers,
                       n_kv_heads, n_res, req_res_off, req_res, mask, route_off, route_res);
    return hipGetLastError();
}

}  // namespace rc
