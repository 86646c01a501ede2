// Work order of the attend kernels: for every layer, the (request, KV
// group) pairs of a batch sorted by their work, longest first, and dealt in
// snake order over the KV-group positions of the grid.
//
// The method itself fixes no order (ReCache Sec. 3, "Structural Pruning",
// only says which kept rows each (request, layer, group) sees); the order is
// a schedule.  Routed resources make the pairs' key streams unequal, so a
// grid that takes the pairs in request order ends on a tail of long streams
// (decode) or hands some XCDs more work than others (prefill, where the
// blocks of one grid position of the KV group share an XCD).  Taking the
// pairs longest first, and dealing each row of G of them to the G positions
// in alternating direction, evens both out.
//
// One block per layer: the work of every pair (in key tiles, by the cost
// model of the attention kernels), a bitonic sort of (work, pair) keys in
// LDS, then the dealt order.  Keys are unique (ties fall to the lower pair
// index), so the order is deterministic.
#include "common.hpp"
#include "kernels.hpp"

namespace rc {

namespace {

constexpr int kPlanThreads = 1024;

__global__ __launch_bounds__(kPlanThreads) void attend_plan_kernel(const PlanArgs a) {
    __shared__ uint64_t key[kMaxPlanPairs];
    const int layer = blockIdx.x;
    const int G = a.n_kv_heads;
    const int n = a.n_req * G;
    int np2 = 1;
    while (np2 < n) np2 <<= 1;

    for (int i = threadIdx.x; i < np2; i += kPlanThreads) {
        uint64_t k = 0;  // padding sorts last
        if (i < n) {
            const int b = i / G, g = i % G;
            const int q_len = a.cu_q[b + 1] - a.cu_q[b];
            const int tc = a.cu_ctx[b + 1] - a.cu_ctx[b];
            const int s_vis = a.route_tokens[((size_t)b * a.n_layers + layer) * G + g];
            // Cost in 64-key tiles: the query tiles of wg_rows rows each see
            // the keys up to their last row (stream positions <= off + row),
            // plus a fixed cost per block.
            long work = 0;
            if (q_len > 0) {
                const long off = (long)s_vis + tc - q_len;
                for (long r0 = 0; r0 < q_len; r0 += a.wg_rows) {
                    const long last = min(r0 + a.wg_rows, (long)q_len) - 1;
                    work += max(off + last, 0L) / 64 + 1 + kPlanBlockCost;
                }
            }
            if (work > 0x7fffffffL) work = 0x7fffffffL;
            k = ((uint64_t)work << 32) | (uint64_t)(0xffffffffu - (uint32_t)i);
        }
        key[i] = k;
    }
    __syncthreads();
    // bitonic sort, descending
    for (int size = 2; size <= np2; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = threadIdx.x; i < np2; i += kPlanThreads) {
                const int j = i ^ stride;
                if (j > i) {
                    const uint64_t x = key[i], y = key[j];
                    // blocks of `size` alternate direction; the block holding
                    // index 0 sorts descending, and so does the final pass
                    const bool desc = (i & size) == 0;
                    if (desc ? (x < y) : (x > y)) {
                        key[i] = y;
                        key[j] = x;
                    }
                }
            }
            __syncthreads();
        }
    }
    // deal: sorted position k goes to grid row k / G, position k % G in even
    // rows and G - 1 - k % G in odd rows
    int32_t* out = a.plan + (size_t)layer * n;
    for (int k = threadIdx.x; k < n; k += kPlanThreads) {
        const int pair = (int)(0xffffffffu - (uint32_t)(key[k] & 0xffffffffu));
        const int row = k / G, c = k % G;
        out[row * G + ((row & 1) ? G - 1 - c : c)] = pair;
    }
}

}  // namespace

hipError_t launch_attend_plan(const PlanArgs& a, hipStream_t stream) {
    if (a.n_req < 1 || a.n_kv_heads < 1 || a.n_layers < 1 || a.wg_rows < 1 ||
        (long)a.n_req * a.n_kv_heads > kMaxPlanPairs)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(attend_plan_kernel, dim3((unsigned)a.n_layers), dim3(kPlanThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace rc
