"""Benchmark of the resource-wise attention hot path on one MI355X.

Headline workload (one JSON line): conversation prefill over cached resources
at the Qwen3-4B attention shape -- 36 layers, 8 requests, each with 8
retrieved resources of U[300, 1200] tokens (all routes visible, no pruning)
and 2048 context tokens causal over themselves; 32 query / 8 KV heads,
head_dim 128, bf16.  One step is the whole pass over the 36 layers: one call
of the library's attend entry point per layer, each launching the MFMA
attention kernel once.  value = effective TFLOP/s = 4 * head_dim * (unmasked
(query, key) pairs per query head, summed over requests, layers and heads) /
step time.  The roofline block is that kernel's: algorithmic FLOPs over its
average launch duration, timed with HIP events on the launch stream around
the timed region.

The same run also measures the other hot-path steps on their own workloads
("rows"), each with a roofline block for its dominant kernel: resource
encoding (one layer, 16 resources of U[200, 1500]), the pruned prefill (25%
of routes, 30% of tokens), batched decode (36 layers, 64 requests over 32
resources each plus 4096 context rows), the kept-row gather, the route build,
a shared-prefix encode, a route-compacted store and the Dense baselines.

Inputs are synthetic (seeded N(0, 1) tensors, see workloads.py) and resident
in HBM before timing starts.  The CPU baseline is the fp64 oracle on one
layer of the headline workload, extrapolated to the 36-layer step.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E
PREWARM_S = 0.3            # untimed load before the headline's warm-up steps (clock ramp)
METRIC = "effective attention TFLOP/s (prefill) & HBM GB/s (decode), % of MI355X peak"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def i32(a, dev):
    import torch

    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, np.int32))).to(dev)


def encode_flops(w) -> float:
    return 4.0 * w.head_dim * w.n_q_heads * w.pairs_per_head()


def encode_row(dev, steps, warmup):
    """Resource encoding (16 resources, one layer): the whole step (one
    recache_encode_resources call: RoPE of K with the cache write, then the
    block-diagonal attention with the query RoPE fused in) and the attention
    kernel alone, each timed with events over back-to-back launches."""
    import torch
    from paper_2608_19662_amd import recache as rc
    from paper_2608_19662_amd.workloads import config

    w = config(2)["encode"]
    T, Hq, Hkv, d = w.total, w.n_q_heads, w.n_kv_heads, w.head_dim
    q, k, v = w.tensors(dev)
    cu = i32(w.cu_len, dev)
    pos = i32(np.concatenate([np.arange(n) for n in w.lengths]), dev)  # resource-local positions
    out = torch.empty_like(q)
    kc = torch.empty(Hkv, T, d, dtype=q.dtype, device=dev)
    vc = torch.empty_like(kc)
    max_len = int(w.lengths.max())
    stream = torch.cuda.current_stream()

    def step():
        rc.encode_resources(q, k, v, cu, max_len, w.rope_base, out, kc, vc)

    def attention():
        rc.encode_attention(q, kc, vc, cu, max_len, w.rope_base, out)

    flops = encode_flops(w)
    ms = timed(step, steps, warm=warmup, prewarm_s=PREWARM_S)
    attn_ms = timed(attention, steps, warm=warmup, prewarm_s=0.1)
    # one RoPE launch takes about 20 us, close to what the host needs to
    # issue it: queue the timed launches behind a 4 GiB fill so that they run
    # back to back
    spacer = torch.empty(1 << 30, dtype=torch.float32, device=dev)
    rope_ms = timed(lambda: rc.rope_kv(k, v, pos, w.rope_base, kc, vc), max(steps, 20), warm=warmup,
                    prewarm_s=0.1, queue_behind=lambda: spacer.fill_(0.0))
    del spacer
    rope_bytes = 4.0 * T * Hkv * d * 2  # read K and V, write both caches
    # The working set (about 330 MB) exceeds the 256 MB last-level cache, so
    # back-to-back steps still find part of it there.  For reference, time
    # steps that each follow a 512 MB write (outside the timed interval),
    # which leaves none of the inputs in that cache, and as a control the
    # same isolated steps (synchronised, events around each) without the write.
    flush = torch.empty(512 << 18, dtype=torch.float32, device=dev)
    cold, isolated = [], []
    for i in range(20):
        if i % 2 == 0:
            flush.fill_(1.0)
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record(stream)
        step()
        e[1].record(stream)
        torch.cuda.synchronize()
        (cold if i % 2 == 0 else isolated).append(e[0].elapsed_time(e[1]))
    del flush
    cold_ms = float(np.median(cold))
    isolated_ms = float(np.median(isolated))
    nbytes = 2.0 * T * d * 2 * (Hq + Hkv)  # Q and O, K and V caches once
    res = {"workload": "config 2: resource encoding, 1 layer, 16 packed resources U[200,1500] "
                       "(%d tokens), 32 q / 8 KV heads, head_dim 128, bf16, RoPE base 1e6" % T,
           "ms_per_step": ms, "tflops": flops / (ms * 1e-3) / 1e12, "flops": flops,
           "pairs_per_head": w.pairs_per_head(), "launches": steps,
           "step": "one recache_encode_resources call: RoPE of K at resource-local positions "
                   "with the head-major cache write, then block-diagonal causal attention with "
                   "fused query RoPE",
           "rope_kv_ms": rope_ms,
           "rope_kv_gbs": rope_bytes / (rope_ms * 1e-3) / 1e9,
           "roofline": roofline("attn_mfma_kernel<128, encode>", "mfma", flops, attn_ms,
                                traffic=measured_traffic(ENCODE_TRAFFIC), launches=steps,
                                algorithmic_bytes=nbytes),
           "cold_cache": {"ms_per_step": round(cold_ms, 5),
                          "tflops": round(flops / (cold_ms * 1e-3) / 1e12, 3),
                          "isolated_warm_ms_per_step": round(isolated_ms, 5),
                          "note": "median of 10 steps, each after a 512 MB write that evicts "
                                  "the inputs from the last-level cache; events around the "
                                  "step. Control: median of 10 such isolated steps without "
                                  "the write"}}
    res["pct_of_peak"] = 100.0 * res["tflops"] / PEAK_BF16_TFLOPS
    del q, k, v, out, kc, vc
    torch.cuda.empty_cache()
    return res


def roofline(kernel, bound, work, avg_ms, traffic=None, launches=None, algorithmic_bytes=None):
    """Roofline block of a kernel: work (FLOPs for "mfma", bytes for "hbm")
    per launch over its average launch duration avg_ms."""
    if bound == "mfma":
        achieved, peak, unit = work / (avg_ms * 1e-3) / 1e12, PEAK_BF16_TFLOPS, "TFLOP/s"
    else:
        achieved, peak, unit = work / (avg_ms * 1e-3) / 1e9, PEAK_HBM_GBS, "GB/s"
    r = {"kernel": kernel, "bound": bound, "achieved": round(achieved, 3), "peak": peak,
         "unit": unit, "frac": round(achieved / peak, 4), "traffic": traffic,
         "avg_kernel_ms": round(avg_ms, 5),
         ("flops_per_launch" if bound == "mfma" else "bytes_per_launch"): work}
    if launches is not None:
        r["launches_timed"] = launches
    if algorithmic_bytes is not None and bound == "mfma":
        r["algorithmic_bytes_per_launch"] = algorithmic_bytes
    return r


def timed(fn, reps, warm=1, prewarm_s=0.1, queue_behind=None):
    """Mean wall time of fn over reps calls (HIP events on the current
    stream), after warm calls and at least prewarm_s of untimed calls (the
    GPU raises its clocks only after some time under load).  queue_behind,
    if given, is enqueued untimed just before the first event: GPU work that
    outlasts the host's launch of the reps calls, so that short kernels run
    back to back instead of waiting on their launches."""
    import torch

    t_end = time.perf_counter() + prewarm_s
    n = 0
    while n < warm or time.perf_counter() < t_end:
        fn()
        torch.cuda.synchronize()
        n += 1
    s = torch.cuda.current_stream()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if queue_behind is not None:
        queue_behind()
    a.record(s)
    for _ in range(reps):
        fn()
    b.record(s)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


def visible_tokens(w):
    """S_vis[b][l][g]: kept rows of b's resources whose route (l, g) is set."""
    kl = w.kept_lengths.astype(np.int64)
    s = np.zeros((w.n_req, w.n_layers, w.n_kv_heads), np.int64)
    for b in range(w.n_req):
        rs = w.req_res[w.req_res_off[b]:w.req_res_off[b + 1]]
        s[b] = np.einsum("r,rlg->lg", kl[rs], w.mask[rs].astype(np.int64))
    return s


def prefill_pairs(w):
    """Unmasked (query, key) pairs per (request, layer, query head):
    Tq * S_vis + Tq (Tq + 1) / 2 + Tq (Tc - Tq)."""
    s_vis = visible_tokens(w)
    tq = w.q_lens.astype(np.int64)[:, None, None]
    tc = w.ctx_lens.astype(np.int64)[:, None, None]
    return tq * s_vis + tq * (tq + 1) // 2 + tq * (tc - tq)


def prefill_setup(k, dev):
    """Config k's 36 layers resident in HBM, its route CSR, and one pass."""
    import torch
    from paper_2608_19662_amd import recache as rc
    from paper_2608_19662_amd.workloads import config

    w = config(k)["attend"]
    L, r = w.n_layers, w.n_q_heads // w.n_kv_heads
    flops = 4.0 * w.head_dim * r * float(prefill_pairs(w).sum())
    # algorithmic bytes of one launch (mean over layers): Q in, O out, and K
    # and V of every route-visible kept row and every context row once per
    # (request, KV group)
    kv_rows = float(visible_tokens(w).sum()) / L + float(w.cu_ctx[-1]) * w.n_kv_heads
    nbytes = (2.0 * float(w.cu_q[-1]) * w.n_q_heads + 2.0 * kv_rows) * w.head_dim * 2
    layers = [w.layer_tensors(l, dev) for l in range(L)]
    outs = [torch.empty_like(t[0]) for t in layers]
    st = _routes(w, dev)

    def run():
        for l in range(L):
            q, ck, cv, rk, rv = layers[l]
            rc.attend_cached(q, ck, cv, st["cu_q"], st["cu_ctx"], int(w.q_lens.max()),
                             int(w.ctx_lens.max()), rk, rv, st["cu_rows"], st["route_off"],
                             st["route_res"], st["route_tokens"], l, L, outs[l],
                             max_route_len=st["max_route_len"], plan=st["plan"])

    return w, flops, nbytes, layers, outs, run


def prefill_row(k, dev, reps):
    import torch

    w, flops, nbytes, layers, outs, run = prefill_setup(k, dev)
    L = w.n_layers
    ms = timed(run, reps)
    res = {"workload": "config %d" % k, "layers": L, "ms_per_pass": ms,
           "tflops": flops / (ms * 1e-3) / 1e12, "flops": flops,
           "roofline": roofline("attn_mfma_kernel<128, attend>", "mfma", flops / L, ms / L,
                                traffic=measured_traffic(PREFILL_TRAFFIC[k]), launches=reps * L,
                                algorithmic_bytes=nbytes)}
    res["pct_of_peak"] = 100.0 * res["tflops"] / PEAK_BF16_TFLOPS
    del layers, outs
    torch.cuda.empty_cache()
    return res


def _routes(w, dev):
    import torch
    from paper_2608_19662_amd import recache as rc

    E = w.n_req * w.n_layers * w.n_kv_heads
    st = {"cu_q": i32(w.cu_q, dev), "cu_ctx": i32(w.cu_ctx, dev), "cu_rows": i32(w.cu_rows, dev),
          "route_off": torch.empty(E + 1, dtype=torch.int32, device=dev),
          "route_res": torch.empty(int(w.req_res_off[-1]) * w.n_layers * w.n_kv_heads,
                                   dtype=torch.int32, device=dev),
          "route_tokens": torch.empty(E, dtype=torch.int32, device=dev),
          "max_route_len": int(np.diff(w.req_res_off).max())}
    st["args"] = (i32(w.req_res_off, dev), i32(w.req_res, dev),
                  torch.from_numpy(w.mask).to(dev), st["cu_rows"], st["route_off"],
                  st["route_res"], st["route_tokens"])
    rc.build_routes(*st["args"])
    st["plan"] = None
    if USE_PLAN:
        st["plan"] = torch.empty(w.n_layers, w.n_req * w.n_kv_heads, dtype=torch.int32, device=dev)
        st["plan_args"] = (st["cu_q"], st["cu_ctx"], st["route_tokens"], w.n_layers, w.n_q_heads,
                           w.n_kv_heads, st["plan"])
        rc.attend_plan(*st["plan_args"])
    return st


def decode_row(dev, reps):
    import torch
    from paper_2608_19662_amd import recache as rc
    from paper_2608_19662_amd.workloads import config

    w = config(5)["attend"]
    L, G, d = w.n_layers, w.n_kv_heads, w.head_dim
    s_vis = visible_tokens(w)
    keys = s_vis + w.ctx_lens.astype(np.int64)[:, None, None]
    kv_bytes = float(keys.sum()) * 2 * d * 2
    qo_bytes = 2.0 * L * w.n_req * w.n_q_heads * d * 2
    max_kv = int(keys.max())
    layers = []
    for l in range(L):
        layers.append(w.layer_tensors(l, dev))
    outs = [torch.empty_like(t[0]) for t in layers]
    st = _routes(w, dev)
    nb = rc.attend_workspace_bytes(w.n_req, 1, int(w.ctx_lens.max()), max_kv, w.n_q_heads, G, d)
    ws = torch.empty(nb // 4, dtype=torch.float32, device=dev)

    def run():
        for l in range(L):
            q, ck, cv, rk, rv = layers[l]
            rc.attend_cached(q, ck, cv, st["cu_q"], st["cu_ctx"], 1, int(w.ctx_lens.max()), rk, rv,
                             st["cu_rows"], st["route_off"], st["route_res"], st["route_tokens"], l,
                             L, outs[l], workspace=ws, max_kv=max_kv,
                             max_route_len=st["max_route_len"], plan=st["plan"])

    ms = timed(run, reps)
    gbs = (kv_bytes + qo_bytes) / (ms * 1e-3) / 1e9
    # both take a few tens of microseconds, close to what the host needs to
    # issue their launches: queue the timed calls behind a 4 GiB fill so that
    # they run back to back
    spacer = torch.empty(1 << 30, dtype=torch.float32, device=dev)
    fill = lambda: spacer.fill_(0.0)
    route_ms = timed(lambda: rc.build_routes(*st["args"]), max(reps, 20), queue_behind=fill)
    plan_ms = (timed(lambda: rc.attend_plan(*st["plan_args"]), max(reps, 20), queue_behind=fill)
               if USE_PLAN else None)
    del spacer
    res = {"workload": "config 5", "layers": L, "ms_per_step": ms, "gbs": gbs,
           "pct_of_peak": 100.0 * gbs / PEAK_HBM_GBS, "bytes": kv_bytes + qo_bytes,
           "resident_gb": sum(t.numel() * t.element_size() for lt in layers for t in lt) / 1e9,
           # per layer: one decode_kernel launch and its ~5 us split merge
           # (combine_kernel), timed together; the bytes are the decode
           # kernel's algorithmic bytes, so the fraction slightly understates it
           "roofline": roofline("decode_kernel<128>", "hbm", (kv_bytes + qo_bytes) / L, ms / L,
                                traffic=measured_traffic(DECODE_TRAFFIC), launches=reps * L)}
    del layers, outs
    torch.cuda.empty_cache()
    return res, {"workload": "config 5 (64 req x 36 layers x 8 groups)", "ms": route_ms,
                 "entries": int(w.n_req * L * G), "plan_ms_36_layers": plan_ms}


def route_store_row(dev, reps):
    """Config 5 with resource state in a route-compacted store: row tables,
    the fused kept-row + route gather of every layer, decode over the store,
    and the allocated resource-KV bytes against the unpruned all-route cache
    (and, for the paper's Omega*_{20,3} of Qwen3-4B, the same accounting)."""
    import torch
    from paper_2608_19662_amd import recache as rc
    from paper_2608_19662_amd.workloads import (OMEGA_20_3_QWEN3_4B_GROUPS,
                                                OMEGA_20_3_QWEN3_4B_LAYERS, config, normal,
                                                omega_star_mask)

    w = config(5)["attend"]
    L, G, d = w.n_layers, w.n_kv_heads, w.head_dim
    n_res = len(w.lengths)
    T, K = int(w.cu_len[-1]), int(w.cu_kept[-1])
    st = _routes(w, dev)
    mask_d = st["args"][2]
    off = torch.empty(L, n_res * G + 1, dtype=torch.int32, device=dev)
    off_ms = timed(lambda: rc.route_store_offsets(mask_d, st["cu_rows"], off, total_kept=K), reps)
    rows = off[:, -1].cpu().numpy().astype(np.int64)
    # one layer's constructed caches serve as the gather source of every layer
    kc = normal((G, T, d), torch.bfloat16, 5, 950, dev)
    vc = normal((G, T, d), torch.bfloat16, 5, 951, dev)
    ks = [torch.empty(int(n), d, dtype=torch.bfloat16, device=dev) for n in rows]
    vs = [torch.empty_like(t) for t in ks]
    idx = (i32(w.cu_len, dev), st["cu_rows"], i32(w.kept_idx, dev))

    def build():
        for l in range(L):
            rc.store_routes(kc, vc, *idx, off, l, ks[l], vs[l], total_kept=K)

    build_ms = timed(build, reps)
    build_bytes = 2.0 * 2 * float(rows.sum()) * d * 2  # read + write of K and V rows
    del kc, vc
    torch.cuda.empty_cache()

    s_vis = visible_tokens(w)
    keys = s_vis + w.ctx_lens.astype(np.int64)[:, None, None]
    io_bytes = float(keys.sum()) * 2 * d * 2 + 2.0 * L * w.n_req * w.n_q_heads * d * 2
    max_kv = int(keys.max())
    layers = [w.layer_tensors(l, dev)[:3] for l in range(L)]
    torch.cuda.empty_cache()
    outs = [torch.empty_like(t[0]) for t in layers]
    nb = rc.attend_workspace_bytes(w.n_req, 1, int(w.ctx_lens.max()), max_kv, w.n_q_heads, G, d)
    ws = torch.empty(nb // 4, dtype=torch.float32, device=dev)

    def run():
        for l in range(L):
            q, ck, cv = layers[l]
            rc.attend_cached(q, ck, cv, st["cu_q"], st["cu_ctx"], 1, int(w.ctx_lens.max()), ks[l],
                             vs[l], st["cu_rows"], st["route_off"], st["route_res"],
                             st["route_tokens"], l, L, outs[l], workspace=ws, max_kv=max_kv,
                             max_route_len=st["max_route_len"], res_off=off[l], plan=st["plan"])

    ms = timed(run, reps)
    gbs = io_bytes / (ms * 1e-3) / 1e9
    row_bytes = 2 * d * 2  # K and V, bf16
    unpruned = float(L * G * T * row_bytes)
    all_routes = float(L * G * K * row_bytes)
    stored = float(rows.sum() * row_bytes)
    paper_mask = omega_star_mask(n_res, L, G, OMEGA_20_3_QWEN3_4B_LAYERS,
                                 OMEGA_20_3_QWEN3_4B_GROUPS)
    kept = np.diff(w.cu_kept).astype(np.int64)
    paper_rows = float(np.einsum("r,rlg->", kept, paper_mask.astype(np.int64)))
    res = {"workload": "config 5, resource state in a route-compacted store", "layers": L,
           "ms_per_step": ms, "gbs": gbs, "pct_of_peak": 100.0 * gbs / PEAK_HBM_GBS,
           "bytes": io_bytes, "store_offsets_ms": off_ms, "store_build_ms_36_layers": build_ms,
           "store_build_gbs": build_bytes / (build_ms * 1e-3) / 1e9,
           "mem": {"unpruned_all_routes_gb": unpruned / 1e9,
                   "kept_all_routes_gb": all_routes / 1e9,
                   "route_store_gb": stored / 1e9,
                   "reduction_vs_unpruned_pct": 100.0 * (1 - stored / unpruned),
                   "omega_20_3_qwen3_4b_store_gb": paper_rows * row_bytes / 1e9,
                   "omega_20_3_qwen3_4b_reduction_pct":
                       100.0 * (1 - paper_rows * row_bytes / unpruned)}}
    del layers, outs, ks, vs
    torch.cuda.empty_cache()
    return res


def prune_row(dev, reps):
    import torch
    from paper_2608_19662_amd import recache as rc
    from paper_2608_19662_amd.workloads import config, normal

    w = config(4)["attend"]
    T, K, d = int(w.cu_len[-1]), int(w.cu_kept[-1]), w.head_dim
    kc = normal((8, T, d), torch.bfloat16, 4, 900, dev)
    vc = normal((8, T, d), torch.bfloat16, 4, 901, dev)
    kk = torch.empty(8, K, d, dtype=torch.bfloat16, device=dev)
    vk = torch.empty_like(kk)
    a = (i32(w.cu_len, dev), i32(w.cu_kept, dev), i32(w.kept_idx, dev))
    # One launch takes about 25 us, close to what the host needs to issue it:
    # queue the timed launches behind a 4 GiB fill (about 1 ms) so that they
    # run back to back.
    spacer = torch.empty(1 << 30, dtype=torch.float32, device=dev)
    reps = max(reps, 20)
    ms = timed(lambda: rc.prune_gather(kc, vc, *a, kk, vk), reps,
               queue_behind=lambda: spacer.fill_(0.0))
    del spacer
    nbytes = 2.0 * 2 * 8 * K * d * 2  # read + write of K and V kept rows
    return {"workload": "config 4, one layer", "ms": ms, "gbs": nbytes / (ms * 1e-3) / 1e9,
            "pct_of_peak": 100.0 * nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, "rows_kept": K,
            "launches": reps, "note": "back-to-back launches queued behind a fill"}


# attend with the per-batch work order (recache_attend_plan), built with the
# routes, outside the timed steps like them
USE_PLAN = True

PROFILES = os.path.join(ROOT, "profiles")
ENCODE_TRAFFIC = ("attn_mfma_encode_config2_traffic.md", ("attn_mfma.hip", "common.hpp", "kernels.hpp"))
PREFILL_TRAFFIC = {
    3: ("attn_mfma_prefill_config3_traffic.md", ("attn_mfma.hip", "common.hpp", "kernels.hpp")),
    4: ("attn_mfma_prefill_config4_traffic.md", ("attn_mfma.hip", "common.hpp", "kernels.hpp")),
}
DECODE_TRAFFIC = ("decode_config5_traffic.md", ("decode.hip", "common.hpp", "kernels.hpp"))


def measured_traffic(spec):
    """HBM bytes per launch from a committed FETCH_SIZE / WRITE_SIZE counter
    summary, or None once the kernel sources differ from the ones the
    counters were taken on (or no summary exists)."""
    import hashlib

    name, sources = spec
    try:
        text = open(os.path.join(PROFILES, name)).read()
    except OSError:
        return None
    fields = dict(l.split(": ", 1) for l in text.splitlines()
                  if l.startswith(("traffic_bytes_per_launch: ", "kernel_sources_sha256: ")))
    if "traffic_bytes_per_launch" not in fields:
        return None
    h = hashlib.sha256()
    for f in sources:
        with open(os.path.join(ROOT, "paper_2608_19662_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    if fields.get("kernel_sources_sha256", "").strip() != h.hexdigest():
        return None
    return float(fields["traffic_bytes_per_launch"])


def prefix_encode_row(dev, reps, P=512):
    """Config 2's resources encoded after a shared P-token prefix (resource
    positions start at P): the attention kernel alone, prefix cache resident."""
    import torch
    from paper_2608_19662_amd import recache as rc
    from paper_2608_19662_amd.workloads import config, normal

    w = config(2)["encode"]
    T, Hq, Hkv, d = w.total, w.n_q_heads, w.n_kv_heads, w.head_dim
    q, k, v = w.tensors(dev)
    cu = i32(w.cu_len, dev)
    pb = i32(np.full(len(w.lengths), P), dev)
    kc = torch.empty(Hkv, T, d, dtype=q.dtype, device=dev)
    vc = torch.empty_like(kc)
    rc.rope_kv(k, v, i32(np.concatenate([P + np.arange(n) for n in w.lengths]), dev), w.rope_base,
               kc, vc)
    pk = normal((Hkv, P, d), q.dtype, 2, 40, dev)
    pv = normal((Hkv, P, d), q.dtype, 2, 41, dev)
    out = torch.empty_like(q)
    L = w.lengths.astype(np.int64)
    flops = 4.0 * d * Hq * float(np.sum(L * (L + 1) // 2 + P * L))
    ms = timed(lambda: rc.encode_attention(q, kc, vc, cu, int(L.max()), w.rope_base, out,
                                           pos_base=pb, prefix_k=pk, prefix_v=pv), reps)
    return {"workload": "config 2 after a shared %d-token prefix" % P, "ms": ms,
            "tflops": flops / (ms * 1e-3) / 1e12, "flops": flops,
            "pct_of_peak": 100.0 * flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}


def dense_prefill_row(dev, reps):
    """Dense baseline of config 4's requests: each request's whole prompt
    [its 8 resources, unpruned, then its 2048 context tokens] as one causal
    sequence at global positions, 36 layers (one layer's tensors reused).
    The attention of such a request is causal attention over the sequence, so
    it runs on the encode kernel with one unit per request."""
    import torch
    from paper_2608_19662_amd import recache as rc
    from paper_2608_19662_amd.workloads import config, normal, prefix

    w = config(4)["attend"]
    L, Hq, Hkv, d = w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim
    lens = np.array([int(w.lengths[w.req_res[w.req_res_off[b]:w.req_res_off[b + 1]]].sum())
                     + int(w.ctx_lens[b]) for b in range(w.n_req)], np.int32)
    N = int(lens.sum())
    q = normal((N, Hq, d), torch.bfloat16, 4, 60, dev)
    k = normal((N, Hkv, d), torch.bfloat16, 4, 61, dev)
    v = normal((N, Hkv, d), torch.bfloat16, 4, 62, dev)
    kc = torch.empty(Hkv, N, d, dtype=q.dtype, device=dev)
    vc = torch.empty_like(kc)
    cu = i32(prefix(lens), dev)
    rc.rope_kv(k, v, i32(np.concatenate([np.arange(n) for n in lens]), dev), 1e6, kc, vc)
    out = torch.empty_like(q)
    n = lens.astype(np.int64)
    flops = 4.0 * d * Hq * float(np.sum(n * (n + 1) // 2)) * L

    def run():
        for _ in range(L):
            rc.encode_attention(q, kc, vc, cu, int(lens.max()), 1e6, out)

    ms = timed(run, reps)
    del q, k, v, kc, vc, out
    torch.cuda.empty_cache()
    return {"workload": "config 4 requests as dense causal prompts (%d tokens), 36 layers" % N,
            "ms_per_pass": ms, "tflops": flops / (ms * 1e-3) / 1e12, "flops": flops,
            "pct_of_peak": 100.0 * flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}


def dense_decode_row(dev, reps):
    """Dense baseline of config 5's decode: every resource row visible in every
    (layer, group), nothing pruned, plus the 4096 context rows; 36 layers over
    one layer's tensors (10 GB of K/V per layer)."""
    import torch
    from paper_2608_19662_amd import recache as rc
    from paper_2608_19662_amd.workloads import config, normal

    w = config(5)["attend"]
    L, G, Hq, d = w.n_layers, w.n_kv_heads, w.n_q_heads, w.head_dim
    R = int(w.cu_len[-1])
    Tc = int(w.cu_ctx[-1])
    q = normal((w.n_req, Hq, d), torch.bfloat16, 5, 70, dev)
    ck = normal((G, Tc, d), torch.bfloat16, 5, 71, dev)
    cv = normal((G, Tc, d), torch.bfloat16, 5, 72, dev)
    rk = normal((G, R, d), torch.bfloat16, 5, 73, dev)
    rv = normal((G, R, d), torch.bfloat16, 5, 74, dev)
    E = w.n_req * L * G
    cu_rows = i32(w.cu_len, dev)
    route_off = torch.empty(E + 1, dtype=torch.int32, device=dev)
    route_res = torch.empty(int(w.req_res_off[-1]) * L * G, dtype=torch.int32, device=dev)
    route_tokens = torch.empty(E, dtype=torch.int32, device=dev)
    mask = torch.ones(w.n_res, L, G, dtype=torch.uint8, device=dev)
    rc.build_routes(i32(w.req_res_off, dev), i32(w.req_res, dev), mask, cu_rows, route_off,
                    route_res, route_tokens)
    cu_q, cu_ctx = i32(w.cu_q, dev), i32(w.cu_ctx, dev)
    plan = None
    if USE_PLAN:
        plan = torch.empty(L, w.n_req * G, dtype=torch.int32, device=dev)
        rc.attend_plan(cu_q, cu_ctx, route_tokens, L, Hq, G, plan)
    per_req = np.array([int(w.lengths[w.req_res[w.req_res_off[b]:w.req_res_off[b + 1]]].sum())
                        for b in range(w.n_req)], np.int64)
    keys = per_req + w.ctx_lens.astype(np.int64)
    max_kv = int(keys.max())
    nb = rc.attend_workspace_bytes(w.n_req, 1, int(w.ctx_lens.max()), max_kv, Hq, G, d)
    ws = torch.empty(nb // 4, dtype=torch.float32, device=dev)
    out = torch.empty_like(q)
    max_route = int(np.diff(w.req_res_off).max())

    def run():
        for l in range(L):
            rc.attend_cached(q, ck, cv, cu_q, cu_ctx, 1, int(w.ctx_lens.max()), rk, rv, cu_rows,
                             route_off, route_res, route_tokens, l, L, out, workspace=ws,
                             max_kv=max_kv, max_route_len=max_route, plan=plan)

    ms = timed(run, reps)
    nbytes = (float(keys.sum()) * G * 4 * d + 2.0 * w.n_req * Hq * d * 2) * L
    del q, ck, cv, rk, rv, ws
    torch.cuda.empty_cache()
    return {"workload": "config 5 dense: all %d resource rows visible, unpruned" % R,
            "ms_per_step": ms, "gbs": nbytes / (ms * 1e-3) / 1e9, "bytes": nbytes,
            "pct_of_peak": 100.0 * nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS}


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(dev, n_req=8):
    """The fp64 oracle on a bounded sample of the headline workload: every
    query row and head of the first n_req requests of layer 0 (by default
    all 8, one whole layer: about 35 s on 16 host threads), timed once.  The
    36-layer step is extrapolated from the sample's share of the step's pairs
    (the layers of this workload have identical structure)."""
    import oracle
    from paper_2608_19662_amd.workloads import config

    w = config(3)["attend"]
    r = w.n_q_heads // w.n_kv_heads
    pairs = prefill_pairs(w)
    flops_sample = 4.0 * w.head_dim * r * float(pairs[:n_req, 0, :].sum())
    flops_step = 4.0 * w.head_dim * r * float(pairs.sum())
    q, ck, cv, rk, rv = (t.cpu() for t in w.layer_tensors(0, dev))
    rb = np.concatenate([np.full(int(w.q_lens[b]), b, np.int32) for b in range(n_req)])
    ri = np.concatenate([np.arange(int(w.q_lens[b]), dtype=np.int32) for b in range(n_req)])
    t0 = time.perf_counter()
    oracle.attend(q, ck, cv, w.cu_q, w.cu_ctx, rk, rv, w.cu_rows, w.req_res_off, w.req_res,
                  w.mask, 0, rows=(rb, ri))
    dt = time.perf_counter() - t0
    return {"value": flops_sample / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.threads(),
            "kind": "oracle", "seconds": dt, "nproc": os.cpu_count(), "cpu_model": cpu_model(),
            "extrapolated_ms_per_step": dt * 1e3 * flops_step / flops_sample,
            "sample": "layer 0 of the config 3 step, requests 0-%d (every query row and head over "
                      "their resources and context, fp64; %.1f%% of the step's FLOPs), timed "
                      "once; the step time is extrapolated by the FLOP ratio"
                      % (n_req - 1, 100.0 * flops_sample / flops_step)}


def headline(args, dev):
    """Config 3's 36-layer prefill pass: W untimed warm-up passes after an
    untimed pre-warm (the GPU raises its clocks only after some time under
    load), then K passes timed with HIP events on the launch stream around
    the whole region.  Each pass is 36 launches of the attention kernel and
    nothing else, so the region's time over 36 K is that kernel's average
    launch duration."""
    import torch

    w, flops, nbytes, layers, outs, run = prefill_setup(3, dev)
    L = w.n_layers
    s = torch.cuda.current_stream()
    t_end = time.perf_counter() + args.prewarm
    while time.perf_counter() < t_end:
        run()
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(s)
    for _ in range(args.steps):
        run()
    b.record(s)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / args.steps
    tokens = int(w.cu_q[-1])
    res = {"w": w, "flops": flops, "ms_per_step": ms, "tflops": flops / (ms * 1e-3) / 1e12,
           "tokens": tokens, "resource_rows": int(w.cu_len[-1]),
           "roofline": roofline("attn_mfma_kernel<128, attend>", "mfma", flops / L, ms / L,
                                traffic=measured_traffic(PREFILL_TRAFFIC[3]),
                                launches=args.steps * L, algorithmic_bytes=nbytes)}
    del layers, outs
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--rows", default="all",
                    help="extra hot-path rows: all | none | comma list of row names")
    ap.add_argument("--reps", type=int, default=5, help="repetitions per extra row")
    ap.add_argument("--prewarm", type=float, default=PREWARM_S,
                    help="seconds of untimed load before the headline's warm-up (clock ramp)")
    ap.add_argument("--skip-headline", action="store_true",
                    help="run only the rows (for counter collection on one row)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-plan", action="store_true",
                    help="attend without the per-batch work order (grid in request order)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain elementwise copy (int32 negation, reads and writes "
                         "MIB MiB) 5 times: the reference kernel for scaling HBM byte counters")
    args = ap.parse_args()
    global USE_PLAN
    USE_PLAN = not args.no_plan
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(sharding is design-only); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n // 4, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            torch.neg(src, out=dst)  # an elementwise kernel, not a DMA copy
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 5}), flush=True)
        return
    h = None
    if not args.skip_headline:
        log("headline: config 3 prefill, 36 layers, %d warmup + %d steps" % (args.warmup, args.steps))
        h = headline(args, dev)
        log("headline done: %.3f ms/step, %.1f TFLOP/s (kernel %.4f ms per launch)" % (
            h["ms_per_step"], h["tflops"], h["roofline"]["avg_kernel_ms"]))
    rows = {}
    if args.rows != "none":
        want = None if args.rows == "all" else set(args.rows.split(","))
        pick = lambda name: want is None or name in want
        for name, fn in (("a1_a3_encode_config2", lambda: encode_row(dev, 50, 5)),
                         ("a4_prune_gather", lambda: prune_row(dev, args.reps)),
                         ("f1_encode_prefix_config2", lambda: prefix_encode_row(dev, args.reps)),
                         ("a6_prefill_config4", lambda: prefill_row(4, dev, args.reps))):
            if pick(name):
                log("row", name)
                rows[name] = fn()
                log("  ", json.dumps(rows[name]))
        if pick("a7_decode_config5") or pick("a5_route_build"):
            log("row a7_decode_config5 + a5_route_build")
            rows["a7_decode_config5"], rows["a5_route_build"] = decode_row(dev, args.reps)
            log("  ", json.dumps(rows["a7_decode_config5"]))
        if pick("f3_route_store_config5"):
            log("row f3_route_store_config5")
            rows["f3_route_store_config5"] = route_store_row(dev, args.reps)
            log("  ", json.dumps(rows["f3_route_store_config5"]))
        for name, fn in (("f2_dense_prefill_config4", lambda: dense_prefill_row(dev, args.reps)),
                         ("f2_dense_decode_config5", lambda: dense_decode_row(dev, args.reps))):
            if pick(name):
                log("row", name)
                rows[name] = fn()
                log("  ", json.dumps(rows[name]))
        # attention-time ratios Dense / ReCache on the same synthetic inputs
        if "f2_dense_prefill_config4" in rows and "a6_prefill_config4" in rows:
            rows["f2_dense_over_recache_prefill"] = round(
                rows["f2_dense_prefill_config4"]["ms_per_pass"]
                / rows["a6_prefill_config4"]["ms_per_pass"], 3)
        if "f2_dense_decode_config5" in rows and "a7_decode_config5" in rows:
            rows["f2_dense_over_recache_decode"] = round(
                rows["f2_dense_decode_config5"]["ms_per_step"]
                / rows["a7_decode_config5"]["ms_per_step"], 3)
    if h is None:
        print(json.dumps({"rows": rows}), flush=True)
        return
    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle, one config 3 layer)")
        cpu = cpu_baseline(dev)
        log("  ", json.dumps(cpu))
    w = h["w"]
    line = {
        "metric": METRIC,
        "value": round(h["tflops"], 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(h["ms_per_step"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "config 3: conversation prefill over cached resources, 36 layers, "
                        "8 requests x (8 resources U[300,1200] = %d resource rows in all, all "
                        "routes visible, no pruning; 2048 context tokens causal), 32 q / 8 KV "
                        "heads, head_dim 128, bf16" % h["resource_rows"],
            "query_tokens": h["tokens"],
            "flops_per_step": h["flops"],
            "step": "36 recache_attend_cached calls (one per layer), each one launch of the "
                    "MFMA attention kernel over routed resource rows then causal context",
            "prewarm_s": args.prewarm,
        },
        "pct_of_peak": round(100.0 * h["tflops"] / PEAK_BF16_TFLOPS, 2),
        "roofline": h["roofline"],
        "cpu_baseline": cpu,
        "rows": rows,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
