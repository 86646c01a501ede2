"""Helpers for the GPU parity tests: device copies of workload structure,
the route build, and the tolerance rules.

Tolerances (stated once, used by every GPU test):
  fp32 inputs:  |gpu - oracle| <= 1e-5 everywhere.
  bf16 inputs:  |gpu - oracle| <= 1e-2 + 2^-8 |oracle| everywhere: the 1e-2
                bound for fp32 accumulation over bf16 inputs, widened by the
                half-ulp of rounding the output to bf16 (at most 2^-8 of the
                value: bf16 keeps 8 significant bits).  The oracle holds
                rotated queries and keys at bf16, as the kernels and a bf16
                backbone do; rotated values written in bf16 (the K cache,
                rotated queries) must then match the oracle's to one bf16 ulp
                plus the absolute error of the fp32 rotation before rounding:
                <= 2^-7 |oracle| + 1e-5 (the absolute term matters where the
                two products of a rotation cancel).
  LSE (fp32 outputs of bf16 calls): |gpu - oracle| <= 1e-2 absolute.  The
                LSE is never rounded to bf16; what moves it is the row sum of
                the bf16-rounded weights the kernels normalise by (each weight
                within 2^-9 relative, so ln of the sum within about 2^-9) and
                fp32 arithmetic (|lse| ~ 10 gives ~1e-6), far inside 1e-2.
                fp32 calls keep the 1e-5 bar for the LSE too.
  index work:   bit-exact.
"""
from __future__ import annotations

import numpy as np
import torch

from paper_2608_19662_amd import recache as rc

DEV = "cuda"


def i32(a):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.int32))).to(DEV)


def f64(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def lse_rule(dtype: str) -> str:
    """Tolerance rule of an LSE output for a call in dtype ("f32" or "bf16")."""
    return "f32" if dtype == "f32" else "lse"


def check(gpu, ref, dtype: str, name: str):
    """Assert the tolerance rule; returns the max abs error."""
    g = f64(gpu)
    ref = np.asarray(ref, np.float64)
    assert g.shape == ref.shape, (name, g.shape, ref.shape)
    err = np.abs(g - ref)
    if dtype == "f32":
        bound = np.full_like(ref, 1e-5)
    elif dtype == "lse":
        bound = np.full_like(ref, 1e-2)
    elif dtype == "bf16-ulp":
        bound = 2.0 ** -7 * np.abs(ref) + 1e-5
    else:
        bound = 1e-2 + 2.0 ** -8 * np.abs(ref)
    bad = ~(err <= bound)
    if bad.any():
        ratio = np.where(np.isnan(err), np.inf, err / bound)
        worst = np.unravel_index(int(np.argmax(ratio)), ratio.shape)
        raise AssertionError("%s: %d of %d out of tolerance; worst at %s: gpu %r, oracle %r, bound %.3g"
                             " (max abs err %.3g)" % (name, int(bad.sum()), bad.size, list(worst),
                                                      g[worst], ref[worst], bound[worst],
                                                      float(np.nanmax(err))))
    return float(err.max()) if err.size else 0.0


class Routes:
    """Device structure of an AttendWorkload plus its route CSR (GPU-built)."""

    def __init__(self, w, stream=None):
        self.w = w
        self.cu_q = i32(w.cu_q)
        self.cu_ctx = i32(w.cu_ctx)
        self.cu_rows = i32(w.cu_rows)
        self.req_res_off = i32(w.req_res_off)
        self.req_res = i32(w.req_res if len(w.req_res) else [0])
        self.mask = torch.from_numpy(np.ascontiguousarray(w.mask.astype(np.uint8))).to(DEV)
        E = w.n_req * w.n_layers * w.n_kv_heads
        self.route_off = torch.empty(E + 1, dtype=torch.int32, device=DEV)
        cap = max(1, int(w.req_res_off[-1]) * w.n_layers * w.n_kv_heads)
        self.route_res = torch.empty(cap, dtype=torch.int32, device=DEV)
        self.route_tokens = torch.empty(E, dtype=torch.int32, device=DEV)
        if len(w.req_res) == 0:
            # no resource anywhere: every route list is empty
            self.route_off.zero_()
            self.route_tokens.zero_()
        else:
            rc.build_routes(self.req_res_off, self.req_res, self.mask, self.cu_rows, self.route_off,
                            self.route_res, self.route_tokens, stream=stream)
        per_req = np.diff(w.req_res_off)
        self.max_route_len = int(per_req.max()) if len(per_req) else 0
        self.max_q = int(np.max(w.q_lens))
        self.max_ctx = int(np.max(w.ctx_lens))

    def max_kv(self, layer=None):
        tok = self.route_tokens.cpu().numpy().reshape(self.w.n_req, self.w.n_layers, -1)
        if layer is not None:
            tok = tok[:, layer]
        return int((tok.reshape(self.w.n_req, -1).max(1) + self.w.ctx_lens).max())

    def workspace(self, max_kv):
        w = self.w
        n = rc.attend_workspace_bytes(w.n_req, self.max_q, self.max_ctx, max_kv, w.n_q_heads,
                                      w.n_kv_heads, w.head_dim)
        return torch.empty(max(n, 4) // 4, dtype=torch.float32, device=DEV) if n else None

    def plan(self, stream=None):
        """GPU-built work order of every layer, [L][n_req * Hkv]."""
        w = self.w
        p = torch.empty(w.n_layers, w.n_req * w.n_kv_heads, dtype=torch.int32, device=DEV)
        rc.attend_plan(self.cu_q, self.cu_ctx, self.route_tokens, w.n_layers, w.n_q_heads,
                       w.n_kv_heads, p, stream=stream)
        return p

    def attend(self, q, ck, cv, rk, rv, layer, lse=True, workspace=None, max_kv=0, stream=None,
               res_off=None, plan=None):
        w = self.w
        out = torch.empty_like(q)
        l = torch.empty(w.n_q_heads, q.shape[0], dtype=torch.float32, device=DEV) if lse else None
        rc.attend_cached(q, ck, cv, self.cu_q, self.cu_ctx, self.max_q, self.max_ctx, rk, rv,
                         self.cu_rows, self.route_off, self.route_res, self.route_tokens, layer,
                         w.n_layers, out, lse=l, workspace=workspace, max_kv=max_kv,
                         max_route_len=max(self.max_route_len, 1), stream=stream,
                         res_off=res_off, plan=plan)
        return out, l


    def store_offsets(self):
        """GPU-built row tables of the route-compacted store, [L][n_res * G + 1]."""
        w = self.w
        off = torch.empty(w.n_layers, len(w.lengths) * w.n_kv_heads + 1, dtype=torch.int32,
                          device=DEV)
        rc.route_store_offsets(self.mask, self.cu_rows, off, total_kept=int(w.cu_rows[-1]))
        return off


def plan_reference(cu_q, cu_ctx, route_tokens, n_layers, n_q_heads, n_kv_heads):
    """The work order the plan builder documents, in plain Python: per layer
    the pairs b * G + g sorted by (work descending, pair ascending), the
    k-th sorted pair at grid row k // G, position k % G (even rows) or
    G - 1 - k % G (odd rows).  Work: for every prefill query tile of wg
    rows, its 64-key tiles (keys up to its last row) plus 3."""
    G = n_kv_heads
    ratio = n_q_heads // G
    h = 8
    while ratio % h:
        h //= 2
    wg = 32 * (8 // h)
    cu_q = np.asarray(cu_q, np.int64)
    cu_ctx = np.asarray(cu_ctx, np.int64)
    n_req = len(cu_q) - 1
    tok = np.asarray(route_tokens, np.int64).reshape(n_req, n_layers, G)
    out = np.zeros((n_layers, n_req * G), np.int32)
    for l in range(n_layers):
        work = []
        for b in range(n_req):
            tq = int(cu_q[b + 1] - cu_q[b])
            tc = int(cu_ctx[b + 1] - cu_ctx[b])
            for g in range(G):
                off = int(tok[b, l, g]) + tc - tq
                wk = 0
                for r0 in range(0, max(tq, 0), wg):
                    wk += max(off + min(r0 + wg, tq) - 1, 0) // 64 + 1 + 3
                work.append(min(wk, 2 ** 31 - 1))
        order = sorted(range(n_req * G), key=lambda i: (-work[i], i))
        for k, pair in enumerate(order):
            row, c = divmod(k, G)
            out[l, row * G + (G - 1 - c if row % 2 else c)] = pair
    return out
