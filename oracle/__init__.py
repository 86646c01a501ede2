"""fp64 CPU oracle for ReCache resource-wise attention (ctypes wrapper).

TEST INFRASTRUCTURE ONLY.  The test suite, the smoke check and the CPU
baseline of the benchmark are the only users.  Nothing in the product package
imports this module, and this module imports nothing from the product package.

The arithmetic lives in ``recache_oracle.c`` (plain C, fp64, OpenMP), which
follows the paper's definitions (ReCache, Sec. 3 and Fig. 2); each function
there names the passage it follows.  This wrapper only marshals numpy arrays.

Inputs are numpy arrays of float32 or float64, or of uint16 holding bfloat16
bit patterns (use :func:`host_view` to get one from a torch tensor).  The oracle
widens every element exactly to double at the point of use.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "recache_oracle.c")
_LIB = os.path.join(_HERE, "librecache_oracle.so")
_lib = None

F32, BF16, F64 = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, no fast-math, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
             "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        _lib = ctypes.CDLL(_LIB)
    return _lib


def threads() -> int:
    """OpenMP threads the oracle runs on."""
    return int(_load().oracle_threads())


def host_view(t):
    """numpy view of a CPU tensor/array: float32 stays float32, bf16 -> uint16 bits."""
    if isinstance(t, np.ndarray):
        if t.dtype not in (np.float32, np.uint16, np.float64):
            raise TypeError("oracle inputs are float32, float64 or uint16 (bf16 bits), got %s"
                            % t.dtype)
        return np.ascontiguousarray(t)
    import torch  # only for dtype inspection of a CPU tensor

    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype in (torch.float32, torch.float64):
        return t.numpy()
    raise TypeError("oracle inputs are float32, float64 or bfloat16, got %s" % t.dtype)


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    if a.dtype == np.float64:
        return F64
    raise TypeError(a.dtype)


def _i32(a):
    return None if a is None else np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc, what):
    if rc != 0:
        raise ValueError("oracle_%s rejected its arguments" % what)


def _rot(x, rot_dtype):
    return _dtype_code(x) if rot_dtype is None else int(rot_dtype)


def round_to(x, dtype: int) -> np.ndarray:
    """Round float64 values to nearest-even at the precision of dtype (F32/BF16/F64)."""
    x = np.ascontiguousarray(np.asarray(x, np.float64))
    f = _load().oracle_round
    f.restype = ctypes.c_double
    f.argtypes = [ctypes.c_double, ctypes.c_int]
    return np.array([f(float(v), int(dtype)) for v in x.ravel()]).reshape(x.shape)


def rope(x, pos, base: float, rot_dtype=None) -> np.ndarray:
    """RoPE of x[T][H][d] at positions pos[T]; returns float64 [T][H][d] whose
    values are rounded to the precision of rot_dtype (default: x's dtype)."""
    x = host_view(x)
    pos = _i32(pos)
    T, H, d = x.shape
    y = np.empty((T, H, d), np.float64)
    lib = _load()
    lib.oracle_rope.restype = ctypes.c_int
    rc = lib.oracle_rope(ctypes.c_int(_dtype_code(x)), ctypes.c_int(T), ctypes.c_int(H),
                         ctypes.c_int(d), ctypes.c_double(base), _p(pos), _p(x), _p(y),
                         ctypes.c_int(_rot(x, rot_dtype)))
    _check(rc, "rope")
    return y


def encode(q, k, v, cu_len, base: float, scale: float | None = None, pos_base=None,
           rot_dtype=None, prefix_k=None, prefix_v=None):
    """Block-diagonal causal encode of packed resources (one layer).

    q[T][Hq][d], k/v[T][Hkv][d] in stored precision.  Rotated queries and keys
    are rounded to the precision of rot_dtype (default: the inputs' dtype).
    An optional shared prefix is given as its rotated cache prefix_k/prefix_v
    [Hkv][P][d] in the inputs' dtype; every resource row attends all of it.
    Returns a dict of float64 arrays: out[T][Hq][d], k_cache/v_cache[Hkv][T][d],
    lse[Hq][T].
    """
    q, k, v = host_view(q), host_view(k), host_view(v)
    if (prefix_k is None) != (prefix_v is None):
        raise ValueError("prefix_k and prefix_v go together")
    p_len = 0
    if prefix_k is not None:
        prefix_k, prefix_v = host_view(prefix_k), host_view(prefix_v)
        if prefix_k.dtype != q.dtype or prefix_v.dtype != q.dtype:
            raise ValueError("the prefix cache has the inputs' dtype")
        p_len = prefix_k.shape[1]
    cu_len = _i32(cu_len)
    pos_base = _i32(pos_base)
    T, Hq, d = q.shape
    Hkv = k.shape[1]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.empty((T, Hq, d), np.float64)
    kc = np.empty((Hkv, T, d), np.float64)
    vc = np.empty((Hkv, T, d), np.float64)
    lse = np.empty((Hq, T), np.float64)
    lib = _load()
    rc = lib.oracle_encode(
        ctypes.c_int(_dtype_code(q)), ctypes.c_int(len(cu_len) - 1), _p(cu_len),
        ctypes.c_int(Hq), ctypes.c_int(Hkv), ctypes.c_int(d), ctypes.c_double(base),
        _p(pos_base), ctypes.c_double(scale), _p(q), _p(k), _p(v),
        ctypes.c_int(p_len), _p(prefix_k), _p(prefix_v),
        _p(out), _p(kc), _p(vc), _p(lse), ctypes.c_int(_rot(q, rot_dtype)))
    _check(rc, "encode")
    return {"out": out, "k_cache": kc, "v_cache": vc, "lse": lse}


def check_kept(cu_len, cu_kept, kept_idx) -> bool:
    cu_len, cu_kept, kept_idx = _i32(cu_len), _i32(cu_kept), _i32(kept_idx)
    return _load().oracle_check_kept(ctypes.c_int(len(cu_len) - 1), _p(cu_len), _p(cu_kept),
                                     _p(kept_idx)) == 0


def prune(k_cache, v_cache, cu_len, cu_kept, kept_idx):
    """Gather kept rows of head-major caches [Hkv][T][d]; byte-exact copies."""
    k_cache, v_cache = host_view(k_cache), host_view(v_cache)
    cu_len, cu_kept, kept_idx = _i32(cu_len), _i32(cu_kept), _i32(kept_idx)
    Hkv, T, d = k_cache.shape
    K = int(cu_kept[-1])
    kk = np.empty((Hkv, K, d), k_cache.dtype)
    vk = np.empty((Hkv, K, d), v_cache.dtype)
    rc = _load().oracle_prune(ctypes.c_int(_dtype_code(k_cache)), ctypes.c_int(len(cu_len) - 1),
                              _p(cu_len), _p(cu_kept), _p(kept_idx), ctypes.c_int(Hkv),
                              ctypes.c_int(d), _p(k_cache), _p(v_cache), _p(kk), _p(vk))
    _check(rc, "prune")
    return kk, vk


def routes(req_res_off, req_res, mask, cu_kept):
    """Route CSR for every (request, layer, group): (route_off, route_res, route_tokens)."""
    req_res_off, req_res, cu_kept = _i32(req_res_off), _i32(req_res), _i32(cu_kept)
    mask = np.ascontiguousarray(np.asarray(mask, dtype=np.uint8))
    n_res, L, G = mask.shape
    n_req = len(req_res_off) - 1
    E = n_req * L * G
    off = np.zeros(E + 1, np.int32)
    res = np.zeros(max(1, int(req_res_off[-1]) * L * G), np.int32)
    tok = np.zeros(E, np.int32)
    rc = _load().oracle_routes(ctypes.c_int(n_req), _p(req_res_off), _p(req_res),
                               ctypes.c_int(n_res), ctypes.c_int(L), ctypes.c_int(G), _p(mask),
                               _p(cu_kept), _p(off), _p(res), _p(tok))
    _check(rc, "routes")
    return off, res[: off[-1]].copy(), tok


def attend(q, ctx_k, ctx_v, cu_q, cu_ctx, res_k, res_v, cu_rows, req_res_off, req_res, mask,
           layer: int, scale: float | None = None, cu_kept=None, kept_idx=None, rows=None,
           store_off=None):
    """Conversation queries over routed resources plus causal context, one layer.

    q[sum Tq][Hq][d] (rotated); ctx_k/ctx_v[Hkv][sum Tc][d]; res_k/res_v
    [Hkv][R][d] with resource r owning rows [cu_rows[r], cu_rows[r+1]);
    mask[n_res][L][G] uint8.  With kept_idx the visible rows of resource r are
    cu_rows[r] + kept_idx[cu_kept[r]:cu_kept[r+1]].  rows = (b_array, i_array)
    picks which queries to evaluate (default: all).  With store_off (this
    layer's row of :func:`store_offsets`), res_k/res_v are a route-compacted
    store [rows][d] and resource r's rows for group g start at
    store_off[r * G + g].  Returns (out[n][Hq][d], lse[n][Hq]) in float64.
    """
    q, ctx_k, ctx_v = host_view(q), host_view(ctx_k), host_view(ctx_v)
    res_k, res_v = host_view(res_k), host_view(res_v)
    cu_q, cu_ctx, cu_rows = _i32(cu_q), _i32(cu_ctx), _i32(cu_rows)
    req_res_off, req_res = _i32(req_res_off), _i32(req_res)
    cu_kept, kept_idx, store_off = _i32(cu_kept), _i32(kept_idx), _i32(store_off)
    mask = np.ascontiguousarray(np.asarray(mask, dtype=np.uint8))
    n_res, L, G = mask.shape
    _, Hq, d = q.shape
    res_stride = res_k.shape[1] if res_k.ndim == 3 else 0
    Hkv = ctx_k.shape[0]
    if G != Hkv:
        raise ValueError("mask groups %d != KV heads %d" % (G, Hkv))
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    n_req = len(cu_q) - 1
    if rows is None:
        rb = np.concatenate([np.full(cu_q[b + 1] - cu_q[b], b, np.int32) for b in range(n_req)])
        ri = np.concatenate([np.arange(cu_q[b + 1] - cu_q[b], dtype=np.int32) for b in range(n_req)])
    else:
        rb, ri = _i32(rows[0]), _i32(rows[1])
    n = len(rb)
    out = np.empty((n, Hq, d), np.float64)
    lse = np.empty((n, Hq), np.float64)
    rc = _load().oracle_attend(
        ctypes.c_int(_dtype_code(q)), ctypes.c_int(n_req), _p(cu_q), _p(cu_ctx),
        ctypes.c_int(Hq), ctypes.c_int(Hkv), ctypes.c_int(d), ctypes.c_double(scale),
        _p(q), _p(ctx_k), _p(ctx_v), ctypes.c_long(ctx_k.shape[1]),
        ctypes.c_int(n_res), _p(cu_rows), ctypes.c_long(res_stride), _p(res_k), _p(res_v),
        _p(cu_kept), _p(kept_idx), _p(req_res_off), _p(req_res),
        ctypes.c_int(L), ctypes.c_int(layer), _p(mask), _p(store_off),
        ctypes.c_int(n), _p(rb), _p(ri), _p(out), _p(lse))
    _check(rc, "attend")
    return out, lse


def store_offsets(mask, cu_kept):
    """Row tables of the route-compacted store: [L][n_res * G + 1] int32.

    Entry [l][r * G + g] is where route (r, g) of layer l starts, the last
    entry of a row the rows stored for that layer."""
    mask = np.ascontiguousarray(np.asarray(mask, dtype=np.uint8))
    cu_kept = _i32(cu_kept)
    n_res, L, G = mask.shape
    off = np.zeros((L, n_res * G + 1), np.int32)
    rc = _load().oracle_store_offsets(ctypes.c_int(n_res), ctypes.c_int(L), ctypes.c_int(G),
                                      _p(mask), _p(cu_kept), _p(off))
    _check(rc, "store_offsets")
    return off


def store_routes(k_cache, v_cache, cu_len, cu_kept, kept_idx, mask, layer: int):
    """One layer of the route-compacted store, gathered from head-major caches
    [Hkv][T][d]: (k_store[rows][d], v_store[rows][d]), byte-exact copies."""
    k_cache, v_cache = host_view(k_cache), host_view(v_cache)
    cu_len, cu_kept, kept_idx = _i32(cu_len), _i32(cu_kept), _i32(kept_idx)
    mask = np.ascontiguousarray(np.asarray(mask, dtype=np.uint8))
    n_res, L, G = mask.shape
    Hkv, _, d = k_cache.shape
    if G != Hkv:
        raise ValueError("mask groups %d != KV heads %d" % (G, Hkv))
    kept = np.diff(cu_kept).astype(np.int64)
    cap = max(1, int((mask[:, layer, :].sum(axis=1) * kept).sum()))
    ks = np.empty((cap, d), k_cache.dtype)
    vs = np.empty((cap, d), v_cache.dtype)
    fn = _load().oracle_store_routes
    fn.restype = ctypes.c_long
    n = fn(ctypes.c_int(_dtype_code(k_cache)), ctypes.c_int(n_res), _p(cu_len), _p(cu_kept),
           _p(kept_idx), ctypes.c_int(Hkv), ctypes.c_int(d), ctypes.c_int(L), ctypes.c_int(layer),
           _p(mask), _p(k_cache), _p(v_cache), _p(ks), _p(vs), ctypes.c_long(cap))
    _check(-1 if n < 0 else 0, "store_routes")
    return ks[:n].copy(), vs[:n].copy()
