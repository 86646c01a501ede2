"""Thin Python binding of librecache.so (the C ABI in include/recache.h).

Argument marshalling only: every function takes torch CUDA tensors, checks
that they are contiguous device tensors of the expected dtype (passing a host
pointer to a kernel would fault the GPU), reads sizes from their shapes and
calls the C entry point of the same name on the current HIP stream.  All
arithmetic happens in the library's HIP kernels; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librecache.so")

OK, EINVAL, EUNSUPPORTED, EWORKSPACE, EHIP = 0, -1, -2, -3, -4
F32, BF16 = 0, 1

_lib = None

_c_int, _c_dbl, _c_flt, _c_p, _c_size = (ctypes.c_int, ctypes.c_double, ctypes.c_float,
                                         ctypes.c_void_p, ctypes.c_size_t)

_SIGS = {
    "recache_version": ([], _c_int),
    "recache_last_error": ([], ctypes.c_char_p),
    "recache_rope_q": ([_c_int, _c_int, _c_int, _c_int, _c_dbl, _c_p, _c_p, _c_p], _c_int),
    "recache_rope_kv": ([_c_int, _c_int, _c_int, _c_int, _c_dbl, _c_p, _c_p, _c_p, _c_p, _c_p,
                         _c_int, _c_int, _c_p], _c_int),
    "recache_encode_resources": ([_c_int, _c_int, _c_p, _c_int, _c_int, _c_int, _c_int, _c_int,
                                  _c_dbl, _c_p, _c_int, _c_p, _c_p, _c_flt, _c_p, _c_p, _c_p,
                                  _c_p, _c_p, _c_p, _c_p, _c_p], _c_int),
    "recache_encode_attention": ([_c_int, _c_int, _c_p, _c_int, _c_int, _c_int, _c_int, _c_int,
                                  _c_dbl, _c_p, _c_int, _c_p, _c_p, _c_flt, _c_p, _c_p, _c_p,
                                  _c_p, _c_p, _c_p], _c_int),
    "recache_prune_gather": ([_c_int, _c_int, _c_p, _c_p, _c_p, _c_int, _c_int, _c_int, _c_int,
                              _c_p, _c_p, _c_p, _c_p, _c_p], _c_int),
    "recache_build_routes": ([_c_int, _c_p, _c_p, _c_int, _c_int, _c_int, _c_int, _c_p, _c_p,
                              _c_p, _c_p, _c_p, _c_p], _c_int),
    "recache_attend_workspace_bytes": ([_c_int] * 7, _c_size),
    "recache_route_store_offsets": ([_c_int, _c_int, _c_int, _c_int, _c_p, _c_p, _c_p, _c_p],
                                    _c_int),
    "recache_store_routes": ([_c_int, _c_int, _c_int, _c_int, _c_p, _c_p, _c_p, _c_int, _c_int,
                              _c_int, _c_int, _c_p, _c_int, _c_p, _c_p, _c_p, _c_p, _c_p], _c_int),
    "recache_attend_cached": ([_c_int, _c_int, _c_int, _c_int, _c_p, _c_p, _c_int, _c_int, _c_int,
                               _c_int, _c_int, _c_int, _c_int, _c_int, _c_flt, _c_p, _c_p, _c_p,
                               _c_int, _c_p, _c_p, _c_int, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p,
                               _c_p, _c_p, _c_p, _c_size, _c_p], _c_int),
    "recache_attend_plan_bytes": ([_c_int, _c_int, _c_int], _c_size),
    "recache_attend_plan": ([_c_int, _c_int, _c_int, _c_int, _c_p, _c_p, _c_p, _c_p, _c_p],
                            _c_int),
    "recache_attend_cached_noalloc": ([_c_int, _c_int, _c_int, _c_int, _c_p, _c_p, _c_int, _c_int,
                                       _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_flt, _c_p,
                                       _c_p, _c_p, _c_int, _c_p, _c_p, _c_int, _c_p, _c_p, _c_p,
                                       _c_p, _c_p, _c_p, _c_p, _c_p, _c_p], _c_int),
    "recache_select_routes": ([_c_int, _c_int, _c_p, _c_p, _c_int, _c_int, _c_p, _c_p, _c_p, _c_p,
                               _c_p, _c_p], _c_int),
    "recache_check_offsets": ([_c_p, _c_int, _c_int, _c_int], _c_int),
    "recache_check_kept": ([_c_p, _c_p, _c_p, _c_int], _c_int),
    "recache_check_encode_lengths": ([_c_p, _c_int, _c_int, _c_int], _c_int),
    "recache_check_requests": ([_c_p, _c_p, _c_int, _c_int, _c_int, _c_int], _c_int),
}

EXPORTS = tuple(_SIGS)


class RecacheError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("%s (status %d)" % (msg, code))
        self.code = code


def lib() -> ctypes.CDLL:
    """Load librecache.so; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("librecache.so is not built; run `python -m paper_2608_19662_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def last_error() -> str:
    return lib().recache_last_error().decode()


def version() -> int:
    return lib().recache_version()


def _call(name, *args):
    rc = getattr(lib(), name)(*args)
    if rc != OK:
        raise RecacheError(rc, "%s: %s" % (name, last_error()))
    return rc


# ------------------------------------------------------------- marshalling

def _dev(t, name, dtypes=None):
    """Device pointer of a contiguous CUDA tensor (None -> NULL)."""
    if t is None:
        return None
    import torch

    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("%s must be a CUDA tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtypes is not None and t.dtype not in dtypes:
        raise TypeError("%s has dtype %s, expected one of %s" % (name, t.dtype, dtypes))
    return t.data_ptr()


def _dtype_code(t):
    import torch

    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError("floating tensors must be float32 or bfloat16, got %s" % t.dtype)


def _stream(stream):
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _i32():
    import torch

    return (torch.int32,)


def _same(ref, *ts):
    for t in ts:
        if t is not None and t.dtype != ref.dtype:
            raise TypeError("all floating tensors of a call share one dtype")


def _shape(t, name, *dims):
    """Raise unless tensor t (if given) has exactly the shape dims.  Checked
    before any pointer is taken: a buffer smaller than the sizes passed to the
    library would turn into a GPU access outside it."""
    if t is None:
        return
    if tuple(t.shape) != tuple(int(x) for x in dims):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(dims)))


def _numel(t, name, n):
    """Raise unless tensor t has exactly n elements (1-d index arrays)."""
    if t is not None and (t.dim() != 1 or t.numel() != int(n)):
        raise ValueError("%s must be 1-d with %d elements, has shape %s"
                         % (name, int(n), tuple(t.shape)))


def _at_least(t, name, n):
    """Raise unless 1-d tensor t holds at least n elements (capacities)."""
    if t is not None and (t.dim() != 1 or t.numel() < int(n)):
        raise ValueError("%s must be 1-d with at least %d elements, has shape %s"
                         % (name, int(n), tuple(t.shape)))


# ------------------------------------------------------------- entry points

def rope_q(x, pos, rope_base: float, stream=None):
    """In-place RoPE of x[T][H][d] at positions pos[T]."""
    T, H, d = x.shape
    _numel(pos, "pos", T)
    _call("recache_rope_q", _dtype_code(x), T, H, d, rope_base, _dev(pos, "pos", _i32()),
          _dev(x, "x"), _stream(stream))


def rope_kv(k, v, pos, rope_base: float, k_cache, v_cache, row0: int = 0, stream=None):
    """Rotated k and plain v into head-major caches [Hkv][rows][d] at row0."""
    T, Hkv, d = k.shape
    _same(k, v, k_cache, v_cache)
    _shape(v, "v", T, Hkv, d)
    _numel(pos, "pos", T)
    if k_cache.dim() != 3 or k_cache.shape[0] != Hkv or k_cache.shape[2] != d:
        raise ValueError("k_cache must be [%d][rows][%d], has shape %s" % (Hkv, d, tuple(k_cache.shape)))
    _shape(v_cache, "v_cache", *k_cache.shape)
    _call("recache_rope_kv", _dtype_code(k), T, Hkv, d, rope_base, _dev(pos, "pos", _i32()),
          _dev(k, "k"), _dev(v, "v"), _dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"),
          k_cache.shape[1], row0, _stream(stream))


def _prefix(prefix_k, prefix_v, like, Hkv):
    """(rows, k, v) of an optional shared prefix cache [Hkv][P][d]."""
    if prefix_k is None and prefix_v is None:
        return 0, None, None
    if prefix_k is None or prefix_v is None or prefix_k.shape != prefix_v.shape:
        raise ValueError("prefix_k and prefix_v must both be given, with one shape")
    if prefix_k.dim() != 3 or prefix_k.shape[0] != Hkv or prefix_k.shape[2] != like.shape[2]:
        raise ValueError("the prefix cache must be [%d][P][%d], has shape %s"
                         % (Hkv, like.shape[2], tuple(prefix_k.shape)))
    _same(like, prefix_k, prefix_v)
    return prefix_k.shape[1], _dev(prefix_k, "prefix_k"), _dev(prefix_v, "prefix_v")


def encode_resources(q, k, v, cu_len, max_len: int, rope_base: float, out, k_cache, v_cache,
                     lse=None, pos_base=None, softmax_scale: float = 0.0, stream=None,
                     prefix_k=None, prefix_v=None):
    """One layer of block-diagonal resource encoding (see recache.h), optionally
    after a shared prefix whose rotated cache is prefix_k / prefix_v [Hkv][P][d]."""
    T, Hq, d = q.shape
    Hkv = k.shape[1]
    n_res = cu_len.numel() - 1
    _same(q, k, v, out, k_cache, v_cache)
    _shape(k, "k", T, Hkv, d)
    _shape(v, "v", T, Hkv, d)
    _shape(out, "out", T, Hq, d)
    _shape(k_cache, "k_cache", Hkv, T, d)
    _shape(v_cache, "v_cache", Hkv, T, d)
    _shape(lse, "lse", Hq, T)
    _numel(pos_base, "pos_base", n_res)
    p_len, pk, pv = _prefix(prefix_k, prefix_v, q, Hkv)
    _call("recache_encode_resources", _dtype_code(q), cu_len.numel() - 1,
          _dev(cu_len, "cu_len", _i32()), T, int(max_len), Hq, Hkv, d, rope_base,
          _dev(pos_base, "pos_base", _i32()), p_len, pk, pv, softmax_scale, _dev(q, "q"),
          _dev(k, "k"), _dev(v, "v"), _dev(out, "out"), _dev(k_cache, "k_cache"),
          _dev(v_cache, "v_cache"), _dev(lse, "lse"), _stream(stream))


def encode_attention(q, k_cache, v_cache, cu_len, max_len: int, rope_base: float, out, lse=None,
                     pos_base=None, softmax_scale: float = 0.0, stream=None, prefix_k=None,
                     prefix_v=None):
    """Attention half of the encode over already built caches [Hkv][T][d]."""
    T, Hq, d = q.shape
    Hkv = k_cache.shape[0]
    n_res = cu_len.numel() - 1
    _same(q, k_cache, v_cache, out)
    _shape(k_cache, "k_cache", Hkv, T, d)
    _shape(v_cache, "v_cache", Hkv, T, d)
    _shape(out, "out", T, Hq, d)
    _shape(lse, "lse", Hq, T)
    _numel(pos_base, "pos_base", n_res)
    p_len, pk, pv = _prefix(prefix_k, prefix_v, q, Hkv)
    _call("recache_encode_attention", _dtype_code(q), cu_len.numel() - 1,
          _dev(cu_len, "cu_len", _i32()), T, int(max_len), Hq, Hkv, d, rope_base,
          _dev(pos_base, "pos_base", _i32()), p_len, pk, pv, softmax_scale, _dev(q, "q"),
          _dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"), _dev(out, "out"), _dev(lse, "lse"),
          _stream(stream))


def prune_gather(k_cache, v_cache, cu_len, cu_kept, kept_idx, k_kept, v_kept, stream=None):
    """Kept-row compaction of one layer's head-major caches."""
    Hkv, T, d = k_cache.shape
    _same(k_cache, v_cache, k_kept, v_kept)
    n_res = cu_len.numel() - 1
    K = k_kept.shape[1]
    _shape(v_cache, "v_cache", Hkv, T, d)
    _shape(k_kept, "k_kept", Hkv, K, d)
    _shape(v_kept, "v_kept", Hkv, K, d)
    _numel(cu_kept, "cu_kept", n_res + 1)
    _numel(kept_idx, "kept_idx", K)
    _call("recache_prune_gather", _dtype_code(k_cache), cu_len.numel() - 1,
          _dev(cu_len, "cu_len", _i32()), _dev(cu_kept, "cu_kept", _i32()),
          _dev(kept_idx, "kept_idx", _i32()), T, k_kept.shape[1], Hkv, d,
          _dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"), _dev(k_kept, "k_kept"),
          _dev(v_kept, "v_kept"), _stream(stream))


def build_routes(req_res_off, req_res, route_mask, cu_kept, route_off, route_res, route_tokens,
                 stream=None):
    """Route CSR for every (request, layer, KV group); route_mask is [n_res][L][G] uint8."""
    import torch

    n_res, L, G = route_mask.shape
    n_req = req_res_off.numel() - 1
    E = n_req * L * G
    _numel(cu_kept, "cu_kept", n_res + 1)
    _numel(route_off, "route_off", E + 1)
    _numel(route_tokens, "route_tokens", E)
    _at_least(route_res, "route_res", req_res.numel() * L * G)
    _call("recache_build_routes", req_res_off.numel() - 1, _dev(req_res_off, "req_res_off", _i32()),
          _dev(req_res, "req_res", _i32()), req_res.numel(), n_res, L, G,
          _dev(route_mask, "route_mask", (torch.uint8,)), _dev(cu_kept, "cu_kept", _i32()),
          _dev(route_off, "route_off", _i32()), _dev(route_res, "route_res", _i32()),
          _dev(route_tokens, "route_tokens", _i32()), _stream(stream))


def route_store_offsets(route_mask, cu_kept, store_off, total_kept: int | None = None,
                        stream=None):
    """Row tables of a route-compacted store: store_off is int32 [L][n_res * G + 1]."""
    import torch

    n_res, L, G = route_mask.shape
    _numel(cu_kept, "cu_kept", n_res + 1)
    _shape(store_off, "store_off", L, n_res * G + 1)
    if total_kept is None:
        total_kept = _total(cu_kept)
    _call("recache_route_store_offsets", n_res, L, G, int(total_kept),
          _dev(route_mask, "route_mask", (torch.uint8,)), _dev(cu_kept, "cu_kept", _i32()),
          _dev(store_off, "store_off", _i32()), _stream(stream))


def _total(cu):
    """Last entry of a device offsets array (one small device-to-host copy)."""
    return int(cu[-1].item())


def store_routes(k_cache, v_cache, cu_len, cu_kept, kept_idx, store_off, layer: int, k_store,
                 v_store, total_kept: int | None = None, stream=None):
    """One layer of a route-compacted store from head-major caches [Hkv][T][d].

    k_store / v_store are [rows][d] with rows = store_off[layer][-1]."""
    Hkv, T, d = k_cache.shape
    _same(k_cache, v_cache, k_store, v_store)
    L = store_off.shape[0]
    n_res = cu_len.numel() - 1
    _shape(v_cache, "v_cache", Hkv, T, d)
    _numel(cu_kept, "cu_kept", n_res + 1)
    _shape(store_off, "store_off", L, n_res * Hkv + 1)
    if k_store.dim() != 2 or k_store.shape[1] != d:
        raise ValueError("k_store must be [rows][%d], has shape %s" % (d, tuple(k_store.shape)))
    _shape(v_store, "v_store", *k_store.shape)
    if total_kept is None:
        total_kept = _total(cu_kept)
    _numel(kept_idx, "kept_idx", total_kept)
    _call("recache_store_routes", _dtype_code(k_cache), layer, L, cu_len.numel() - 1,
          _dev(cu_len, "cu_len", _i32()), _dev(cu_kept, "cu_kept", _i32()),
          _dev(kept_idx, "kept_idx", _i32()), T, int(total_kept), Hkv, d,
          _dev(store_off, "store_off", _i32()), k_store.shape[0], _dev(k_cache, "k_cache"),
          _dev(v_cache, "v_cache"), _dev(k_store, "k_store"), _dev(v_store, "v_store"),
          _stream(stream))


def attend_workspace_bytes(n_req, max_q, max_ctx, max_kv, n_q_heads, n_kv_heads, head_dim) -> int:
    return int(lib().recache_attend_workspace_bytes(n_req, max_q, max_ctx, max_kv, n_q_heads,
                                                    n_kv_heads, head_dim))


def attend_plan_bytes(n_req: int, n_layers: int, n_kv_heads: int) -> int:
    return int(lib().recache_attend_plan_bytes(n_req, n_layers, n_kv_heads))


def attend_plan(cu_q, cu_ctx, route_tokens, n_layers: int, n_q_heads: int, n_kv_heads: int, plan,
                stream=None):
    """Work order of the attend kernels for every layer of a batch (int32
    plan[n_layers][n_req * n_kv_heads]); pass it as attend_cached(plan=...)."""
    n_req = cu_q.numel() - 1
    _numel(cu_ctx, "cu_ctx", n_req + 1)
    _numel(route_tokens, "route_tokens", n_req * n_layers * n_kv_heads)
    _shape(plan, "plan", n_layers, n_req * n_kv_heads)
    _call("recache_attend_plan", n_layers, n_req, n_q_heads, n_kv_heads,
          _dev(cu_q, "cu_q", _i32()), _dev(cu_ctx, "cu_ctx", _i32()),
          _dev(route_tokens, "route_tokens", _i32()), _dev(plan, "plan", _i32()), _stream(stream))


def _attend_args(q, ctx_k, ctx_v, cu_q, cu_ctx, max_q, max_ctx, res_k, res_v, cu_kept, route_off,
                 route_res, route_tokens, layer, n_layers, out, max_route_len, lse, max_kv,
                 softmax_scale, res_off, plan):
    """Checked C arguments shared by the two attend entry points, up to
    plan / out / lse (the caller appends the rest)."""
    total_q, Hq, d = q.shape
    Hkv = ctx_k.shape[0]
    n_req = cu_q.numel() - 1
    n_res = cu_kept.numel() - 1
    E = n_req * n_layers * Hkv
    _same(q, ctx_k, ctx_v, res_k, res_v, out)
    _shape(out, "out", total_q, Hq, d)
    _shape(lse, "lse", Hq, total_q)
    if ctx_k.dim() != 3 or ctx_k.shape[2] != d:
        raise ValueError("ctx_k must be [%d][rows][%d], has shape %s" % (Hkv, d, tuple(ctx_k.shape)))
    _shape(ctx_v, "ctx_v", *ctx_k.shape)
    _numel(cu_ctx, "cu_ctx", n_req + 1)
    _numel(route_off, "route_off", E + 1)
    _numel(route_tokens, "route_tokens", E)
    _shape(plan, "plan", n_layers, n_req * Hkv)
    if res_off is not None:
        _numel(res_off, "res_off", n_res * Hkv + 1)
        if res_k.dim() != 2 or res_k.shape[1] != d:
            raise ValueError("a route-compacted store is [rows][%d], res_k has shape %s"
                             % (d, tuple(res_k.shape)))
        res_rows = res_k.shape[0]
    else:
        if res_k.dim() != 3 or res_k.shape[0] != Hkv or res_k.shape[2] != d:
            raise ValueError("res_k must be [%d][rows][%d], has shape %s"
                             % (Hkv, d, tuple(res_k.shape)))
        res_rows = res_k.shape[1]
    _shape(res_v, "res_v", *res_k.shape)
    return (_dtype_code(q), layer, n_layers, n_req, _dev(cu_q, "cu_q", _i32()),
            _dev(cu_ctx, "cu_ctx", _i32()), total_q, int(max_q), int(max_ctx), int(max_kv),
            int(max_route_len), Hq, Hkv, d, softmax_scale, _dev(q, "q"), _dev(ctx_k, "ctx_k"),
            _dev(ctx_v, "ctx_v"), ctx_k.shape[1], _dev(res_k, "res_k"), _dev(res_v, "res_v"),
            res_rows, _dev(cu_kept, "cu_kept", _i32()), _dev(res_off, "res_off", _i32()),
            _dev(route_off, "route_off", _i32()), _dev(route_res, "route_res", _i32()),
            _dev(route_tokens, "route_tokens", _i32()), _dev(plan, "plan", _i32()),
            _dev(out, "out"), _dev(lse, "lse"))


def route_len_bound(req_res_off) -> int:
    """[host] max_route_len for recache_attend_cached: the most resources any
    request lists (a host copy of req_res_off), which bounds every route list."""
    a = np.asarray(req_res_off, dtype=np.int64)
    return int(np.diff(a).max()) if len(a) > 1 else 0


def attend_cached(q, ctx_k, ctx_v, cu_q, cu_ctx, max_q: int, max_ctx: int, res_k, res_v, cu_kept,
                  route_off, route_res, route_tokens, layer: int, n_layers: int, out, *,
                  max_route_len: int, lse=None, workspace=None, max_kv: int = 0,
                  softmax_scale: float = 0.0, res_off=None, plan=None, stream=None):
    """Conversation queries over routed kept resource rows + causal context (one layer).

    res_k / res_v are [Hkv][rows][d] kept rows, or with res_off (this layer's
    row of a store table) a route-compacted store [rows][d].  max_route_len
    bounds the resources of every route list (route_len_bound of the request
    lists; at most 1024).  plan, from attend_plan for this batch, only
    reorders the grid (results bit-identical)."""
    args = _attend_args(q, ctx_k, ctx_v, cu_q, cu_ctx, max_q, max_ctx, res_k, res_v, cu_kept,
                        route_off, route_res, route_tokens, layer, n_layers, out, max_route_len,
                        lse, max_kv, softmax_scale, res_off, plan)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _call("recache_attend_cached", *args, _dev(workspace, "workspace"), ws_bytes, _stream(stream))


def attend_cached_noalloc(q, ctx_k, ctx_v, cu_q, cu_ctx, max_q: int, max_ctx: int, res_k, res_v,
                          cu_kept, route_off, route_res, route_tokens, layer: int, n_layers: int,
                          out, *, max_route_len: int, lse=None, max_kv: int = 0,
                          softmax_scale: float = 0.0, res_off=None, plan=None, stream=None):
    """attend_cached without a workspace: decode's split partials live in the
    library's static per-GPU scratch (see recache.h: calls that overlap on one
    GPU race)."""
    args = _attend_args(q, ctx_k, ctx_v, cu_q, cu_ctx, max_q, max_ctx, res_k, res_v, cu_kept,
                        route_off, route_res, route_tokens, layer, n_layers, out, max_route_len,
                        lse, max_kv, softmax_scale, res_off, plan)
    _call("recache_attend_cached_noalloc", *args, _stream(stream))


def check_offsets(cu, total: int, strict: bool = True) -> None:
    """Host validator of packing offsets (numpy / list)."""
    a = np.ascontiguousarray(np.asarray(cu, dtype=np.int32))
    _call("recache_check_offsets", a.ctypes.data, len(a) - 1, int(total), int(strict))


def check_kept(cu_len, cu_kept, kept_idx) -> None:
    """Host validator of kept-token lists (numpy / list)."""
    a = np.ascontiguousarray(np.asarray(cu_len, dtype=np.int32))
    b = np.ascontiguousarray(np.asarray(cu_kept, dtype=np.int32))
    c = np.ascontiguousarray(np.asarray(kept_idx, dtype=np.int32))
    _call("recache_check_kept", a.ctypes.data, b.ctypes.data, c.ctypes.data, len(a) - 1)


def check_encode_lengths(cu_len, max_len: int) -> None:
    """Host validator of an encode call's packing offsets against max_len."""
    a = np.ascontiguousarray(np.asarray(cu_len, dtype=np.int32))
    _call("recache_check_encode_lengths", a.ctypes.data, len(a) - 1, int(a[-1]), int(max_len))


def check_requests(req_res_off, req_res, n_res: int, max_route_len: int) -> None:
    """Host validator of request lists against n_res and max_route_len."""
    a = np.ascontiguousarray(np.asarray(req_res_off, dtype=np.int32))
    b = np.ascontiguousarray(np.asarray(req_res, dtype=np.int32))
    _call("recache_check_requests", a.ctypes.data, b.ctypes.data if b.size else None, len(a) - 1,
          int(a[-1]), int(n_res), int(max_route_len))


def select_routes(s_layer, s_group, k_layers: int, k_groups: int) -> dict:
    """[host] Omega* = top-k_layers layers x top-k_groups groups by contribution
    weight (see recache.h).  Returns route_mask[L][G] (uint8), the weights,
    rho and the contribution coverages."""
    import numpy as np

    sl = np.ascontiguousarray(s_layer, dtype=np.float64)
    sg = np.ascontiguousarray(s_group, dtype=np.float64)
    L, G = len(sl), len(sg)
    mask = np.zeros((L, G), np.uint8)
    wl, wg = np.zeros(L), np.zeros(G)
    out = (ctypes.c_double * 3)()
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    _call("recache_select_routes", L, G, p(sl), p(sg), int(k_layers), int(k_groups), p(mask),
          p(wl), p(wg), ctypes.byref(out, 0), ctypes.byref(out, 8), ctypes.byref(out, 16))
    return {"mask": mask, "w_layer": wl, "w_group": wg, "rho": out[0], "cc_layer": out[1],
            "cc_group": out[2]}
