"""C-ABI contract checks that need no GPU: the library loads, exports every
symbol declared in include/recache.h, and rejects bad arguments on the host
with the documented status before any HIP call (so fake, non-null device
pointers below are never dereferenced)."""
import os
import re

import pytest

from paper_2608_19662_amd import recache as rc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "recache.h")
FAKE = 0x1000  # never reaches a kernel: every call below fails validation


def declared_symbols():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(recache_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = rc.lib()
    names = declared_symbols()
    assert len(names) >= 10
    for n in names:
        assert hasattr(L, n), n
    assert sorted(rc.EXPORTS) == names


def test_version_and_clean_error():
    assert rc.version() == 100
    rc.check_offsets([0, 3, 5], 5)
    assert rc.last_error() == ""


def test_check_offsets():
    rc.check_offsets([0, 1, 1, 4], 4, strict=False)
    for bad, total, strict in [([1, 2], 2, True), ([0, 2, 1], 1, False), ([0, 2, 2], 2, True),
                               ([0, 2, 3], 4, True)]:
        with pytest.raises(rc.RecacheError) as e:
            rc.check_offsets(bad, total, strict)
        assert e.value.code == rc.EINVAL
        assert rc.last_error()


def test_check_kept():
    rc.check_kept([0, 3, 5], [0, 2, 3], [0, 2, 1])
    for cu_kept, kept in [([0, 2, 3], [2, 0, 1]), ([0, 2, 3], [0, 3, 1]), ([0, 0, 1], [1]),
                          ([0, 2, 3], [1, 1, 0]), ([0, 4, 5], [0, 1, 2, 2, 0])]:
        with pytest.raises(rc.RecacheError) as e:
            rc.check_kept([0, 3, 5], cu_kept, kept)
        assert e.value.code == rc.EINVAL


def enc(**kw):
    a = dict(dtype=1, n_res=2, cu_len=FAKE, total_T=10, max_len=6, Hq=32, Hkv=8, d=128,
             base=1e6, pos_base=None, p_len=0, pk=None, pv=None, scale=0.0, q=FAKE, k=FAKE,
             v=FAKE, out=FAKE, kc=FAKE, vc=FAKE, lse=None, stream=None)
    a.update(kw)
    return rc.lib().recache_encode_resources(*a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(d=96), rc.EUNSUPPORTED),
    (dict(dtype=2), rc.EUNSUPPORTED),
    (dict(Hq=30), rc.EINVAL),
    (dict(Hq=72), rc.EUNSUPPORTED),  # 9 query heads per KV head on the bf16 kernels
    (dict(n_res=0), rc.EINVAL),
    (dict(total_T=1), rc.EINVAL),
    (dict(max_len=0), rc.EINVAL),
    (dict(max_len=11), rc.EINVAL),
    (dict(q=None), rc.EINVAL),
    (dict(cu_len=None), rc.EINVAL),
    (dict(base=0.5), rc.EINVAL),
    (dict(scale=float("nan")), rc.EINVAL),
    (dict(p_len=-1), rc.EINVAL),
    (dict(p_len=4), rc.EINVAL),  # prefix rows without prefix caches
    (dict(p_len=4, pk=FAKE), rc.EINVAL),
])
def test_encode_rejects(kw, code):
    assert enc(**kw) == code
    assert rc.last_error()


def test_encode_fp32_any_ratio_passes_head_check():
    # fp32 path accepts 9 query heads per KV head; the next check (null q) still fires
    assert enc(dtype=0, Hq=72, q=None) == rc.EINVAL
    assert "null" in rc.last_error()


def att(**kw):
    a = dict(dtype=1, layer=0, n_layers=36, n_req=2, cu_q=FAKE, cu_ctx=FAKE, total_q=2, max_q=1,
             max_ctx=16, max_kv=0, max_route_len=32, Hq=32, Hkv=8, d=128, scale=0.0, q=FAKE,
             ck=FAKE, cv=FAKE, ctx_rows=32, rk=FAKE, rv=FAKE, res_rows=8, cu_kept=FAKE,
             res_off=None, route_off=FAKE, route_res=FAKE, route_tokens=FAKE, plan=None, out=FAKE,
             lse=None, ws=None, ws_bytes=0, stream=None)
    a.update(kw)
    return rc.lib().recache_attend_cached(*a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(layer=36), rc.EINVAL),
    (dict(layer=-1), rc.EINVAL),
    (dict(max_q=17), rc.EINVAL),          # Tq > Tc
    (dict(max_q=0), rc.EINVAL),
    (dict(total_q=1), rc.EINVAL),
    (dict(max_route_len=2000), rc.EUNSUPPORTED),
    (dict(d=80), rc.EUNSUPPORTED),
    (dict(res_rows=0), rc.EINVAL),
    (dict(route_res=None), rc.EINVAL),
    (dict(ws=None), rc.EWORKSPACE),       # decode needs split-KV scratch
    (dict(ws=FAKE, ws_bytes=16), rc.EWORKSPACE),
    (dict(plan=FAKE + 2), rc.EINVAL),     # a plan is int32
])
def test_attend_rejects(kw, code):
    assert att(**kw) == code
    assert rc.last_error()


def test_workspace_sizes():
    n = rc.attend_workspace_bytes(64, 1, 4096, 9000, 32, 8, 128)
    assert n > 0 and n % 4 == 0
    assert rc.attend_workspace_bytes(8, 2048, 2048, 0, 32, 8, 128) == 0


def test_prune_and_routes_reject():
    L = rc.lib()
    assert L.recache_prune_gather(1, 2, FAKE, FAKE, FAKE, 10, 11, 8, 128, FAKE, FAKE, FAKE, FAKE,
                                  None) == rc.EINVAL
    assert L.recache_prune_gather(1, 2, FAKE, FAKE, FAKE, 10, 1, 8, 128, FAKE, FAKE, FAKE, FAKE,
                                  None) == rc.EINVAL
    assert L.recache_prune_gather(1, 2, FAKE, FAKE, None, 10, 4, 8, 128, FAKE, FAKE, FAKE, FAKE,
                                  None) == rc.EINVAL
    assert L.recache_build_routes(0, FAKE, FAKE, 4, 4, 36, 8, FAKE, FAKE, FAKE, FAKE, FAKE,
                                  None) == rc.EINVAL
    assert L.recache_build_routes(2, FAKE, FAKE, 2 ** 28, 4, 36, 8, FAKE, FAKE, FAKE, FAKE, FAKE,
                                  None) == rc.EINVAL
    assert L.recache_rope_kv(1, 8, 8, 128, 1e4, FAKE, FAKE, FAKE, FAKE, FAKE, 10, 4,
                             None) == rc.EINVAL  # rows [4, 12) overflow 10


def store(**kw):
    a = dict(dtype=1, layer=0, n_layers=36, n_res=4, cu_len=FAKE, cu_kept=FAKE, kept_idx=FAKE,
             T=100, kept=30, Hkv=8, d=128, off=FAKE, rows=60, kc=FAKE, vc=FAKE, ks=FAKE,
             vs=FAKE, stream=None)
    a.update(kw)
    return rc.lib().recache_store_routes(*a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(layer=36), rc.EINVAL),
    (dict(kept=101), rc.EINVAL),          # more kept rows than rows
    (dict(kept=3), rc.EINVAL),            # fewer than one per resource
    (dict(rows=241), rc.EINVAL),          # more than every route of every kept row
    (dict(rows=-1), rc.EINVAL),
    (dict(off=None), rc.EINVAL),
    (dict(ks=None), rc.EINVAL),
    (dict(d=96), rc.EUNSUPPORTED),
    (dict(dtype=7), rc.EUNSUPPORTED),
])
def test_store_routes_rejects(kw, code):
    assert store(**kw) == code
    assert rc.last_error()


def test_store_offsets_rejects():
    L = rc.lib()
    assert L.recache_route_store_offsets(0, 36, 8, 10, FAKE, FAKE, FAKE, None) == rc.EINVAL
    assert L.recache_route_store_offsets(4, 36, 8, 3, FAKE, FAKE, FAKE, None) == rc.EINVAL
    assert L.recache_route_store_offsets(4, 36, 8, 2 ** 28, FAKE, FAKE, FAKE, None) == rc.EINVAL
    assert L.recache_route_store_offsets(4, 36, 8, 10, None, FAKE, FAKE, None) == rc.EINVAL
    # an empty store is valid and launches nothing
    assert store(rows=0, ks=None, vs=None) == rc.OK


def test_python_binding_refuses_host_tensors():
    torch = pytest.importorskip("torch")
    x = torch.zeros(4, 2, 64)
    with pytest.raises(TypeError):
        rc.rope_q(x, torch.zeros(4, dtype=torch.int32), 1e4)


def test_check_encode_lengths():
    rc.check_encode_lengths([0, 3, 5, 9], 4)
    for cu, max_len in [([0, 3, 5, 9], 3),      # a resource of 4 tokens, max_len 3
                        ([0, 3, 3, 9], 6),      # an empty resource
                        ([1, 3], 5)]:           # offsets not from 0
        with pytest.raises(rc.RecacheError) as e:
            rc.check_encode_lengths(cu, max_len)
        assert e.value.code == rc.EINVAL
        assert rc.last_error()


def test_check_requests():
    rc.check_requests([0, 2, 2, 5], [1, 0, 3, 2, 1], 4, 3)
    rc.check_requests([0, 0], [], 4, 0)           # a request with no resources
    for off, res, n_res, bound in [([0, 2, 2, 5], [1, 0, 3, 2, 1], 4, 2),  # 3 listed, bound 2
                                   ([0, 2], [0, 4], 4, 8),                 # id outside [0, 4)
                                   ([0, 2], [0, 1], 4, 1025),              # over the 1024 limit
                                   ([0, 3, 2], [0, 1, 2], 4, 8)]:          # decreasing offsets
        with pytest.raises(rc.RecacheError) as e:
            rc.check_requests(off, res, n_res, bound)
        assert e.value.code == rc.EINVAL
    assert rc.route_len_bound([0, 2, 2, 5]) == 3


def test_python_binding_checks_shapes_first():
    """Every tensor's shape is checked against the call's sizes before any
    device pointer is taken (a buffer smaller than the sizes passed on would
    become an access outside it); host tensors of the right shapes are then
    refused as host memory."""
    torch = pytest.importorskip("torch")
    bf = torch.bfloat16
    z = lambda *s, dt=bf: torch.zeros(*s, dtype=dt)
    i = lambda n: torch.zeros(n, dtype=torch.int32)
    T, Hq, Hkv, d = 10, 8, 2, 64
    good = dict(q=z(T, Hq, d), k=z(T, Hkv, d), v=z(T, Hkv, d), cu_len=i(3), max_len=6,
                rope_base=1e6, out=z(T, Hq, d), k_cache=z(Hkv, T, d), v_cache=z(Hkv, T, d),
                lse=z(Hq, T, dt=torch.float32))
    for key, bad in [("out", z(T - 1, Hq, d)), ("k_cache", z(Hkv, T + 1, d)),
                     ("v", z(T, Hkv + 1, d)), ("lse", z(Hq, T - 1, dt=torch.float32))]:
        with pytest.raises(ValueError):
            rc.encode_resources(**dict(good, **{key: bad}))
    with pytest.raises(TypeError):
        rc.encode_resources(**good)
    n_req, L = 2, 3
    E = n_req * L * Hkv
    ga = dict(q=z(4, Hq, d), ctx_k=z(Hkv, 9, d), ctx_v=z(Hkv, 9, d), cu_q=i(n_req + 1),
              cu_ctx=i(n_req + 1), max_q=2, max_ctx=5, res_k=z(Hkv, 7, d), res_v=z(Hkv, 7, d),
              cu_kept=i(4), route_off=i(E + 1), route_res=i(30), route_tokens=i(E), layer=0,
              n_layers=L, out=z(4, Hq, d), max_route_len=3)
    for key, bad in [("out", z(5, Hq, d)), ("route_off", i(E)), ("route_tokens", i(E + 1)),
                     ("res_v", z(Hkv, 6, d)), ("ctx_v", z(Hkv, 8, d)), ("cu_ctx", i(n_req))]:
        with pytest.raises(ValueError):
            rc.attend_cached(**dict(ga, **{key: bad}))
    with pytest.raises(ValueError):  # a store table row of the wrong length
        rc.attend_cached(**dict(ga, res_k=z(7, d), res_v=z(7, d), res_off=i(3 * Hkv)))
    with pytest.raises(TypeError):  # max_route_len has no default
        rc.attend_cached(**{k: v for k, v in ga.items() if k != "max_route_len"})
    with pytest.raises(TypeError):
        rc.attend_cached(**ga)


def test_noalloc_rejects_partials_beyond_the_scratch():
    """The allocation-free attend checks its scratch need on the host, before
    any HIP call: 4096 decode requests x 64 query heads need 4096 * 64 *
    (128 + 2) * 4 bytes of split partials, more than the 32 MiB static array."""
    L = rc.lib()
    need = rc.attend_workspace_bytes(4096, 1, 64, 0, 64, 8, 128)
    assert need > 32 * 1024 * 1024
    code = L.recache_attend_cached_noalloc(1, 0, 1, 4096, FAKE, FAKE, 4096, 1, 64, 0, 4, 64, 8,
                                           128, 0.0, FAKE, FAKE, FAKE, 64, FAKE, FAKE, 8, FAKE, None,
                                           FAKE, FAKE, FAKE, None, FAKE, None, None)
    assert code == rc.EWORKSPACE
    assert "static scratch" in rc.last_error()
    # and the ordinary argument checks come first
    assert L.recache_attend_cached_noalloc(1, 5, 1, 4096, FAKE, FAKE, 4096, 1, 64, 0, 4, 64, 8,
                                           128, 0.0, FAKE, FAKE, FAKE, 64, FAKE, FAKE, 8, FAKE,
                                           None, FAKE, FAKE, FAKE, None, FAKE, None, None) == rc.EINVAL


def test_attend_plan_sizes_and_checks():
    """The work-order builder: its size, and its host checks (no HIP call)."""
    L = rc.lib()
    assert rc.attend_plan_bytes(8, 36, 8) == 36 * 8 * 8 * 4
    assert rc.attend_plan_bytes(0, 36, 8) == 0
    # n_layers, n_req, n_q_heads, n_kv_heads, cu_q, cu_ctx, route_tokens, plan, stream
    assert L.recache_attend_plan(36, 8, 32, 8, FAKE, FAKE, FAKE, None, None) == rc.EINVAL
    assert "null" in rc.last_error()
    assert L.recache_attend_plan(0, 8, 32, 8, FAKE, FAKE, FAKE, FAKE, None) == rc.EINVAL
    assert L.recache_attend_plan(36, 8, 30, 8, FAKE, FAKE, FAKE, FAKE, None) == rc.EINVAL
    assert L.recache_attend_plan(36, 8, 32, 8, FAKE, FAKE, FAKE, FAKE + 1, None) == rc.EINVAL
    assert "aligned" in rc.last_error()
    # more pairs than one plan sorts in LDS
    assert L.recache_attend_plan(1, 1025, 32, 8, FAKE, FAKE, FAKE, FAKE, None) == rc.EUNSUPPORTED
    assert "8192" in rc.last_error()
