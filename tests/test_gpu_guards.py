"""GPU tests of the size guards: a call whose sizes understate its inputs
(a resource longer than max_len, a request with more queries than max_q, a
route list longer than the 1024 the kernels take, a decode request with more
than one query) gets NaN in the affected outputs instead of rows left
unwritten or resources dropped.  Every access stays inside the buffers the
call describes; the host validators reject the same inputs before a launch
(tests/test_abi.py)."""
import numpy as np
import pytest
import torch

from gpu_helpers import DEV, Routes, i32
from paper_2608_19662_amd import recache as rc
from paper_2608_19662_amd.workloads import EncodeWorkload, normal, prefix
from test_gpu_parity import many_segments, small_attend

pytestmark = pytest.mark.gpu


def print_case(*a):
    print("case:", *a, flush=True)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_encode_resource_longer_than_max_len(dtype):
    print_case("guard: encode max_len", dtype)
    lengths = np.array([40, 300, 17], np.int32)
    w = EncodeWorkload(seed=81, lengths=lengths, n_q_heads=8, n_kv_heads=2, head_dim=128,
                       dtype=dtype, rope_base=1e6)
    q, k, v = w.tensors(DEV)
    T = w.total
    out = torch.zeros_like(q)
    kc = torch.empty(2, T, 128, dtype=q.dtype, device=DEV)
    vc = torch.empty_like(kc)
    lse = torch.zeros(8, T, dtype=torch.float32, device=DEV)
    with pytest.raises(rc.RecacheError):
        rc.check_encode_lengths(w.cu_len, 200)
    rc.encode_resources(q, k, v, i32(w.cu_len), 200, w.rope_base, out, kc, vc, lse=lse)
    torch.cuda.synchronize()
    cu = w.cu_len
    # rows of the long resource past what a grid sized by max_len = 200 covers
    # are NaN in every head; the short resources are computed normally
    # (fp32: one wave per row up to max_len; bf16 with 4 query heads per KV
    # head: 32-row tiles, ceil(200 / 32) = 7 of them)
    covered = 200 if dtype == "f32" else 224
    assert torch.isnan(out[cu[1] + covered:cu[2]].float()).all()
    assert torch.isnan(lse[:, cu[1] + covered:cu[2]]).all()
    assert torch.isfinite(out[cu[0]:cu[1]].float()).all()
    assert torch.isfinite(out[cu[2]:cu[3]].float()).all()


def test_prefill_queries_past_max_q():
    print_case("guard: prefill max_q")
    w = small_attend(82, 2, 4, 32, 8, 128, "bf16", [300, 40], [300, 60])
    rt = Routes(w)
    rt.max_q = 170  # understates request 0's 300 queries (total 340 = n_req * max_q)
    q, ck, cv, rk, rv = w.layer_tensors(0, DEV)
    out, lse = rt.attend(q, ck, cv, rk, rv, 0)
    torch.cuda.synchronize()
    # the grid covers ceil(170 / 32) = 6 tiles of 32 rows per request
    assert torch.isnan(out[192:300].float()).all() and torch.isnan(lse[:, 192:300]).all()
    assert torch.isfinite(out[300:340].float()).all()


@pytest.mark.parametrize("ql,cl", [([70, 1], [100, 5]), ([1, 1], [1, 300])])
def test_route_list_over_the_limit(ql, cl):
    print_case("guard: route list over 1024", ql, cl)
    w = many_segments(83, ql, cl, n_res=1100)
    rt = Routes(w)
    rt.max_route_len = 1024  # understates the 1100 resources every request lists
    q, ck, cv, rk, rv = w.layer_tensors(0, DEV)
    mk = rt.max_kv(0)
    out, lse = rt.attend(q, ck, cv, rk, rv, 0, workspace=rt.workspace(mk), max_kv=mk)
    torch.cuda.synchronize()
    assert torch.isnan(out.float()).all() and torch.isnan(lse).all()


def test_decode_request_with_two_queries():
    print_case("guard: decode with Tq = 2")
    w = small_attend(84, 3, 4, 32, 8, 128, "bf16", [1, 2, 1], [50, 60, 70])
    rt = Routes(w)
    rt.max_q = 1  # the decode path, but request 1 has two queries
    q, ck, cv, rk, rv = w.layer_tensors(0, DEV)
    mk = rt.max_kv(0)
    out = torch.zeros_like(q)
    lse = torch.zeros(32, 4, dtype=torch.float32, device=DEV)
    # total_q = 4 > n_req * max_q = 3 is refused on the host
    with pytest.raises(rc.RecacheError):
        rc.attend_cached(q, ck, cv, rt.cu_q, rt.cu_ctx, 1, 70, rk, rv, rt.cu_rows, rt.route_off,
                         rt.route_res, rt.route_tokens, 0, w.n_layers, out, lse=lse,
                         workspace=rt.workspace(mk), max_kv=mk, max_route_len=4)
    # with the per-request counts disagreeing (0 and 2, total still n_req) the
    # kernels answer NaN for the request whose count is not one
    cu_q = i32([0, 1, 1, 3])
    q3 = q[:3].contiguous()
    out3 = torch.zeros_like(q3)
    lse3 = torch.zeros(32, 3, dtype=torch.float32, device=DEV)
    rc.attend_cached(q3, ck, cv, cu_q, rt.cu_ctx, 1, 70, rk, rv, rt.cu_rows, rt.route_off,
                     rt.route_res, rt.route_tokens, 0, w.n_layers, out3, lse=lse3,
                     workspace=rt.workspace(mk), max_kv=mk, max_route_len=4)
    torch.cuda.synchronize()
    assert torch.isfinite(out3[0].float()).all()
    assert torch.isnan(out3[1].float()).all() and torch.isnan(lse3[:, 1]).all()
