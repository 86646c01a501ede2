"""The allocation-free attend entry point against the one that takes a
workspace: the same kernels on the same inputs, so every output must be
bit-identical.  Two decode calls in a row on one GPU (the second smaller,
after the first left its partials in the shared static scratch), then a
prefill call (which uses no scratch).  The host-side rejection of a decode
whose partials exceed the scratch is checked in test_abi.py."""
import numpy as np
import pytest
import torch

from gpu_helpers import DEV, Routes
from paper_2608_19662_amd import recache as rc
from test_gpu_parity import small_attend

pytestmark = pytest.mark.gpu


def both(w, layer):
    """(out, lse) from recache_attend_cached with a workspace and from
    recache_attend_cached_noalloc, on one layer of w."""
    rt = Routes(w)
    q, ck, cv, rk, rv = w.layer_tensors(layer, DEV)
    mk = rt.max_kv(layer)
    ref_out, ref_lse = rt.attend(q, ck, cv, rk, rv, layer, workspace=rt.workspace(mk), max_kv=mk)
    out = torch.full_like(q, float("nan"))
    lse = torch.full((w.n_q_heads, q.shape[0]), float("nan"), dtype=torch.float32, device=DEV)
    rc.attend_cached_noalloc(q, ck, cv, rt.cu_q, rt.cu_ctx, rt.max_q, rt.max_ctx, rk, rv,
                             rt.cu_rows, rt.route_off, rt.route_res, rt.route_tokens, layer,
                             w.n_layers, out, lse=lse, max_kv=mk,
                             max_route_len=max(rt.max_route_len, 1))
    torch.cuda.synchronize()
    return (ref_out, ref_lse), (out, lse)


def test_noalloc_decode_twice_then_prefill():
    cases = [
        # a larger decode first, then a smaller one reusing the same scratch
        (small_attend(91, 6, 10, 32, 8, 128, "bf16", [1] * 6, [3000, 17, 1200, 64, 2500, 900],
                      max_len=900), 1),
        (small_attend(92, 2, 4, 8, 2, 64, "bf16", [1, 1], [40, 300], max_len=300), 0),
        # prefill: no scratch involved
        (small_attend(93, 3, 6, 32, 8, 128, "bf16", [100, 1, 64], [130, 1, 200]), 2),
    ]
    for w, layer in cases:
        print("case: noalloc", w.seed, list(w.q_lens), list(w.ctx_lens), flush=True)
        (ro, rl), (o, l) = both(w, layer)
        assert torch.equal(o, ro), "out differs from recache_attend_cached"
        assert torch.equal(l, rl), "lse differs from recache_attend_cached"
