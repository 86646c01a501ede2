"""GPU parity where the softmax's reference max has to move.

With N(0,1) inputs the logits of later keys never rise far above the first
tile's, so the kernels' rescale paths (the attention kernel's reference max,
the decode kernel's running max) would stay untested.  Here one dimension of
Q and K carries a large component that grows along the key stream (about 16
in log2 units per 64-key tile, so that weights relative to the first tile's
max pass 2^16 tile after tile), plus single keys far above everything before
them (weights past the fp32 range relative to the reference) and a stream
whose logits fall.  Results are checked against the fp64 oracle with the
usual bf16 rules (Sec. 3 softmax attention; the final mask of Fig. 2).
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, Routes, check, lse_rule
from paper_2608_19662_amd.workloads import EncodeWorkload

from test_gpu_parity import gpu_encode, print_case, small_attend

pytestmark = pytest.mark.gpu


def ramp(n, step, dtype):
    return (step * torch.arange(n, dtype=torch.float32)).to(dtype)


@pytest.mark.parametrize("Hq,Hkv,d", [(32, 8, 128), (8, 2, 64), (12, 4, 64)])
def test_reference_moves_encode(Hq, Hkv, d):
    """Encode: a rising resource with two spikes, a falling one, short ones."""
    print_case("softmax reference, encode", Hq, Hkv, d)
    lengths = np.array([700, 300, 129, 65, 1], np.int32)
    w = EncodeWorkload(seed=61, lengths=lengths, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=d,
                       dtype="bf16", rope_base=1e6)
    q, k, v = w.tensors("cpu")
    # dimension d/2 - 1 pairs with d - 1 and turns by 1e6^(-(d - 2)/d) rad per
    # position, so the large component keeps its sign along a resource
    c = d // 2 - 1
    q[:, :, c] = 4.0
    for r, n in enumerate(lengths):
        o = int(w.cu_len[r])
        up = ramp(int(n), 0.5, k.dtype)
        k[o:o + n, :, c] = (up if r != 1 else up.flip(0))[:, None]
    o0 = int(w.cu_len[0])
    k[o0 + 400, :, c] = 900.0   # about 360 above the reference in log2 units
    k[o0 + 450, :, c] = 1200.0  # and again past the moved reference
    out, kc, vc, lse = gpu_encode(w, q.to(DEV), k.to(DEV), v.to(DEV))
    ref = oracle.encode(q, k, v, w.cu_len, w.rope_base)
    check(out, ref["out"], "bf16", "out")
    check(lse, ref["lse"], "lse", "lse")
    check(kc, ref["k_cache"], "bf16-ulp", "k_cache")
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()


@pytest.mark.parametrize("Hq,Hkv,d", [(32, 8, 128), (12, 4, 64)])
@pytest.mark.parametrize("q_lens,ctx_lens", [([100, 1, 64], [330, 1, 700]),   # prefill
                                             ([1, 1, 1], [300, 1200, 64])])  # decode
def test_reference_moves_attend(q_lens, ctx_lens, Hq, Hkv, d):
    """Prefill and decode over kept resource rows and context rows whose keys
    rise along their buffers, with spikes in both."""
    print_case("softmax reference, attend", q_lens, ctx_lens, Hq, Hkv, d)
    w = small_attend(62, 3, 6, Hq, Hkv, d, "bf16", q_lens, ctx_lens, max_len=400, mask_p=0.7)
    layer = 1
    q, ck, cv, rk, rv = w.layer_tensors(layer, DEV, compacted=True)
    q[:, :, 0] = 4.0
    ck[:, :, 0] = ramp(ck.shape[1], 0.25, ck.dtype).to(DEV)[None, :]
    rk[:, :, 0] = ramp(rk.shape[1], 0.25, rk.dtype).to(DEV)[None, :]
    ck[:, ck.shape[1] // 2, 0] = 700.0
    rk[:, rk.shape[1] // 3, 0] = 900.0
    rt = Routes(w)
    max_kv = rt.max_kv(layer)
    out, lse = rt.attend(q, ck, cv, rk, rv, layer, workspace=rt.workspace(max_kv), max_kv=max_kv)
    torch.cuda.synchronize()
    rout, rlse = oracle.attend(q.cpu(), ck.cpu(), cv.cpu(), w.cu_q, w.cu_ctx, rk.cpu(), rv.cpu(),
                               w.cu_rows, w.req_res_off, w.req_res, w.mask, layer)
    check(out, rout, "bf16", "attend out")
    check(lse, rlse.T, lse_rule("bf16"), "attend lse")
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
