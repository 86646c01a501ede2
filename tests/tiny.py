"""Tiny random scenarios shared by the oracle pin tests (inputs only)."""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from paper_2608_19662_amd.workloads import prefix


@dataclass
class Tiny:
    lengths: np.ndarray          # resource pool lengths
    q: np.ndarray                # [T][Hq][d] raw resource queries
    k: np.ndarray                # [T][Hkv][d]
    v: np.ndarray
    req_res_off: np.ndarray
    req_res: np.ndarray
    mask: np.ndarray             # [n_res][L][G]
    cu_kept: np.ndarray | None
    kept_idx: np.ndarray | None
    ctx_q: list                  # per request raw [Tc][Hq][d]
    ctx_k: list
    ctx_v: list
    ctx_pos: list                # per request [Tc]
    q_lens: np.ndarray
    base: float

    @property
    def cu_len(self):
        return prefix(self.lengths)

    def kept_list(self, r):
        if self.kept_idx is None:
            return None
        return self.kept_idx[self.cu_kept[r]:self.cu_kept[r + 1]]


def make_tiny(seed, n_res=5, Hq=4, Hkv=2, d=8, L=2, n_req=3, max_len=9, prune=True,
              mask_p=0.5, dtype=np.float64, base=10000.0, max_ctx=7, shared=True):
    rng = np.random.default_rng(seed)
    lengths = rng.integers(1, max_len + 1, size=n_res).astype(np.int32)
    T = int(lengths.sum())
    q = rng.standard_normal((T, Hq, d)).astype(dtype)
    k = rng.standard_normal((T, Hkv, d)).astype(dtype)
    v = rng.standard_normal((T, Hkv, d)).astype(dtype)
    reqs = []
    for b in range(n_req):
        if shared:
            m = int(rng.integers(1, n_res + 1))
            reqs.append(rng.permutation(n_res)[:m])
        else:
            reqs.append(np.array([b % n_res]))
    req_res_off = prefix([len(x) for x in reqs])
    req_res = np.concatenate(reqs).astype(np.int32)
    mask = (rng.random((n_res, L, Hkv)) < mask_p).astype(np.uint8)
    cu_kept = kept_idx = None
    if prune:
        kept = []
        for D in lengths:
            kk = int(rng.integers(1, D + 1))
            idx = np.sort(rng.choice(D, size=kk, replace=False))
            kept.append(idx.astype(np.int32))
        cu_kept = prefix([len(x) for x in kept])
        kept_idx = np.concatenate(kept).astype(np.int32)
    ctx_q, ctx_k, ctx_v, ctx_pos, q_lens = [], [], [], [], []
    for b in range(n_req):
        Tc = int(rng.integers(1, max_ctx + 1))
        Tq = int(rng.integers(1, Tc + 1))
        ctx_q.append(rng.standard_normal((Tc, Hq, d)).astype(dtype))
        ctx_k.append(rng.standard_normal((Tc, Hkv, d)).astype(dtype))
        ctx_v.append(rng.standard_normal((Tc, Hkv, d)).astype(dtype))
        DR = int(lengths[reqs[b]].sum())
        ctx_pos.append((DR + np.arange(Tc)).astype(np.int32))
        q_lens.append(Tq)
    return Tiny(lengths, q, k, v, req_res_off, req_res, mask, cu_kept, kept_idx, ctx_q, ctx_k,
                ctx_v, ctx_pos, np.array(q_lens, np.int32), base)


def head_major(x):
    """[T][H][d] -> [H][T][d] contiguous."""
    return np.ascontiguousarray(np.transpose(x, (1, 0, 2)))
