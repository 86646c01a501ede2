"""Seeded synthetic inputs for resource-wise attention.

This module draws inputs only: resource lengths, route masks, kept-token
lists and N(0, 1) tensors.  It holds none of the method's arithmetic, so the
GPU path and the CPU oracle can both consume what it produces.

Structure (lengths, masks, kept lists) comes from ``numpy.random.default_rng``
(PCG64) seeded with the workload's seed, drawn in this order: lengths, route
masks, kept lists.  Tensors come from a ``torch.Generator`` on the target
device seeded with ``seed * 1000 + tensor_id``, drawn in float32 and rounded
to the storage dtype.

The workloads stand in for the paper's tool/skill-schema datasets (ReCache,
Sec. 4.1), which are not available: shapes follow the Qwen3 attention layout
(Sec. 4.3; 32 query heads over 8 KV groups, head_dim 128, 36 layers), the
resource-length ranges cover the paper's D_R buckets (Sec. 6, efficiency
scaling), and the route / kept fractions sit near the paper's budgets
(Sec. 5; 20 of 36 layers x 3 of 8 groups, about a third of tokens kept).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

try:  # torch is only needed for tensor draws
    import torch
except ImportError:  # pragma: no cover
    torch = None


# ---------------------------------------------------------------- structure

def draw_lengths(rng: np.random.Generator, n: int, lo: int, hi: int) -> np.ndarray:
    """n lengths uniform on the integers lo..hi inclusive."""
    return rng.integers(lo, hi + 1, size=n).astype(np.int32)


def prefix(lengths) -> np.ndarray:
    """Exclusive prefix sums [0, l0, l0+l1, ...] as int32 (the packing offsets)."""
    out = np.zeros(len(lengths) + 1, np.int64)
    np.cumsum(np.asarray(lengths, np.int64), out=out[1:])
    if out[-1] > np.iinfo(np.int32).max:
        raise ValueError("packed length overflows int32")
    return out.astype(np.int32)


def draw_route_mask_exact(rng, n_res: int, L: int, G: int, frac: float) -> np.ndarray:
    """Each resource gets exactly round(frac * L * G) visible (layer, group) routes."""
    per = int(round(frac * L * G))
    m = np.zeros((n_res, L * G), np.uint8)
    for r in range(n_res):
        m[r, rng.choice(L * G, size=per, replace=False)] = 1
    return m.reshape(n_res, L, G)


def draw_route_mask_bernoulli(rng, n_res: int, L: int, G: int, p: float) -> np.ndarray:
    """Independent Bernoulli(p) route bit per (resource, layer, group)."""
    return (rng.random((n_res, L, G)) < p).astype(np.uint8)


# Omega*_{20,3} of Qwen3-4B, the paper's primary backbone (36 layers, 8 KV
# groups): the 20 layers and 3 groups of largest contribution weight in its
# appendix table of per-layer and per-group weights, 0-based.  Qwen3-4B has
# the 36-layer, 32/8-head, d-128 attention shape of the decode workload.
OMEGA_20_3_QWEN3_4B_LAYERS = (13, 15, 16, 17, 18, 19, 20, 21, 22, 23, 24, 26, 27, 29, 30, 31, 32,
                              33, 34, 35)
OMEGA_20_3_QWEN3_4B_GROUPS = (2, 3, 5)


def omega_star_mask(n_res: int, L: int, G: int, layers, groups) -> np.ndarray:
    """The same route set L* x G* for every resource, as a [n_res][L][G] mask."""
    m = np.zeros((n_res, L, G), np.uint8)
    m[:, np.asarray(layers)[:, None], np.asarray(groups)[None, :]] = 1
    return m


def draw_kept(rng, lengths, frac: float):
    """Kept-token lists: the final token of every resource, plus a uniform
    sample without replacement of the others, k_i = max(1, floor(frac*D_i + 0.5))
    tokens in total, sorted ascending.  Returns (cu_kept, kept_idx)."""
    kept = []
    for D in np.asarray(lengths):
        k = max(1, int(np.floor(frac * D + 0.5)))
        others = rng.choice(int(D) - 1, size=k - 1, replace=False) if k > 1 else np.zeros(0, int)
        idx = np.sort(np.concatenate([others, [int(D) - 1]])).astype(np.int32)
        kept.append(idx)
    cu_kept = prefix([len(k) for k in kept])
    return cu_kept, np.concatenate(kept).astype(np.int32)


# ---------------------------------------------------------------- tensors

def normal(shape, dtype, seed: int, tensor_id: int, device="cpu"):
    """N(0, 1) tensor drawn in float32 from a seeded generator on ``device``,
    then rounded (RNE) to ``dtype``."""
    if torch is None:  # pragma: no cover
        raise RuntimeError("torch is required for tensor draws")
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1000 + int(tensor_id))
    t = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
    return t if dtype == torch.float32 else t.to(dtype)


def torch_dtype(name: str):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


# ---------------------------------------------------------------- workloads

@dataclass
class EncodeWorkload:
    """One layer of packed resource encoding."""
    seed: int
    lengths: np.ndarray
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str
    rope_base: float

    @property
    def cu_len(self):
        return prefix(self.lengths)

    @property
    def total(self):
        return int(np.sum(self.lengths, dtype=np.int64))

    def tensors(self, device="cpu", ids=(1, 2, 3)):
        """(q[T][Hq][d], k[T][Hkv][d], v[T][Hkv][d])"""
        T, dt = self.total, torch_dtype(self.dtype)
        q = normal((T, self.n_q_heads, self.head_dim), dt, self.seed, ids[0], device)
        k = normal((T, self.n_kv_heads, self.head_dim), dt, self.seed, ids[1], device)
        v = normal((T, self.n_kv_heads, self.head_dim), dt, self.seed, ids[2], device)
        return q, k, v

    def pairs_per_head(self) -> int:
        """Unmasked (query, key) pairs per head: sum D_i (D_i + 1) / 2."""
        L = self.lengths.astype(np.int64)
        return int(np.sum(L * (L + 1) // 2))


@dataclass
class AttendWorkload:
    """Requests of conversation tokens over cached resources, n_layers layers.

    Resource r owns rows [cu_len[r], cu_len[r+1]) of the unpruned caches and
    rows [cu_kept[r], cu_kept[r+1]) of the compacted ones.  Request b lists
    resources req_res[req_res_off[b]:req_res_off[b+1]] (request order).
    """
    seed: int
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str
    lengths: np.ndarray
    req_res_off: np.ndarray
    req_res: np.ndarray
    q_lens: np.ndarray
    ctx_lens: np.ndarray
    mask: np.ndarray                 # [n_res][L][G] uint8
    cu_kept: np.ndarray | None = None
    kept_idx: np.ndarray | None = None
    extra: dict = field(default_factory=dict)

    @property
    def n_req(self):
        return len(self.q_lens)

    @property
    def n_res(self):
        return len(self.lengths)

    @property
    def cu_len(self):
        return prefix(self.lengths)

    @property
    def cu_q(self):
        return prefix(self.q_lens)

    @property
    def cu_ctx(self):
        return prefix(self.ctx_lens)

    @property
    def kept_lengths(self):
        if self.cu_kept is None:
            return self.lengths
        return np.diff(self.cu_kept).astype(np.int32)

    @property
    def cu_rows(self):
        """Offsets of the compacted (kept) rows; equal to cu_len without pruning."""
        return self.cu_len if self.cu_kept is None else self.cu_kept

    def layer_tensors(self, layer: int, device="cpu", compacted=True):
        """Per-layer tensors: q[sum Tq][Hq][d], ctx_k/ctx_v[Hkv][sum Tc][d],
        res_k/res_v[Hkv][R][d] where R is the kept total (compacted=True) or
        the unpruned total."""
        dt = torch_dtype(self.dtype)
        base = 10 + 10 * layer
        Hq, Hkv, d = self.n_q_heads, self.n_kv_heads, self.head_dim
        R = int(self.cu_rows[-1]) if compacted else int(self.cu_len[-1])
        q = normal((int(self.cu_q[-1]), Hq, d), dt, self.seed, base + 0, device)
        ck = normal((Hkv, int(self.cu_ctx[-1]), d), dt, self.seed, base + 1, device)
        cv = normal((Hkv, int(self.cu_ctx[-1]), d), dt, self.seed, base + 2, device)
        rk = normal((Hkv, R, d), dt, self.seed, base + 3, device)
        rv = normal((Hkv, R, d), dt, self.seed, base + 4, device)
        return q, ck, cv, rk, rv


def encode_config1_like(seed=1):
    return EncodeWorkload(seed=seed, lengths=np.array([37, 64, 91, 120], np.int32),
                          n_q_heads=8, n_kv_heads=2, head_dim=64, dtype="f32", rope_base=1e4)


def config(k: int) -> dict:
    """The five synthetic workloads, by number.

    1: tiny fp32 layer -- 8/2 heads, d 64, resources 37/64/91/120 (local RoPE,
       base 1e4), one request with 48 context tokens (positions 312 + j),
       Bernoulli(0.5) route per (resource, KV head), no pruning.
    2: encode, one layer, 32/8 heads, d 128, bf16, 16 resources of U[200,1500],
       RoPE base 1e6.
    3: prefill, 36 layers, 32/8, d 128, bf16, 8 requests x (8 resources of
       U[300,1200] + 2048 context tokens causal), all routes, no pruning.
    4: as 3 with seed 4, exactly 25% of the 288 routes of every resource
       visible and 30% of each resource's tokens kept (suffix included).
    5: decode, 36 layers, 32/8, d 128, bf16, 64 requests x 1 new token, each
       over 32 distinct resources of U[200,2000] (30% kept, 25% of routes)
       plus 4096 conversation tokens that include the new one.
    """
    if k == 1:
        enc = encode_config1_like(seed=1)
        rng = np.random.default_rng(1)
        mask = draw_route_mask_bernoulli(rng, 4, 1, 2, 0.5)
        att = AttendWorkload(
            seed=1, n_layers=1, n_q_heads=8, n_kv_heads=2, head_dim=64, dtype="f32",
            lengths=enc.lengths, req_res_off=np.array([0, 4], np.int32),
            req_res=np.arange(4, dtype=np.int32), q_lens=np.array([48], np.int32),
            ctx_lens=np.array([48], np.int32), mask=mask,
            extra={"ctx_pos0": int(enc.total), "rope_base": 1e4})
        return {"encode": enc, "attend": att}
    if k == 2:
        rng = np.random.default_rng(2)
        enc = EncodeWorkload(seed=2, lengths=draw_lengths(rng, 16, 200, 1500), n_q_heads=32,
                             n_kv_heads=8, head_dim=128, dtype="bf16", rope_base=1e6)
        return {"encode": enc}
    if k in (3, 4):
        rng = np.random.default_rng(k)
        B, per, L, G = 8, 8, 36, 8
        lengths = draw_lengths(rng, B * per, 300, 1200)
        if k == 3:
            mask = np.ones((B * per, L, G), np.uint8)
            cu_kept = kept_idx = None
        else:
            mask = draw_route_mask_exact(rng, B * per, L, G, 0.25)
            cu_kept, kept_idx = draw_kept(rng, lengths, 0.30)
        att = AttendWorkload(
            seed=k, n_layers=L, n_q_heads=32, n_kv_heads=G, head_dim=128, dtype="bf16",
            lengths=lengths, req_res_off=prefix([per] * B), req_res=np.arange(B * per, dtype=np.int32),
            q_lens=np.full(B, 2048, np.int32), ctx_lens=np.full(B, 2048, np.int32), mask=mask,
            cu_kept=cu_kept, kept_idx=kept_idx)
        return {"attend": att}
    if k == 5:
        rng = np.random.default_rng(5)
        B, per, L, G = 64, 32, 36, 8
        lengths = draw_lengths(rng, B * per, 200, 2000)
        mask = draw_route_mask_exact(rng, B * per, L, G, 0.25)
        cu_kept, kept_idx = draw_kept(rng, lengths, 0.30)
        att = AttendWorkload(
            seed=5, n_layers=L, n_q_heads=32, n_kv_heads=G, head_dim=128, dtype="bf16",
            lengths=lengths, req_res_off=prefix([per] * B), req_res=np.arange(B * per, dtype=np.int32),
            q_lens=np.ones(B, np.int32), ctx_lens=np.full(B, 4096, np.int32), mask=mask,
            cu_kept=cu_kept, kept_idx=kept_idx)
        return {"attend": att}
    raise ValueError("no workload %r" % k)
