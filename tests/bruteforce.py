"""Brute-force checker for the oracle: the paper's final mask as an explicit
dense N x N boolean matrix (ReCache, Fig. 2 "Final ReCache Mask"), applied
to one request laid out as one sequence [R_1 ... R_n, context].

It is written independently of ``oracle/``: RoPE is applied in complex form
((x_i + i x_{i+d/2}) * exp(i p theta_i)), the mask is built entry by entry
from its definition, and attention is a dense masked softmax over all N keys.
Only tiny inputs are meant here.
"""
from __future__ import annotations

import numpy as np


def rope_complex(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """x[N][H][d] (float64) rotated at positions pos[N], complex formulation."""
    d = x.shape[-1]
    half = d // 2
    inv = base ** (-2.0 * np.arange(half) / d)
    z = x[..., :half] + 1j * x[..., half:]
    z = z * np.exp(1j * np.outer(pos, inv))[:, None, :]
    return np.concatenate([z.real, z.imag], axis=-1)


def final_mask(lengths, kept, route_bits, n_ctx: int) -> np.ndarray:
    """Dense boolean mask M[a][c] over the sequence [R_1..R_n, ctx].

    M[a][c] is set iff (i) a and c lie in the same resource and c <= a, or
    (ii) both are context tokens and c <= a, or (iii) a is a context token, c
    lies in resource r, r's route bit is set for this (layer, group), and
    c's local index is in r's kept list (all indices if kept[r] is None).
    """
    seg, loc = [], []
    for r, D in enumerate(lengths):
        seg += [r] * int(D)
        loc += list(range(int(D)))
    seg += [-1] * n_ctx
    loc += list(range(n_ctx))
    N = len(seg)
    M = np.zeros((N, N), bool)
    for a in range(N):
        for c in range(N):
            if seg[a] >= 0:
                M[a, c] = seg[c] == seg[a] and c <= a
            elif seg[c] < 0:
                M[a, c] = c <= a
            else:
                r = seg[c]
                visible = bool(route_bits[r])
                in_kept = kept[r] is None or loc[c] in set(int(x) for x in kept[r])
                M[a, c] = visible and in_kept
    return M


def dense_masked_attention(q, k, v, M, scale):
    """q[N][d], k[N][d], v[N][d], M[N][N] -> (out[N][d], lse[N]) (float64).
    Masked logits are -inf (left out of the normaliser)."""
    s = scale * (q @ k.T)
    s = np.where(M, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    w = np.exp(s - m)
    den = w.sum(axis=1, keepdims=True)
    return (w @ v) / den, (m + np.log(den))[:, 0]


def rne_bits(x: np.ndarray, mant_bits: int) -> np.ndarray:
    """Round float64 values to nearest-even with mant_bits explicit mantissa
    bits (7 for bf16, 23 for fp32), by integer arithmetic on the IEEE bits."""
    x = np.ascontiguousarray(np.asarray(x, np.float64))
    b = x.view(np.uint64).copy()
    drop = np.uint64(52 - mant_bits)
    lsb = (b >> drop) & np.uint64(1)
    b = b + ((np.uint64(1) << (drop - np.uint64(1))) - np.uint64(1)) + lsb
    b &= ~((np.uint64(1) << drop) - np.uint64(1))
    return b.view(np.float64)


def request(res_q, res_k, res_v, ctx_q, ctx_k, ctx_v, ctx_pos, kept, route_bits_lg, base,
            scale, n_q, round_rot=None):
    """One request, one layer.

    res_q/res_k/res_v: lists (request order) of raw [D][Hq|Hkv][d] arrays;
    ctx_*: raw [Tc][H][d]; ctx_pos[Tc]: context positions; kept: list of index
    arrays or None; route_bits_lg[r][g]: route bit of resource r for KV group g
    in this layer; n_q: the last n_q context tokens are the queries.

    Returns (res_out[D_R][Hq][d], ctx_out[n_q][Hq][d], res_lse[D_R][Hq],
    ctx_lse[n_q][Hq], mask_popcount_per_group[G]).  round_rot, if given, is
    applied to the rotated queries and keys.
    """
    lengths = [a.shape[0] for a in res_q]
    Tc = ctx_q.shape[0]
    Hq, d = ctx_q.shape[1], ctx_q.shape[2]
    Hkv = ctx_k.shape[1]
    ratio = Hq // Hkv
    pos = np.concatenate([np.arange(D) for D in lengths] + [np.asarray(ctx_pos)]).astype(np.float64)
    Q = np.concatenate(list(res_q) + [ctx_q], axis=0).astype(np.float64)
    K = np.concatenate(list(res_k) + [ctx_k], axis=0).astype(np.float64)
    V = np.concatenate(list(res_v) + [ctx_v], axis=0).astype(np.float64)
    Qr, Kr = rope_complex(Q, pos, base), rope_complex(K, pos, base)
    if round_rot is not None:  # rotated Q / K held at a storage precision
        Qr, Kr = round_rot(Qr), round_rot(Kr)
    N, DR = Q.shape[0], sum(lengths)
    out = np.zeros((N, Hq, d))
    lse = np.zeros((N, Hq))
    pop = []
    for g in range(Hkv):
        bits = [route_bits_lg[r][g] for r in range(len(lengths))]
        M = final_mask(lengths, kept, bits, Tc)
        qrows = np.r_[np.arange(DR), np.arange(N - n_q, N)]
        pop.append(int(M[qrows].sum()))
        for h in range(g * ratio, (g + 1) * ratio):
            o, l = dense_masked_attention(Qr[:, h], Kr[:, g], V[:, g], M, scale)
            out[:, h], lse[:, h] = o, l
    return out[:DR], out[N - n_q:], lse[:DR], lse[N - n_q:], pop
