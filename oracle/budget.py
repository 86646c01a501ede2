"""Structural budget selection, written out from the paper (oracle).

TEST INFRASTRUCTURE ONLY: used by the test suite to check the library's
route-selection call; nothing in the product imports it.

ReCache, Sec. 3 "Structural Pruning": each layer (or KV head group) i has a
leave-one-in contribution s_i; its contribution weight is
w_i = max(s_i, 0) / sum_j max(s_j, 0); the retained units are the top K by w
(L* for layers, G* for groups) and the route set is Omega* = L* x G*.
Sec. "Structural Budget Analysis": structural sparsity
rho = 1 - |L*| |G*| / (L G), and the contribution coverage CC of a budget is
the summed weight of the retained units.  Units of equal weight are taken in
increasing index order (the paper lists its zero-weight units that way).
"""
from __future__ import annotations

import numpy as np


def contribution_weights(s) -> np.ndarray:
    s = np.asarray(s, dtype=np.float64)
    pos = np.where(s > 0, s, 0.0)
    total = pos.sum()
    if not total > 0:
        raise ValueError("no unit has a positive contribution")
    return pos / total


def top_k(w, k: int) -> list[int]:
    order = sorted(range(len(w)), key=lambda i: (-w[i], i))
    return sorted(order[:k])


def select_routes(s_layer, s_group, k_layers: int, k_groups: int) -> dict:
    wl, wg = contribution_weights(s_layer), contribution_weights(s_group)
    L, G = len(wl), len(wg)
    if not (0 <= k_layers <= L and 0 <= k_groups <= G):
        raise ValueError("budget outside the unit counts")
    ls, gs = top_k(wl, k_layers), top_k(wg, k_groups)
    mask = np.zeros((L, G), np.uint8)
    for l in ls:
        for g in gs:
            mask[l, g] = 1
    return {"w_layer": wl, "w_group": wg, "layers": ls, "groups": gs, "mask": mask,
            "rho": 1.0 - (k_layers * k_groups) / (L * G),
            "cc_layer": float(sum(wl[i] for i in ls)), "cc_group": float(sum(wg[i] for i in gs))}
