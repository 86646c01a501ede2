"""Structural budget selection (Sec. 3, "Structural Pruning"): the oracle
against the paper's printed contribution weights, coverages and sparsity
(tests/golden/structural_budget_weights.json, from the appendix table of
contribution weights and the table of selected budgets), and the library's
host call against the oracle."""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

from oracle import budget
from paper_2608_19662_amd import recache as rc
from paper_2608_19662_amd.workloads import (OMEGA_20_3_QWEN3_4B_GROUPS, OMEGA_20_3_QWEN3_4B_LAYERS,
                                            omega_star_mask)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "structural_budget_weights.json")
MODELS = ("Qwen3-4B", "Qwen3-1.7B")


def load(model):
    m = json.load(open(GOLDEN))["models"][model]
    # printed weights by unit index (the paper numbers units from 1)
    wl = np.zeros(m["n_layers"])
    wg = np.zeros(m["n_groups"])
    for row in m["layers"]:
        wl[row["unit"] - 1] = row["w_percent"]
    for row in m["groups"]:
        wg[row["unit"] - 1] = row["w_percent"]
    return m, wl, wg


@pytest.mark.parametrize("model", MODELS)
def test_printed_coverage_column_is_the_running_sum_of_printed_weights(model):
    """CC at rank k is the summed weight of the top k units (to print precision)."""
    m, _, _ = load(model)
    for kind in ("layers", "groups"):
        rows = sorted(m[kind], key=lambda r: r["rank"])
        run = np.cumsum([r["w_percent"] for r in rows])
        cc = np.array([r["cc_percent"] for r in rows])
        # 0.05 from rounding CC, plus up to 0.005 per summed weight
        assert np.all(np.abs(run - cc) <= 0.05 + 0.005 * np.arange(1, len(rows) + 1) + 1e-9)


@pytest.mark.parametrize("model", MODELS)
def test_oracle_reproduces_printed_budget(model):
    """Feeding the printed weights back as contributions reproduces the
    printed selection, coverage and sparsity."""
    m, wl, wg = load(model)
    sel = budget.select_routes(wl, wg, m["k_layers"], m["k_groups"])
    top_l = sorted(r["unit"] - 1 for r in m["layers"] if r["rank"] <= m["k_layers"])
    top_g = sorted(r["unit"] - 1 for r in m["groups"] if r["rank"] <= m["k_groups"])
    assert sel["layers"] == top_l and sel["groups"] == top_g
    assert abs(100 * sel["cc_layer"] - m["cc_layers_percent"]) <= 0.1
    assert abs(100 * sel["cc_group"] - m["cc_groups_percent"]) <= 0.1
    assert round(100 * sel["rho"], 1) == m["rho_percent"]
    assert sel["mask"].sum() == m["k_layers"] * m["k_groups"]
    # ranking agrees with the printed ranks wherever the printed weights differ
    w = sel["w_layer"]
    rows = sorted(m["layers"], key=lambda r: r["rank"])
    for a, b in zip(rows, rows[1:]):
        if a["w_percent"] > b["w_percent"]:
            assert w[a["unit"] - 1] > w[b["unit"] - 1]


def test_qwen3_4b_route_set():
    """Omega*_{20,3} of the primary backbone, as 0-based (layer, group) sets,
    and the constant the workloads carry for it."""
    m, wl, wg = load("Qwen3-4B")
    sel = budget.select_routes(wl, wg, 20, 3)
    assert sel["layers"] == [13, 15, 16, 17, 18, 19, 20, 21, 22, 23, 24, 26, 27, 29, 30, 31, 32,
                             33, 34, 35]
    assert sel["groups"] == [2, 3, 5]
    assert list(OMEGA_20_3_QWEN3_4B_LAYERS) == sel["layers"]
    assert list(OMEGA_20_3_QWEN3_4B_GROUPS) == sel["groups"]
    mask = omega_star_mask(4, 36, 8, OMEGA_20_3_QWEN3_4B_LAYERS, OMEGA_20_3_QWEN3_4B_GROUPS)
    assert np.array_equal(mask[2], sel["mask"])


def test_oracle_weights_closed_forms():
    """Negative contributions weigh zero; weights sum to one; ties keep the
    lower index; the budget extremes give empty and full route sets."""
    w = budget.contribution_weights([2.0, -1.0, 0.0, 6.0])
    assert np.allclose(w, [0.25, 0.0, 0.0, 0.75])
    assert budget.top_k([0.5, 0.25, 0.25], 2) == [0, 1]
    full = budget.select_routes([1, 2, 3], [1, 1], 3, 2)
    assert full["mask"].all() and full["rho"] == 0.0 and full["cc_layer"] == 1.0
    empty = budget.select_routes([1, 2, 3], [1, 1], 0, 2)
    assert not empty["mask"].any() and empty["rho"] == 1.0 and empty["cc_layer"] == 0.0
    with pytest.raises(ValueError):
        budget.contribution_weights([-1.0, 0.0])


@pytest.mark.parametrize("model", MODELS)
def test_library_matches_oracle(model):
    m, wl, wg = load(model)
    rng = np.random.default_rng(3)
    for sl, sg in ((wl, wg), (rng.normal(size=len(wl)), rng.normal(size=len(wg)))):
        for kl, kg in ((m["k_layers"], m["k_groups"]), (0, 1), (len(wl), len(wg)), (7, 5)):
            ref = budget.select_routes(sl, sg, kl, kg)
            got = rc.select_routes(sl, sg, kl, kg)
            assert np.array_equal(got["mask"], ref["mask"])
            assert np.allclose(got["w_layer"], ref["w_layer"], rtol=0, atol=1e-15)
            assert np.allclose(got["w_group"], ref["w_group"], rtol=0, atol=1e-15)
            assert got["rho"] == ref["rho"]
            assert abs(got["cc_layer"] - ref["cc_layer"]) < 1e-14
            assert abs(got["cc_group"] - ref["cc_group"]) < 1e-14


def test_library_rejects_bad_budgets():
    for args in (([1.0], [1.0], 2, 1), ([1.0], [1.0], 1, -1), ([-1.0], [1.0], 1, 1),
                 ([float("nan")], [1.0], 1, 1), ([1.0], [0.0, -2.0], 1, 1)):
        with pytest.raises(rc.RecacheError) as e:
            rc.select_routes(*args)
        assert e.value.code == rc.EINVAL


def test_library_writes_nothing_on_error():
    """Valid layer contributions, invalid group ones: every output keeps its
    previous contents."""
    import ctypes

    L, G = 3, 2
    sl = np.array([1.0, 2.0, 3.0])
    sg = np.array([-1.0, 0.0])
    mask = np.full(L * G, 7, np.uint8)
    wl, wg = np.full(L, -5.0), np.full(G, -5.0)
    out = np.full(3, -5.0)
    p = lambda a: a.ctypes.data
    code = rc.lib().recache_select_routes(L, G, p(sl), p(sg), 1, 1, p(mask), p(wl), p(wg), p(out),
                                          ctypes.c_void_p(p(out) + 8), ctypes.c_void_p(p(out) + 16))
    assert code == rc.EINVAL
    assert (mask == 7).all() and (wl == -5.0).all() and (wg == -5.0).all() and (out == -5.0).all()
