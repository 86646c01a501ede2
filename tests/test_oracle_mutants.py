"""Plant plausible mistakes into copies of the oracle (on the CPU) and check
that the pins catch every one of them.

Each mutant is one textual edit of ``oracle/recache_oracle.c``: a sign, a
dropped term, a wrong index, a transposed operand or an off-by-one.  The
mutated copy is compiled into a temporary directory, swapped in for the real
library, and the pin tests run against it; at least one must fail.
"""
import ctypes
import os
import subprocess

import pytest

import oracle
import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "recache_oracle.c")

MUTANTS = {
    "rope_sign": ("y[i] = a * c - b * s;", "y[i] = a * c + b * s;"),
    "rope_second_half_sign": ("y[i + half] = b * c + a * s;", "y[i + half] = b * c - a * s;"),
    "rope_freq_exponent": ("pow(base, -2.0 * (double)i / (double)d)",
                           "pow(base, -1.0 * (double)i / (double)d)"),
    "rope_interleaved_pairs": ("double a = x[i], b = x[i + half];",
                               "double a = x[(2 * i) % d], b = x[(2 * i + 1) % d];"),
    "encode_no_local_reset": ("double p = (double)((pos_base ? pos_base[r] : 0) + (t - cu_len[r]));",
                              "double p = (double)((pos_base ? pos_base[r] : 0) + t);"),
    "encode_drops_diagonal": ("for (int u = 0; u <= j; ++u) {",
                              "for (int u = 0; u <= j - (j > 0); ++u) {"),
    "scale_dropped_encode": ("z[prefix_len + u] = scale * dot;",
                             "z[prefix_len + u] = dot;"),
    "prefix_scale_dropped": ("z[u] = scale * dot;\n            }\n            for (int u = 0; u <= j; ++u) {",
                             "z[u] = dot;\n            }\n            for (int u = 0; u <= j; ++u) {"),
    "prefix_not_visible": ("z[u] = scale * dot;\n            }\n            for (int u = 0; u <= j; ++u) {",
                           "z[u] = -INFINITY;\n            }\n            for (int u = 0; u <= j; ++u) {"),
    "prefix_v_row_shifted": ("return x->vc + ((size_t)x->g * x->T + x->row0 + (u - x->p_len)) * x->d;",
                             "return x->vc + ((size_t)x->g * x->T + x->row0 + u) * x->d;"),
    "scale_dropped_attend": ("z[u] = scale * dot;\n            }\n            struct att_vctx",
                             "z[u] = dot;\n            }\n            struct att_vctx"),
    "gqa_modulo": ("int s = (int)(sh / Hq), h = (int)(sh % Hq), g = h / ratio;",
                   "int s = (int)(sh / Hq), h = (int)(sh % Hq), g = h % Hkv;"),
    "lse_without_max": ("return m + log(denom);", "return log(denom);"),
    "causal_top_left": ("int last_ctx = Tc - Tq + i;", "int last_ctx = i;"),
    "mask_index_transposed": ("if (!mask[((size_t)r * n_layers + layer) * Hkv + g]) continue;",
                              "if (!mask[((size_t)r * Hkv + g) * n_layers + layer]) continue;"),
    "kept_ignored": ("key_row[n++] = (int64_t)cu_rows[r] + kept_idx[t];",
                     "key_row[n++] = (int64_t)cu_rows[r] + (t - cu_kept[r]);"),
    "prune_wrong_source": ("size_t src = ((size_t)g * T + cu_len[r] + kept_idx[j]) * row;",
                           "size_t src = ((size_t)g * T + cu_len[r] + j - cu_kept[r]) * row;"),
    "routes_count_resources": ("tokens += cu_kept[r + 1] - cu_kept[r];", "tokens += 1;"),
    "routes_skip_mask": ("if (mask[((size_t)r * L + l) * G + g]) {", "if (1) {"),
    "vcache_from_k": ("v_cache[((size_t)g * T + t) * d + e] = widen(v, dtype,",
                      "v_cache[((size_t)g * T + t) * d + e] = widen(k, dtype,"),
    "softmax_no_normalise": ("for (int e = 0; e < d; ++e) out[e] /= denom;", ""),
    "round_truncates": ("return ldexp(rint(ldexp(m, 8)), e - 8);",
                        "return ldexp(trunc(ldexp(m, 8)), e - 8);"),
    "round_keeps_9_bits": ("return ldexp(rint(ldexp(m, 8)), e - 8);",
                           "return ldexp(rint(ldexp(m, 9)), e - 9);"),
    "encode_query_not_rounded": ("for (int e = 0; e < d; ++e) qr[e] = round_to(qr[e], rot_dtype);",
                                 ""),
    "rope_not_rounded": ("for (int e = 0; e < d; ++e) yr[e] = round_to(yr[e], rot_dtype);", ""),
    "store_offsets_group_major": ("store_off[l * stride + (size_t)r * G + g] = (int32_t)run;",
                                  "store_off[l * stride + (size_t)g * n_res + r] = (int32_t)run;"),
    "store_offsets_count_routes": ("if (mask[((size_t)r * L + l) * G + g]) run += cu_kept[r + 1] - cu_kept[r];",
                                   "if (mask[((size_t)r * L + l) * G + g]) run += 1;"),
    "store_ignores_mask": ("if (!mask[((size_t)r * L + layer) * Hkv + g]) continue;", ""),
    "store_wrong_head": ("const size_t from = ((size_t)g * T + cu_len[r] + kept_idx[j]) * row;",
                         "const size_t from = ((size_t)0 * T + cu_len[r] + kept_idx[j]) * row;"),
    "attend_store_group_major": ("key_row[n++] = (int64_t)store_off[(size_t)r * Hkv + g] + t;",
                                 "key_row[n++] = (int64_t)store_off[(size_t)g * n_res + r] + t;"),
}

PINS = [
    pins.test_round_to_bf16_tie_cases_and_bit_level_rne,
    pins.test_rope_rounds_to_storage_precision,
    pins.test_encode_bf16_storage_precision_matches_bruteforce,
    pins.test_rope_d2_closed_form,
    pins.test_rope_matches_complex_form_and_identities,
    pins.test_encode_single_resource_is_textbook_causal_attention,
    pins.test_encode_blockdiag_matches_bruteforce_and_lse,
    pins.test_encode_first_token_is_its_value_row,
    pins.test_encode_zero_queries_give_running_mean,
    lambda: pins.test_encode_with_prefix_is_causal_attention_over_prefix_then_resource(False),
    lambda: pins.test_encode_with_prefix_is_causal_attention_over_prefix_then_resource(True),
    lambda: pins.test_attend_matches_bruteforce_final_mask(3),
    lambda: pins.test_attend_matches_bruteforce_final_mask(4),
    pins.test_attend_all_ones_mask_is_causal_over_concatenation,
    pins.test_attend_all_zeros_mask_is_context_only,
    pins.test_attend_decode_row_sees_every_context_row,
    pins.test_prune_matches_fancy_indexing_and_extremes,
    pins.test_routes_match_python_loops,
    pins.test_store_offsets_closed_forms,
    pins.test_store_routes_places_rows_where_offsets_say,
    lambda: pins.test_attend_over_store_equals_attend_over_pruned_cache(44),
    pins.test_store_size_factorises_for_a_shared_route_set,
]


@pytest.fixture(scope="module")
def source():
    oracle._load()
    with open(SRC) as f:
        return f.read()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, source, tmp_path, monkeypatch):
    old, new = MUTANTS[name]
    assert source.count(old) == 1, "mutation target not found exactly once: %r" % old
    path = tmp_path / ("m_%s.c" % name)
    path.write_text(source.replace(old, new))
    so = tmp_path / ("m_%s.so" % name)
    subprocess.check_call(["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-w",
                           "-o", str(so), str(path), "-lm"])
    monkeypatch.setattr(oracle, "_lib", ctypes.CDLL(str(so)))
    caught = []
    for pin in PINS:
        try:
            pin()
        except (AssertionError, ValueError):
            caught.append(getattr(pin, "__name__", "lambda"))
    assert caught, "mutant %s survived every pin" % name


# ------------------------------------------------------------------ route-budget oracle

import test_route_budget as budget_pins  # noqa: E402

BUDGET_SRC = os.path.join(os.path.dirname(oracle.__file__), "budget.py")

BUDGET_MUTANTS = {
    "negative_contributions_kept": ("pos = np.where(s > 0, s, 0.0)", "pos = s"),
    "ties_to_higher_index": ("key=lambda i: (-w[i], i)", "key=lambda i: (-w[i], -i)"),
    "smallest_weights_kept": ("key=lambda i: (-w[i], i)", "key=lambda i: (w[i], i)"),
    "sparsity_additive": ("1.0 - (k_layers * k_groups) / (L * G)",
                          "1.0 - (k_layers + k_groups) / (L + G)"),
    "coverage_of_everything": ("float(sum(wl[i] for i in ls))", "float(sum(wl))"),
    "budget_off_by_one": ("return sorted(order[:k])", "return sorted(order[:k + 1])"),
    "unnormalised": ("return pos / total", "return pos"),
}

BUDGET_PINS = [
    lambda: budget_pins.test_oracle_reproduces_printed_budget("Qwen3-4B"),
    lambda: budget_pins.test_oracle_reproduces_printed_budget("Qwen3-1.7B"),
    budget_pins.test_qwen3_4b_route_set,
    budget_pins.test_oracle_weights_closed_forms,
]


@pytest.mark.parametrize("name", sorted(BUDGET_MUTANTS))
def test_budget_pins_catch_mutant(name, monkeypatch):
    import types

    old, new = BUDGET_MUTANTS[name]
    src = open(BUDGET_SRC).read()
    assert src.count(old) == 1, "mutation target not found exactly once: %r" % old
    mod = types.ModuleType("budget_mutant")
    exec(compile(src.replace(old, new), "budget_mutant.py", "exec"), mod.__dict__)
    monkeypatch.setattr(budget_pins, "budget", mod)
    caught = []
    for pin in BUDGET_PINS:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            caught.append(getattr(pin, "__name__", "lambda"))
    assert caught, "mutant %s survived every pin" % name
