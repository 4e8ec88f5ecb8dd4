"""Plant plausible mistakes in a copy of the oracle; some pin must catch each.

Every mutation below is a one-line change to the oracle's source of the kind
a reader might make when transcribing the paper (a dropped term, a wrong
index or sign, a transposed operand, another rounding rule).  The mutated
copy is loaded as a separate module; the real oracle is never modified.
"""
import inspect
import types

import pytest

from oracle import conduit_oracle
from tests import oracle_pins

MUTATIONS = {
    "bf16_shift_15": ("return (x.astype(np.uint32) << 16).view(np.float32)",
                      "return (x.astype(np.uint32) << 15).view(np.float32)"),
    "bf16_as_float16": ("return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)",
                        "return x.view(np.float16).astype(np.float64)"),
    "scale_1_over_d": ("scale = 1.0 / np.sqrt(d)", "scale = 1.0 / d", 3),
    "gqa_modulo_mapping": ("kv = h // group", "kv = h % n_kv_heads", 3),
    "causal_excludes_self": ("k_cache[: p + 1, kv, :], scale)\n                alpha = alpha[P_vis]",
                             "k_cache[: p, kv, :], scale)\n                alpha = alpha[P_vis]", 2),
    "visual_column_off_by_one": ("alpha = alpha[P_vis]", "alpha = alpha[P_vis - 1]", 2),
    "head_mean_over_kv_heads": ("a = col_sum / (n_q * n_q_heads)", "a = col_sum / (n_q * n_kv_heads)"),
    "no_query_mean": ("a = col_sum / (n_q * n_q_heads)", "a = col_sum / n_q_heads"),
    "squared_norm": ("return np.sqrt(np.sum(v_rows * v_rows, axis=1))",
                     "return np.sum(v_rows * v_rows, axis=1)"),
    "per_head_norm": ("v_rows = v_cache[P_vis].reshape(len(P_vis), -1)",
                      "v_rows = v_cache[P_vis][:, 0, :]"),
    "rms_without_root": ("        a = np.sqrt(a)\n", "        a = a\n"),
    "rms_not_squared": ("col_sum += alpha if agg == AGG_MEAN else alpha * alpha", "col_sum += alpha"),
    "attention_rule_uses_s": ("base = s if rule == RANK_COMPOSITE else A / len(layers)", "base = s"),
    "attention_rule_no_layer_mean": ("base = s if rule == RANK_COMPOSITE else A / len(layers)",
                                     "base = s if rule == RANK_COMPOSITE else A"),
    "quota_ignores_c": ("w = np.array([np.float32(c[j]) * np.float32(n[j])", "w = np.array([np.float32(n[j])"),
    "quota_no_cap": ("capped = [j for j in range(K) if live[j] and share[j] >= np.float32(n[j])]",
                     "capped = []"),
    "quota_ties_to_upper_image": ("key=lambda j: (-frac[j], j)", "key=lambda j: (-frac[j], -j)"),
    "explicit_bottom_k": ("lo + topk_select(s[lo:lo + int(n[j])], int(quota[j]))",
                          "lo + topk_select(-s[lo:lo + int(n[j])], int(quota[j]))"),
    "text_rows_are_visual": ("return np.flatnonzero(~is_visual).astype(np.int64)",
                             "return np.flatnonzero(is_visual).astype(np.int64)"),
    "text_rows_drop_last": ("is_visual = np.zeros(int(n_ctx), dtype=bool)",
                            "is_visual = np.zeros(int(n_ctx), dtype=bool); is_visual[-1:] = True"),
    "recompute_drops_text": ("np.asarray(sel_pos, np.int64), np.asarray(text_pos, np.int64)])",
                             "np.asarray(sel_pos, np.int64), np.asarray(text_pos, np.int64)[:0]])"),
    "paged_ignores_table": ("out[t] = pages[int(block_table[t // P]), t % P]", "out[t] = pages[t // P, t % P]"),
    "paged_row_from_page_index": ("out[t] = pages[int(block_table[t // P]), t % P]",
                                  "out[t] = pages[int(block_table[t // P]), (t // P) % P]"),
    "iso_per_head_dim": ("dim = z.shape[2] * z.shape[3]", "dim = z.shape[3]"),
    "iso_variance_not_std": ("sigma = kappa * value_norms(v_cache, img_pos, img_off) / np.sqrt(dim)",
                             "sigma = kappa ** 2 * value_norms(v_cache, img_pos, img_off) ** 2 / dim"),
    "residual_keeps_refreshed": ("alpha = np.where(keep, alpha, 0.0)", "alpha = alpha"),
    "residual_drops_kept": ("alpha = np.where(keep, alpha, 0.0)", "alpha = np.where(keep, 0.0, alpha)"),
    "residual_wrong_kv_head": ("y = alpha @ xi[m, :, kv, :]", "y = alpha @ xi[m, :, 0, :]"),
    "residual_not_squared": ("err[m, i, h] = y @ y", "err[m, i, h] = np.sqrt(y @ y)"),
    "residual_visual_renormalised": ("                alpha, _ = attention_row(q[i, h], k_cache[: p + 1, kv, :], scale)\n                alpha = alpha[P_vis]\n            else:\n                alpha, _ = attention_row(q[i, h], k_cache[P_vis, kv, :], scale)\n            alpha = np.where",
                                     "                alpha, _ = attention_row(q[i, h], k_cache[P_vis, kv, :], scale)\n            else:\n                alpha, _ = attention_row(q[i, h], k_cache[P_vis, kv, :], scale)\n            alpha = np.where"),
    "lse_log2": ("return e / total, m + np.log(total)", "return e / total, m + np.log2(total)"),
    "lse_drops_max": ("return e / total, m + np.log(total)", "return e / total, np.log(total)"),
    "layer_sum_not_mean": ("return s / n_layers, A", "return s, A"),
    "mean_product": ("s += np.asarray(a_l, np.float64) * np.asarray(v_l, np.float64)",
                     "s += np.asarray(a_l, np.float64) * np.mean(np.asarray(v_l, np.float64))"),
    "g_no_layer_mean": ("g[j] = np.sum(A[lo:hi]) / (n_layers * (hi - lo))",
                        "g[j] = np.sum(A[lo:hi]) / (hi - lo)"),
    "g_sum_not_mean": ("g[j] = np.sum(A[lo:hi]) / (n_layers * (hi - lo))",
                       "g[j] = np.sum(A[lo:hi]) / n_layers"),
    "lambda_swapped": ("c = (1.0 - lam) + lam * g / g_bar", "c = lam + (1.0 - lam) * g / g_bar"),
    "c_inverted": ("c = (1.0 - lam) + lam * g / g_bar", "c = (1.0 - lam) + lam * g_bar / g"),
    "c_by_token_not_image": ("return s * c[pi]", "return s * c[np.minimum(np.arange(len(s)), len(c) - 1)]"),
    "ties_to_upper_index": ("order = np.lexsort((t, -s_hat))", "order = np.lexsort((-t, -s_hat))"),
    "bottom_k": ("order = np.lexsort((t, -s_hat))", "order = np.lexsort((t, s_hat))"),
    "budget_rounds": ("return (int(r_num) * int(n_vis)) // int(r_den)",
                      "return int(round(r_num * n_vis / r_den))"),
    "budget_float_floor": ("return (int(r_num) * int(n_vis)) // int(r_den)",
                           "return int(math.floor(r_num / r_den * n_vis))"),
    "mask_missing": ("    mask[idx] = 1\n    return idx, P_vis[idx], mask",
                     "    pass\n    return idx, P_vis[idx], mask"),
    "refresh_excludes_self": ("k_merged[: p + 1, kv, :], scale)", "k_merged[: p, kv, :], scale)"),
    "refresh_gqa_modulo": ("            kv = h // group\n            alpha, lse[i, h] = attention_row(q_sel",
                           "            kv = h % n_kv_heads\n            alpha, lse[i, h] = attention_row(q_sel"),
    "refresh_reads_stale_cache": ("out, lse = refresh_attention(q_sel, k_m, v_m, pos",
                                  "out, lse = refresh_attention(q_sel, k_cache, v_cache, pos"),
    "merge_drops_last_row": ("merged[pos] = new_rows", "merged[pos[:-1]] = new_rows[:-1]"),
    "zero_budget_scores_anyway": ("    if k == 0:\n        idx, pos, mask = refresh_mask",
                                  "    if k == -1:\n        idx, pos, mask = refresh_mask"),
    "image_image_positions_shifted": ("positions.append(int(img_pos[j]) + u)",
                                      "positions.append(int(img_pos[j]) + u + 1)"),
}


def _mutant(old, new, count=1):
    src = inspect.getsource(conduit_oracle)
    assert src.count(old) == count, f"mutation anchor must occur {count}x: {old!r}"
    mod = types.ModuleType("oracle_mutant")
    src = src.replace(old, new).replace("from __future__ import annotations\n", "")
    exec(compile("import math\n" + src, "oracle_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name):
    mod = _mutant(*MUTATIONS[name])
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(mod)
        except Exception:  # noqa: BLE001 - any failure counts as caught
            caught.append(pin.__name__)
    assert caught, f"no pin catches mutation {name}"


def test_unmutated_copy_passes_every_pin():
    mod = _mutant("NORM_VISUAL_ONLY = 1", "NORM_VISUAL_ONLY = 1")
    for pin in oracle_pins.ALL_PINS:
        pin(mod)
