"""Shapes at the edges of what the library takes, end to end on the GPU
against the CPU oracle: the most images an image table holds, the most KV
heads, one span row, one refreshed row, images of one token and images back
to back without separators."""
import numpy as np
import pytest

from oracle import conduit_oracle as O
from paper_2609_05821_amd import workloads as W
from tests.gpu_helpers import assert_attention, assert_scores, assert_selection, oracle_refresh_rows, to_f64
from tests.test_gpu_end_to_end import run_step

pytestmark = pytest.mark.gpu

CASES = {
    # 256 images (the table's maximum) of 1 to 9 tokens, one separator each
    "max_images": lambda: W.custom(2, 8, 2, 64, 12, 20, [1 + (j * 5) % 9 for j in range(256)], 1, "bf16",
                                   n_relevant=3, seed=21),
    # 256 KV heads (the maximum), one query head each, d = 64
    "max_kv_heads": lambda: W.custom(1, 256, 256, 64, 5, 9, [40, 23], 2, "bf16", seed=22),
    # a span of one token
    "one_span_row": lambda: W.custom(2, 28, 4, 128, 1, 30, [100, 60], 3, "bf16", n_relevant=1, seed=23),
    # images back to back (no separators) and the span right after them
    "no_separators": lambda: W.custom(1, 28, 4, 128, 7, 0, [64, 1, 33, 1, 90], 0, "bf16", seed=24),
    "no_separators_f32": lambda: W.custom(1, 8, 8, 64, 7, 0, [64, 1, 33, 1, 90], 0, "f32", seed=25),
}


@pytest.mark.parametrize("norm", [O.NORM_CAUSAL_ROW, O.NORM_VISUAL_ONLY], ids=["causal", "visual"])
@pytest.mark.parametrize("case", sorted(CASES))
def test_edge_step_matches_oracle(case, norm):
    w = CASES[case]()
    layers_np = [w.layer(li) for li in range(w.n_layers)]
    for k in sorted({1, max(1, w.n_vis // 7)}):  # (run_step copies the stale caches afresh)
        step, layers, idx = run_step(w, layers_np, k, norm=norm)
        ref = O.select([{"q": L["q"], "k": L["k"], "v": L["v"]} for L in layers_np], w.q_pos0, w.img_pos,
                       w.img_off, k, lam=1.0, norm=norm)
        assert_scores(to_f64(step.shat), ref["s_hat"], what=f"s_hat k={k}")
        assert_selection(idx, ref["s_hat"], k)
        P = w.vis_positions()
        for li, L in enumerate(layers_np):
            km, vm, o_ref, lse_ref = oracle_refresh_rows(L["k"], L["v"], P[idx], L["k_star"][idx],
                                                         L["v_star"][idx], L["q_star"][idx], range(k))
            assert_attention(to_f64(step.out[li][:k]), o_ref, w.dtype, what=f"O layer {li} k={k}")
            assert_scores(to_f64(step.lse[li][:k]), lse_ref, what=f"lse layer {li} k={k}")
            np.testing.assert_array_equal(to_f64(layers[li]["k"]), km)
            np.testing.assert_array_equal(to_f64(layers[li]["v"]), vm)
