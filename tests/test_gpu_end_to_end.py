"""The whole refresh step on the GPU (score every layer, select once, merge and
refresh every layer) against the CPU oracle, plus the paper's anchors."""
import numpy as np
import pytest
import torch

from oracle import conduit_oracle as O
from paper_2609_05821_amd import api, workloads as W
from tests.gpu_helpers import (DEV, assert_attention, assert_scores, assert_selection, bits,
                               oracle_refresh_rows, to_dev, to_f64)

pytestmark = pytest.mark.gpu


def run_step(w, layers_np, k, lam=1.0, norm=O.NORM_CAUSAL_ROW):
    layers = [{"k": to_dev(L["k"]), "v": to_dev(L["v"]), "q": to_dev(L["q"])} for L in layers_np]
    img = api.ImageTable(w.img_pos, w.img_off)
    step = api.RefreshStep(layers, w.n_q_heads, w.q_pos0, img, k, lam=lam, norm=norm, device=DEV)
    step.score_and_select()
    torch.cuda.synchronize()
    idx = step.idx[:k].cpu().numpy()
    fresh = [{"k_new": to_dev(L["k_star"][idx]), "v_new": to_dev(L["v_star"][idx]),
              "q_sel": to_dev(L["q_star"][idx])} for L in layers_np]
    step.refresh(fresh)
    torch.cuda.synchronize()
    return step, layers, idx


@pytest.mark.parametrize("cfg,n_layers,budget",
                         [(1, 1, "10%"), (1, 1, "10%-stated"), (2, 1, "10%"),
                          (3, 3, "5%"), (3, 3, "10%"), (3, 3, "20%"), (4, 1, "10%")])
def test_refresh_step_matches_oracle(cfg, n_layers, budget):
    """Every refreshed row of every layer is compared with the oracle (the
    16k workload: all 1,638 rows, in the benchmark's launch configuration)."""
    w = W.config(cfg, n_layers=n_layers)
    k = w.budgets[budget]
    layers_np = [w.layer(li) for li in range(n_layers)]
    step, layers, idx = run_step(w, layers_np, k)
    ref = O.select([{"q": L["q"], "k": L["k"], "v": L["v"]} for L in layers_np], w.q_pos0,
                   w.img_pos, w.img_off, k, lam=1.0)
    assert_scores(to_f64(step.shat), ref["s_hat"], what="s_hat")
    assert_scores(to_f64(step.c), ref["c"], what="c_j")
    assert_selection(idx, ref["s_hat"], k)
    P = w.vis_positions()
    np.testing.assert_array_equal(step.pos[:k].cpu().numpy(), P[idx])
    mask = np.zeros(w.n_vis, np.uint8)
    mask[idx] = 1
    np.testing.assert_array_equal(step.mask.cpu().numpy(), mask)
    for li, L in enumerate(layers_np):
        km, vm, o_ref, lse_ref = oracle_refresh_rows(L["k"], L["v"], P[idx], L["k_star"][idx],
                                                     L["v_star"][idx], L["q_star"][idx], range(k))
        assert_attention(to_f64(step.out[li][:k]), o_ref, w.dtype, what=f"O layer {li}")
        assert_scores(to_f64(step.lse[li][:k]), lse_ref, what=f"lse layer {li}")
        np.testing.assert_array_equal(to_f64(layers[li]["k"]), km)
        np.testing.assert_array_equal(to_f64(layers[li]["v"]), vm)


def test_visual_only_normalisation_end_to_end():
    w = W.custom(2, 28, 4, 128, 16, 40, [96, 160, 64], 8, "bf16", n_sinks=4, n_relevant=1, seed=9)
    layers_np = [w.layer(li) for li in range(2)]
    k = 32
    step, _, idx = run_step(w, layers_np, k, norm=O.NORM_VISUAL_ONLY)
    ref = O.select([{"q": L["q"], "k": L["k"], "v": L["v"]} for L in layers_np], w.q_pos0,
                   w.img_pos, w.img_off, k, lam=1.0, norm=O.NORM_VISUAL_ONLY)
    assert_scores(to_f64(step.shat), ref["s_hat"], what="s_hat")
    assert_selection(idx, ref["s_hat"], k)


def test_zero_budget_is_cache_reuse():
    """0% budget: nothing is scored or selected and the caches keep their bytes."""
    w = W.config(2)
    layers_np = [w.layer(0)]
    layers = [{"k": to_dev(L["k"]), "v": to_dev(L["v"]), "q": to_dev(L["q"])} for L in layers_np]
    before = [(bits(L["k"]).tobytes(), bits(L["v"]).tobytes()) for L in layers]
    img = api.ImageTable(w.img_pos, w.img_off)
    step = api.RefreshStep(layers, w.n_q_heads, w.q_pos0, img, 0, device=DEV)
    step.mask.fill_(5)
    step.score_and_select()
    step.refresh([])
    torch.cuda.synchronize()
    assert not step.mask.any()
    after = [(bits(L["k"]).tobytes(), bits(L["v"]).tobytes()) for L in layers]
    assert after == before


def test_full_budget_selects_every_token():
    w = W.config(2)
    layers_np = [w.layer(0)]
    step, _, idx = run_step(w, layers_np, w.n_vis)
    np.testing.assert_array_equal(idx, np.arange(w.n_vis))
    assert step.mask.all()


def test_single_image_reduces_to_token_selection():
    """K = 1: c = 1 for every lambda and the selection is the top-k of s."""
    w = W.config(2)
    layers_np = [w.layer(0)]
    k = w.budgets["10%"]
    picks = []
    for lam in (0.0, 0.5, 1.0):
        step, _, idx = run_step(w, layers_np, k, lam=lam)
        np.testing.assert_array_equal(bits(step.c), np.array([0x3F800000], np.uint32))
        picks.append(idx)
    np.testing.assert_array_equal(picks[0], picks[1])
    np.testing.assert_array_equal(picks[0], picks[2])


def test_step_is_deterministic():
    w = W.config(3, n_layers=2)
    layers_np = [w.layer(li) for li in range(2)]
    k = w.budgets["10%"]
    s1, l1, i1 = run_step(w, layers_np, k)
    s2, l2, i2 = run_step(w, layers_np, k)
    np.testing.assert_array_equal(i1, i2)
    for a, b in ((s1.shat, s2.shat), (s1.out[0], s2.out[0]), (s1.out[1], s2.out[1]),
                 (l1[1]["k"], l2[1]["k"])):
        np.testing.assert_array_equal(bits(a), bits(b))


def test_method_behaviour_sinks_are_demoted():
    """Directional check of the method (not parity): planted sinks draw high
    attention but carry small value norms, so the value-norm proxy ranks fewer
    of them into the budget than attention-only ranking does."""
    w = W.custom(1, 28, 4, 128, 32, 64, [512, 512, 512, 512], 16, "bf16", n_sinks=40, seed=21)
    k = 205
    step, _, idx = run_step(w, [w.layer(0)], k, lam=1.0)
    a = to_f64(step.a_acc)
    attn_only = np.sort(np.argsort(-a, kind="stable")[:k])
    sinks = set(w.shared()["sinks"].tolist())
    assert len(sinks & set(attn_only.tolist())) >= 30
    assert len(sinks & set(idx.tolist())) < len(sinks & set(attn_only.tolist()))


def test_method_behaviour_relevant_image_is_amplified():
    """Directional check of the method (not parity): the query-relevant image
    gets c_j > 1 and a larger share of the budget than without reweighting."""
    w = W.custom(1, 28, 4, 128, 32, 64, [512, 512, 512, 512], 16, "bf16", n_relevant=1, seed=22)
    w.rel_cos = 0.02  # weak alignment, so the images' score ranges overlap
    layers_np = [w.layer(0)]
    k = 205
    step, _, idx1 = run_step(w, layers_np, k, lam=1.0)
    rel = int(w.shared()["relevant"][0])
    c = to_f64(step.c)
    assert c[rel] > 1.0 and np.all(np.delete(c, rel) < 1.0)
    _, _, idx0 = run_step(w, layers_np, k, lam=0.0)
    lo, hi = w.img_off[rel], w.img_off[rel + 1]
    share = lambda ix: int(np.sum((ix >= lo) & (ix < hi)))
    assert share(idx0) < k
    assert share(idx1) > share(idx0)
