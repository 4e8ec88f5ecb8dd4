"""The synthetic diagnostic harness (paper_2609_05821_amd.diagnostics) on the
GPU: every error it reports equals the oracle's error for the same refresh
set, and the rules' sets are the oracle's top-k of the same scores."""
import numpy as np
import pytest
import torch

from oracle import conduit_oracle as O
from paper_2609_05821_amd import api, diagnostics as D, workloads as W
from tests.gpu_helpers import DEV, assert_selection, to_dev, to_f64

pytestmark = pytest.mark.gpu


def test_harness_matches_oracle():
    w = W.custom(1, 28, 4, 128, 19, 13, [37, 250, 301], 5, "bf16", n_sinks=6, n_relevant=1, seed=3)
    L = w.layer(0, fresh=False)
    k, v, q = (to_dev(L[x]) for x in ("k", "v", "q"))
    kv = api.kv_desc(k, v, w.n_q_heads)
    img = api.ImageTable(w.img_pos, w.img_off)
    zs = W.iso_directions(w, 0, 5)
    ratios = ((10, 100), (30, 100))
    res = D.rule_errors(kv, q, w.q_pos0, img, to_dev(zs), ratios=ratios, seed=4)
    # oracle errors for the harness's own sets
    sc = D.layer_scores(kv, q, w.q_pos0, img)
    a_rms, vn, _ = O.score_layer(L["q"], L["k"], L["v"], w.q_pos0, w.img_pos, w.img_off, agg=O.AGG_RMS)
    xi_iso = O.iso_displacements(L["v"], w.img_pos, w.img_off, zs, 0.5)
    xi_proj = O.projected_displacements(L["v"], w.img_pos, w.img_off)
    for ri, (num, den) in enumerate(ratios):
        kk = res["budgets"][ri]
        assert kk == O.budget(w.n_vis, num, den)
        masks = D.rule_masks(kv, q, w.q_pos0, img, kk, sc, seed=4 * 1000 + ri)
        for name, target in (("vnorm", vn), ("rms_attention", a_rms), ("rms_attention_x_vnorm", a_rms * vn)):
            assert_selection(np.flatnonzero(masks[name].cpu().numpy()), target, kk)
        for name in D.RULES:
            m = masks[name].cpu().numpy()
            assert int(m.sum()) == kk
            proj = O.residual_error(L["q"][-1:], L["k"], w.q_pos0 + w.n_q - 1, w.img_pos, w.img_off, m,
                                    xi_proj)
            iso = O.residual_error(L["q"], L["k"], w.q_pos0, w.img_pos, w.img_off, m, xi_iso)
            np.testing.assert_allclose(res["projected"][name][ri], proj.sum(), rtol=2e-2)
            np.testing.assert_allclose(res["iso"][name][ri], O.iso_estimate(iso), rtol=2e-2)
    red = res["projected_reduction_vs_random"]
    assert red["random"] == [1.0, 1.0]
