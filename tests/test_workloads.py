"""The seeded workload generator: layouts, reproducibility, planted structure."""
import numpy as np
import pytest
import torch

from paper_2609_05821_amd import workloads as W

LAYOUTS = {  # cfg: (N_vis, N_ctx, q_pos0, K, first image position, k at 10%)
    1: (576, 672, 640, 1, 64, 57),
    2: (1024, 1344, 1280, 1, 256, 102),
    3: (5184, 5408, 5312, 4, 128, 518),
    4: (16384, 17280, 17152, 16, 528, 1638),
    5: (65536, 66816, 66560, 64, 1024, 6553),
}


@pytest.mark.parametrize("cfg", sorted(LAYOUTS))
def test_layout(cfg):
    w = W.config(cfg)
    n_vis, n_ctx, q0, K, p0, k10 = LAYOUTS[cfg]
    assert (w.n_vis, w.n_ctx, w.q_pos0, w.n_images, int(w.img_pos[0])) == (n_vis, n_ctx, q0, K, p0)
    assert w.budgets["10%"] == k10
    assert w.q_pos0 + w.n_q == w.n_ctx
    P = w.vis_positions()
    assert len(P) == n_vis and np.all(np.diff(P) > 0) and P[-1] < w.q_pos0


def test_separators_in_16k_layout():
    w = W.config(4)
    assert np.all(np.diff(w.img_pos) == 1024 + 16)
    assert w.img_pos[0] == 512 + 16


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000) * 10.0 ** np.random.default_rng(1).integers(-8, 8, 100000)
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(W.bf16_bits(x), ref)
    np.testing.assert_array_equal(W.bf16_to_f32(ref), torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_seed_reproducible_and_distinct():
    a = W.config(2).layer(0, fresh=False)
    b = W.config(2).layer(0, fresh=False)
    c = W.config(2, seed=1).layer(0, fresh=False)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])
    assert not np.array_equal(a["k"], c["k"])


def test_planted_sinks_and_value_norms():
    w = W.config(1)
    L = w.layer(0)
    sh = w.shared()
    P = w.vis_positions()
    assert len(sh["sinks"]) == 5
    v = L["v"].astype(np.float64).reshape(w.n_ctx, -1)
    rho = np.linalg.norm(v, axis=1)
    ordinary = np.setdiff1d(np.arange(w.n_ctx), P[sh["sinks"]])
    # LogNormal(0, 0.5): median 1, log-sd 0.5
    assert abs(np.median(np.log(rho[ordinary]))) < 0.06
    assert abs(np.std(np.log(rho[ordinary])) - 0.5) < 0.05
    assert np.all(rho[P[sh["sinks"]]] < 0.05 * 4)
    # sink logits are ~6 on average, ordinary ones ~0
    q = L["q"].astype(np.float64)
    k = L["k"].astype(np.float64)
    z = np.einsum("ihd,thd->iht", q, k) / np.sqrt(w.head_dim)
    assert 4.5 < z[:, :, P[sh["sinks"]]].mean() < 7.5
    assert abs(z[:, :, ordinary].mean()) < 0.1


def test_relevant_images_aligned():
    w = W.config(3, n_layers=1)
    L = w.layer(0, fresh=False)
    sh = w.shared()
    assert len(sh["relevant"]) == 1
    q = W.bf16_to_f32(L["q"]).astype(np.float64)
    k = W.bf16_to_f32(L["k"]).astype(np.float64)
    G = w.group
    logits = []
    for j in range(w.n_images):
        lo = int(w.img_pos[j])
        hi = lo + 1296
        kk = np.repeat(k[lo:hi], G, axis=1)
        logits.append((np.einsum("ihd,thd->iht", q[:8], kk) / np.sqrt(128)).mean())
    rel = int(sh["relevant"][0])
    assert 2.5 < logits[rel] < 4.5
    assert all(abs(logits[j]) < 0.3 for j in range(w.n_images) if j != rel)


def test_fresh_rows_follow_isotropic_model():
    w = W.config(2)
    L = w.layer(0)
    P = w.vis_positions()
    k = W.bf16_to_f32(L["k"]).astype(np.float64)[P].reshape(len(P), -1)
    ks = W.bf16_to_f32(L["k_star"]).astype(np.float64).reshape(len(P), -1)
    ratio = np.sum((ks - k) ** 2, axis=1) / np.sum(k ** 2, axis=1)
    assert abs(ratio.mean() - 0.25) < 0.01          # kappa^2
    assert L["q_star"].shape == (1024, 28, 128)
