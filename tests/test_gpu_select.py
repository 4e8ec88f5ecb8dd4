"""Reweighting and global top-k on the GPU (conduit_select_topk) against the
CPU oracle."""
import zlib

import numpy as np
import pytest
import torch

from oracle import conduit_oracle as O
from paper_2609_05821_amd import api
from tests.gpu_helpers import DEV, assert_scores, bits, to_f64

pytestmark = pytest.mark.gpu


def layout(sizes, gap=3, start=5):
    pos, off, cur = [], [0], start
    for n in sizes:
        pos.append(cur)
        cur += n + gap
        off.append(off[-1] + n)
    return np.array(pos), np.array(off)


def run_select(s_acc, a_acc, n_layers, img_pos, img_off, lam, k):
    img = api.ImageTable(img_pos, img_off)
    nv = img.n_vis
    s = torch.from_numpy(s_acc.astype(np.float32)).to(DEV)
    a = torch.from_numpy(a_acc.astype(np.float32)).to(DEV)
    out = {"idx": torch.full((max(k, 1),), -1, dtype=torch.int32, device=DEV),
           "pos": torch.full((max(k, 1),), -1, dtype=torch.int32, device=DEV),
           "mask": torch.full((nv,), 7, dtype=torch.uint8, device=DEV),
           "shat": torch.zeros(nv, device=DEV), "c": torch.zeros(len(img_pos), device=DEV)}
    api.conduit_select_topk(s, a, n_layers, img, lam, k, out["idx"], out["pos"], mask_out=out["mask"],
                            shat_out=out["shat"], c_out=out["c"])
    torch.cuda.synchronize()
    return {key: val.cpu().numpy() for key, val in out.items()}


def reference(s_acc, a_acc, n_layers, img_pos, img_off, lam):
    """Oracle Eq. 8-10 from the same fp32 inputs (decoded exactly)."""
    s = s_acc.astype(np.float32).astype(np.float64)
    A = a_acc.astype(np.float32).astype(np.float64)
    _, pi = O.visual_layout(img_pos, img_off)
    g, _, c = O.image_coefficients(A, n_layers, img_off, lam)
    return c, O.composite_score(s / n_layers, c, pi)


SIZES = {
    "one_token": [1],
    "single_image_ragged": [1000],
    "three_images": [37, 250, 301],
    "sixteen_images": [1024] * 16,
    # 16,385 .. 32,768 keys: 32 keys per thread in registers
    "twenty_four_images_ragged": [1024] * 23 + [999],
    "thirty_two_images": [1024] * 32,
    "long_document": [1024] * 64,
    "many_small": [7] * 256,
    # several workgroups of 4,096 tokens, up to ~110 images each
    "many_small_multi": [37] * 250,
    "ragged_long": [1024] * 40 + [513],
}


@pytest.mark.parametrize("lam", [0.0, 0.5, 1.0])
@pytest.mark.parametrize("name", sorted(SIZES))
def test_select_matches_oracle(name, lam):
    rng = np.random.default_rng(zlib.crc32(f"{name}/{lam}".encode()))
    img_pos, img_off = layout(SIZES[name])
    nv = int(img_off[-1])
    n_layers = 3
    a = rng.random(nv) * 1e-3 * np.repeat(rng.random(len(img_pos)) * 4, np.diff(img_off))
    s = a * rng.lognormal(0, 0.5, nv) * n_layers
    for k in sorted({0, 1, max(1, nv // 10), max(1, nv - 1), nv}):
        got = run_select(s, a, n_layers, img_pos, img_off, lam, k)
        assert not (got["mask"] > 1).any()
        if k == 0:
            assert not got["mask"].any()
            continue
        c, shat = reference(s, a, n_layers, img_pos, img_off, lam)
        assert_scores(got["c"], c, rtol=1e-5, what="c_j")
        assert_scores(got["shat"], shat, rtol=1e-5, what="s_hat")
        # bit-exact against the oracle's top-k on the GPU's own fp32 scores
        ref_idx = O.topk_select(got["shat"].astype(np.float64), k)
        np.testing.assert_array_equal(got["idx"][:k], ref_idx)
        P, _ = O.visual_layout(img_pos, img_off)
        np.testing.assert_array_equal(got["pos"][:k], P[ref_idx])
        m = np.zeros(nv, np.uint8)
        m[ref_idx] = 1
        np.testing.assert_array_equal(got["mask"], m)


# 4,096 / 4,097 and 131,072 / 131,073 straddle the one-workgroup, the
# multi-workgroup and the streaming kernels.
@pytest.mark.parametrize("n", [5, 1000, 4096, 4097, 16384, 16385, 24576, 32767, 32768, 65536, 100000,
                               131072, 131073])
def test_ties_go_to_lower_index(n):
    """Heavy ties: few distinct scores, so the boundary value repeats often."""
    rng = np.random.default_rng(n)
    img_pos, img_off = layout([n])
    s = rng.integers(0, 6, size=n).astype(np.float64) / 8.0
    s[rng.integers(0, n, size=max(1, n // 50))] = 0.0
    for k in sorted({1, n // 3 + 1, n // 2, n}):
        got = run_select(s, np.ones(n), 1, img_pos, img_off, 1.0, k)
        ref_idx = O.topk_select(s, k)
        np.testing.assert_array_equal(got["idx"][:k], ref_idx)


@pytest.mark.parametrize("n", [1000, 4097, 16385, 32768, 65536, 131073])
def test_all_equal_scores_take_lowest_indices(n):
    """No bit varies between the keys: the threshold is the common value and
    the k lowest indices are taken (one-workgroup, multi-workgroup and
    streaming kernels)."""
    img_pos, img_off = layout([n])
    s = np.full(n, 0.25)
    for k in sorted({1, 100, n - 1, n}):
        got = run_select(s, np.ones(n), 1, img_pos, img_off, 1.0, k)
        np.testing.assert_array_equal(got["idx"][:k], np.arange(k))
        assert got["mask"].sum() == k


def test_single_image_coefficient_is_one():
    rng = np.random.default_rng(1)
    img_pos, img_off = layout([777])
    for lam in (0.0, 0.3, 1.0):
        got = run_select(rng.random(777), rng.random(777), 2, img_pos, img_off, lam, 50)
        np.testing.assert_array_equal(bits(torch.from_numpy(got["c"])), np.array([0x3F800000], np.uint32))


def test_lambda_zero_drops_coefficients():
    rng = np.random.default_rng(2)
    img_pos, img_off = layout([100, 200, 50])
    got = run_select(rng.random(350), rng.random(350), 1, img_pos, img_off, 0.0, 35)
    np.testing.assert_array_equal(got["c"], np.ones(3, np.float32))


def test_zero_attention_gives_unit_coefficients():
    img_pos, img_off = layout([10, 20])
    got = run_select(np.zeros(30), np.zeros(30), 1, img_pos, img_off, 1.0, 4)
    np.testing.assert_array_equal(got["c"], np.ones(2, np.float32))
    np.testing.assert_array_equal(got["idx"][:4], [0, 1, 2, 3])


def test_worked_example():
    """The hand-worked reweighting example (tests/golden/worked_examples.json)."""
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")))
    g = g["topk_reweighting"]
    a, v = np.array(g["a"]), np.array(g["v"])
    for case in g["cases"]:
        got = run_select(a * v, a, 1, np.array(g["img_pos"]), np.array(g["img_off"]), case["lam"], g["k"])
        assert list(got["idx"][:2]) == case["idx"]
        np.testing.assert_allclose(got["c"], case["c"], rtol=1e-6)
