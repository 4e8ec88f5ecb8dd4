"""Pins for the CPU oracle: checks that do not reuse the oracle's own formulas.

Each pin takes the oracle module as its argument and raises AssertionError (or
any exception) when the oracle is wrong, so the same pins can be run against
deliberately broken copies of the oracle (see test_oracle_mutations.py).

What pins what:
  * bf16 inputs          hand-worked bit patterns (sign, exponent, mantissa
                          fields; subnormal, largest finite, infinities) and
                          random patterns against torch's bfloat16 decoder;
  * budget (Eq. 2)       exact rational floor via fractions.Fraction, and the
                          hand-computed budgets of the workloads;
  * scoring (Eq. 6)      a hand-worked example, closed forms for equal keys,
                          scipy's softmax for a single row, and torch's
                          scaled_dot_product_attention with one-hot values
                          (whose output rows are the attention weights);
  * value norm (Eq. 7)   numpy.linalg.norm and a hand-worked 3-4-5 row;
  * layer mean (Eq. 7)   closed forms with identical / permuted layers;
  * c_j (Eq. 8-9)        the normalisation sum_j c_j = K (App. C.2), K = 1 and
                          lambda = 0 reductions, a two-image closed form;
  * top-k (Eq. 11)       the hand-worked reweighting example, and brute force
                          over all subsets of Lemma 1's objective;
  * refresh              torch SDPA over the merged cache, the 100% budget
                          (full prefill) and 0% budget (cache reuse) anchors,
                          and closed forms for equal keys / equal values;
  * RMS aggregation (Eq. 4)  SDPA weights squared and averaged per column, and
                          the closed form of equal keys over rows of growing
                          length;
  * value-norm table     numpy.linalg.norm, and the identity of scoring with
                          the table and scoring from the cache (Sec. 4.3);
  * attention-only rule  s_hat rebuilt from SDPA weights and c_j, brute-force
                          ranking;
  * explicit quotas      hand-worked apportionments (proportional, capped,
                          tied), an exact rational implementation on random
                          cases away from ties, and brute-force in-image top-k;
  * text rows            brute-force set complement of the image runs; with
                          every visual row selected plus the text rows the
                          recompute equals SDPA full prefill at every position;
                          a partial selection plus text rows equals SDPA over
                          the merged cache;
  * paged caches         a hand-worked page table, and random page
                          permutations that must give back the original cache;
  * residual error       (Eq. 3, App. D.1/D.3) torch SDPA whose values are the
                          displacements, zeroed outside the non-refreshed
                          visual keys; zero when every visual token is
                          refreshed; the moments App. D.1 states for the
                          isotropic samples (mean 0, E||xi||^2 =
                          kappa^2 ||V||^2, checked with numpy.linalg.norm over
                          many samples); unbiasedness of the estimate against
                          the closed form built from SDPA weights.
"""
from __future__ import annotations

import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import scipy.special
import torch

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "worked_examples.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def _rand_layout(rng, n_imgs, prefix, sep):
    sizes = [int(x) for x in rng.integers(1, 6, size=n_imgs)]
    img_pos, img_off, cur = [], [0], prefix
    for n in sizes:
        cur += sep
        img_pos.append(cur)
        cur += n
        img_off.append(img_off[-1] + n)
    return np.array(img_pos), np.array(img_off), cur


def _p_vis(img_pos, img_off):
    return np.concatenate([np.arange(p, p + img_off[j + 1] - img_off[j])
                           for j, p in enumerate(img_pos)])


def _sdpa_weights(q, k, mask):
    """Attention weights via torch SDPA: values are one-hot over the keys.

    q [n, H_q, d], k [N, H_kv, d], mask [n, N] boolean (True = may attend).
    Grouped heads are expanded with repeat_interleave (query head h reads
    KV head h // G).  Returns weights [n, H_q, N] float64.
    """
    n, hq, d = q.shape
    N, hkv, _ = k.shape
    qt = torch.from_numpy(q).permute(1, 0, 2).unsqueeze(0)            # [1, H_q, n, d]
    kt = torch.from_numpy(k).permute(1, 0, 2).unsqueeze(0)
    kt = kt.repeat_interleave(hq // hkv, dim=1)                        # [1, H_q, N, d]
    eye = torch.eye(N, dtype=torch.float64).expand(1, hq, N, N)
    w = torch.nn.functional.scaled_dot_product_attention(
        qt, kt, eye, attn_mask=torch.from_numpy(mask)[None, None])
    return w[0].permute(1, 0, 2).numpy()


def _sdpa_out(q, k, v, mask):
    n, hq, d = q.shape
    N, hkv, _ = k.shape
    g = hq // hkv
    qt = torch.from_numpy(q).permute(1, 0, 2).unsqueeze(0)
    kt = torch.from_numpy(k).permute(1, 0, 2).unsqueeze(0).repeat_interleave(g, dim=1)
    vt = torch.from_numpy(v).permute(1, 0, 2).unsqueeze(0).repeat_interleave(g, dim=1)
    o = torch.nn.functional.scaled_dot_product_attention(
        qt, kt, vt, attn_mask=torch.from_numpy(mask)[None, None])
    return o[0].permute(1, 0, 2).numpy()


# ---------------------------------------------------------------------------

def pin_bf16_decode(o):
    """bf16 inputs are decoded by the oracle itself (uint16 bit patterns: the
    top half of an IEEE binary32).  Hand-worked patterns (sign, 8 exponent
    bits, 7 mantissa bits) and random patterns against torch's own bfloat16
    decoder."""
    cases = {
        0x3F80: 1.0,                          # exponent 127, mantissa 0
        0xC040: -3.0,                         # sign, exponent 128, mantissa 1/2 -> -1.5 * 2
        0x3E80: 0.25,                         # exponent 125
        0x4049: 3.140625,                     # exponent 128, mantissa 73/128
        0x0001: 2.0 ** -133,                  # smallest subnormal: 2^-7 * 2^-126
        0x7F7F: (2.0 - 2.0 ** -7) * 2.0 ** 127,  # largest finite
        0x0080: 2.0 ** -126,                  # smallest normal
        0x7F80: math.inf,
        0xFF80: -math.inf,
    }
    bits = np.array(list(cases), dtype=np.uint16)
    got = o.to_f64(bits)
    assert got.dtype == np.float64
    for b, want, g in zip(cases, cases.values(), got):
        assert g == want, (hex(b), g, want)
    neg_zero = o.to_f64(np.array([0x8000], dtype=np.uint16))[0]
    assert neg_zero == 0.0 and math.copysign(1.0, neg_zero) < 0
    rng = np.random.default_rng(11)
    r = rng.integers(0, 1 << 16, size=(64, 3, 8), dtype=np.uint16)
    r = np.where((r & 0x7F80) == 0x7F80, r & 0x807F, r)  # no inf/NaN patterns
    ref = torch.from_numpy(r.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    got = o.to_f64(r)
    assert got.shape == r.shape
    assert np.array_equal(got, ref)
    f = rng.standard_normal(17).astype(np.float32)
    assert np.array_equal(o.to_f64(f), f.astype(np.float64))


def pin_budget(o):
    gold = _golden()["budget"]["cases"]
    for c in gold:
        assert o.budget(c["n_vis"], *c["r"]) == c["k"], c
    for den in (10, 100, 1000):
        for num in range(0, den + 1, max(1, den // 50)):
            for n in (1, 7, 99, 100, 576, 1000, 5184, 16384, 65536):
                assert o.budget(n, num, den) == math.floor(Fraction(num, den) * n)


def pin_layout(o):
    P, pi = o.visual_layout(np.array([3, 10]), np.array([0, 2, 5]))
    assert list(P) == [3, 4, 10, 11, 12]
    assert list(pi) == [0, 0, 1, 1, 1]


def pin_scoring_worked_example(o):
    g = _golden()["scoring_alpha"]
    k = np.array(g["keys"]).reshape(-1, 1, 1)
    q = np.ones((1, 1, 1))
    v = np.ones_like(k)
    for norm, a_ref, lse_ref in ((o.NORM_CAUSAL_ROW, g["a_causal"], g["lse_causal"]),
                                 (o.NORM_VISUAL_ONLY, g["a_visual_only"], g["lse_visual_only"])):
        a, _, lse = o.score_layer(q, k, v, g["q_pos0"], np.array(g["img_pos"]),
                                  np.array(g["img_off"]), norm=norm, scale=1.0)
        np.testing.assert_allclose(a, a_ref, rtol=1e-13)
        np.testing.assert_allclose(lse[0, 0], lse_ref, rtol=1e-13)


def pin_scoring_equal_keys(o):
    """Equal keys: every row is uniform over its domain (closed form)."""
    rng = np.random.default_rng(1)
    img_pos, img_off, cur = _rand_layout(rng, 3, prefix=4, sep=2)
    n_q, hq, hkv, d = 3, 4, 2, 8
    n_ctx = cur + n_q
    k = np.tile(rng.standard_normal((1, hkv, d)), (n_ctx, 1, 1))
    q = rng.standard_normal((n_q, hq, d))
    v = rng.standard_normal((n_ctx, hkv, d))
    n_vis = img_off[-1]
    a, _, lse = o.score_layer(q, k, v, cur, img_pos, img_off, norm=o.NORM_CAUSAL_ROW)
    expect = np.mean([1.0 / (cur + i + 1) for i in range(n_q)])
    np.testing.assert_allclose(a, np.full(n_vis, expect), rtol=1e-12)
    for i in range(n_q):
        for h in range(hq):
            z = (q[i, h] @ k[0, h // 2]) / math.sqrt(d)
            np.testing.assert_allclose(lse[i, h], z + math.log(cur + i + 1), rtol=1e-12,
                                       atol=1e-12)
    a, _, lse = o.score_layer(q, k, v, cur, img_pos, img_off, norm=o.NORM_VISUAL_ONLY)
    np.testing.assert_allclose(a, np.full(n_vis, 1.0 / n_vis), rtol=1e-12)


def pin_scoring_single_row_scipy(o):
    rng = np.random.default_rng(2)
    d, n_ctx = 16, 12
    k = rng.standard_normal((n_ctx, 1, d))
    q = rng.standard_normal((1, 1, d))
    v = rng.standard_normal((n_ctx, 1, d))
    img_pos, img_off = np.array([2, 7]), np.array([0, 3, 6])
    a, _, lse = o.score_layer(q, k, v, n_ctx - 1, img_pos, img_off, scale=0.3)
    alpha = scipy.special.softmax(0.3 * (k[:, 0, :] @ q[0, 0]))
    np.testing.assert_allclose(a, alpha[_p_vis(img_pos, img_off)], rtol=1e-12)
    np.testing.assert_allclose(lse[0, 0], scipy.special.logsumexp(0.3 * (k[:, 0, :] @ q[0, 0])),
                               rtol=1e-12)


def pin_scoring_sdpa(o):
    """Random GQA shapes: a_t equals the visual columns of SDPA's weights."""
    rng = np.random.default_rng(3)
    for trial, (hq, hkv, d, n_q, n_img) in enumerate([(4, 2, 8, 3, 2), (6, 3, 4, 2, 3),
                                                       (3, 1, 8, 4, 1), (2, 2, 4, 1, 2)]):
        img_pos, img_off, cur = _rand_layout(rng, n_img, prefix=3, sep=trial % 2)
        n_ctx = cur + n_q
        q = rng.standard_normal((n_q, hq, d))
        k = rng.standard_normal((n_ctx, hkv, d))
        v = rng.standard_normal((n_ctx, hkv, d))
        P = _p_vis(img_pos, img_off)
        causal = np.arange(n_ctx)[None, :] <= (cur + np.arange(n_q))[:, None]
        w = _sdpa_weights(q, k, causal)
        a, _, _ = o.score_layer(q, k, v, cur, img_pos, img_off, norm=o.NORM_CAUSAL_ROW)
        np.testing.assert_allclose(a, w[:, :, P].sum(axis=(0, 1)) / (n_q * hq), rtol=1e-10)
        vis_only = np.zeros((n_q, n_ctx), bool)
        vis_only[:, P] = True
        w = _sdpa_weights(q, k, vis_only)
        a, _, _ = o.score_layer(q, k, v, cur, img_pos, img_off, norm=o.NORM_VISUAL_ONLY)
        np.testing.assert_allclose(a, w[:, :, P].sum(axis=(0, 1)) / (n_q * hq), rtol=1e-10)


def pin_value_norm(o):
    g = _golden()["value_norm"]
    v = np.zeros((3, 2, 2))
    v[1] = np.array(g["v_row"])
    k = np.zeros_like(v)
    q = np.zeros((1, 2, 2))
    _, vn, _ = o.score_layer(q, k, v, 2, np.array([1]), np.array([0, 1]))
    np.testing.assert_allclose(vn, [g["norm"]], rtol=1e-14)
    rng = np.random.default_rng(4)
    img_pos, img_off, cur = _rand_layout(rng, 2, prefix=2, sep=1)
    v = rng.standard_normal((cur + 1, 3, 4))
    _, vn, _ = o.score_layer(rng.standard_normal((1, 6, 4)), rng.standard_normal((cur + 1, 3, 4)),
                             v, cur, img_pos, img_off)
    P = _p_vis(img_pos, img_off)
    np.testing.assert_allclose(vn, np.linalg.norm(v[P].reshape(len(P), -1), axis=1), rtol=1e-13)


def pin_layer_mean(o):
    rng = np.random.default_rng(5)
    a1, v1, a2, v2 = (rng.random(7) for _ in range(4))
    s, A = o.aggregate_layers([a1], [v1])
    np.testing.assert_allclose(s, a1 * v1, rtol=1e-15)
    np.testing.assert_allclose(A, a1, rtol=1e-15)
    s, A = o.aggregate_layers([a1, a1], [v1, v1])
    np.testing.assert_allclose(s, a1 * v1, rtol=1e-14)
    np.testing.assert_allclose(A, 2 * a1, rtol=1e-14)
    s12, _ = o.aggregate_layers([a1, a2], [v1, v2])
    s21, _ = o.aggregate_layers([a2, a1], [v2, v1])
    np.testing.assert_allclose(s12, s21, rtol=1e-14)
    # the product is taken per layer, not as a product of layer means
    np.testing.assert_allclose(s12, (a1 * v1 + a2 * v2) / 2, rtol=1e-14)


def pin_coefficients(o):
    rng = np.random.default_rng(6)
    img_off = np.array([0, 3, 4, 9, 11])
    K = len(img_off) - 1
    A = rng.random(11)
    for lam in (0.0, 0.25, 0.5, 0.75, 1.0):
        g, g_bar, c = o.image_coefficients(A, 2, img_off, lam)
        # g_j is the per-image mean over layers and tokens
        for j in range(K):
            lo, hi = img_off[j], img_off[j + 1]
            np.testing.assert_allclose(g[j], A[lo:hi].mean() / 2, rtol=1e-14)
        np.testing.assert_allclose(g_bar, g.mean(), rtol=1e-14)
        np.testing.assert_allclose(c.sum(), K, rtol=1e-13)   # App. C.2 normalisation
        if lam == 0.0:
            np.testing.assert_array_equal(c, np.ones(K))      # drop-c_j ablation
    # two images, lambda = 1: c_1 = 2 g_1 / (g_1 + g_2)
    g, _, c = o.image_coefficients(np.array([0.2, 0.4, 0.1]), 1, np.array([0, 2, 3]), 1.0)
    np.testing.assert_allclose(c, [2 * 0.3 / 0.4, 2 * 0.1 / 0.4], rtol=1e-14)
    # one image: c = 1 for every lambda (single-image limit, Sec. 3.5)
    for lam in (0.0, 0.3, 1.0):
        _, _, c = o.image_coefficients(rng.random(5), 3, np.array([0, 5]), lam)
        np.testing.assert_allclose(c, [1.0], rtol=1e-15)
    # equal image means: c = 1
    _, _, c = o.image_coefficients(np.array([0.1, 0.3, 0.2, 0.2]), 1, np.array([0, 2, 4]), 0.7)
    np.testing.assert_allclose(c, [1.0, 1.0], rtol=1e-14)
    # zero attention everywhere: c = 1
    _, _, c = o.image_coefficients(np.zeros(4), 1, np.array([0, 2, 4]), 1.0)
    np.testing.assert_array_equal(c, [1.0, 1.0])


def pin_topk_worked_example(o):
    g = _golden()["topk_reweighting"]
    img_pos, img_off = np.array(g["img_pos"]), np.array(g["img_off"])
    _, pi = o.visual_layout(img_pos, img_off)
    s, A = o.aggregate_layers([np.array(g["a"])], [np.array(g["v"])])
    np.testing.assert_allclose(s, g["s"], rtol=1e-14)
    for case in g["cases"]:
        gg, _, c = o.image_coefficients(A, 1, img_off, case["lam"])
        np.testing.assert_allclose(gg, g["g"], rtol=1e-14)
        np.testing.assert_allclose(c, case["c"], rtol=1e-14)
        s_hat = o.composite_score(s, c, pi)
        idx, pos, mask = o.refresh_mask(s_hat, g["k"], img_pos, img_off)
        assert list(idx) == case["idx"], case
        P = _p_vis(img_pos, img_off)
        assert list(pos) == list(P[case["idx"]])
        assert list(np.nonzero(mask)[0]) == case["idx"]
    assert list(o.topk_select(np.array(g["a"]), g["k"])) == g["attention_only_idx"]


def pin_topk_bruteforce(o):
    """Lemma 1: top-k maximises sum of squared scores; ties to lower indices."""
    rng = np.random.default_rng(7)
    for trial in range(40):
        n = int(rng.integers(1, 11))
        s_hat = rng.integers(0, 5, size=n).astype(np.float64) / 4.0   # many exact ties
        for k in range(n + 1):
            best, best_set = -1.0, None
            for sub in itertools.combinations(range(n), k):    # ascending tuples, lexicographic
                val = sum(s_hat[t] ** 2 for t in sub)
                if val > best:
                    best, best_set = val, sub
            got = o.topk_select(s_hat, k)
            assert tuple(int(t) for t in got) == best_set, (s_hat, k, got, best_set)


def pin_merge(o):
    rng = np.random.default_rng(8)
    cache = rng.standard_normal((10, 2, 3))
    before = cache.copy()
    pos = np.array([1, 4, 7])
    new = rng.standard_normal((3, 2, 3))
    merged, stale = o.merge_cache(cache, pos, new)
    np.testing.assert_array_equal(cache, before)
    np.testing.assert_array_equal(stale, before[pos])
    for r in range(10):
        if r in pos:
            np.testing.assert_array_equal(merged[r], new[list(pos).index(r)])
        else:
            np.testing.assert_array_equal(merged[r], before[r])


def _refresh_case(rng, hq=4, hkv=2, d=8, n_img=2):
    img_pos, img_off, cur = _rand_layout(rng, n_img, prefix=3, sep=1)
    n_ctx = cur + 2
    k = rng.standard_normal((n_ctx, hkv, d))
    v = rng.standard_normal((n_ctx, hkv, d))
    P = _p_vis(img_pos, img_off)
    k_star = rng.standard_normal((len(P), hkv, d))
    v_star = rng.standard_normal((len(P), hkv, d))
    q_star = rng.standard_normal((len(P), hq, d))
    return img_pos, img_off, k, v, P, k_star, v_star, q_star


def pin_refresh_full_budget(o):
    """100% budget: refresh equals full-prefill attention at the visual rows."""
    rng = np.random.default_rng(9)
    for hq, hkv in ((4, 2), (3, 3), (6, 1)):
        img_pos, img_off, k, v, P, ks, vs, qs = _refresh_case(rng, hq, hkv)
        idx = o.topk_select(rng.random(len(P)), len(P))
        assert list(idx) == list(range(len(P)))
        km, vm, out, _ = o.refresh_layer(k, v, P[idx], ks[idx], vs[idx], qs[idx])
        full_k, full_v = k.copy(), v.copy()
        full_k[P], full_v[P] = ks, vs
        n_ctx = len(k)
        q_full = np.zeros((n_ctx, hq, k.shape[2]))
        q_full[P] = qs
        causal = np.arange(n_ctx)[None, :] <= np.arange(n_ctx)[:, None]
        ref = _sdpa_out(q_full, full_k, full_v, causal)[P]
        np.testing.assert_allclose(out, ref, rtol=1e-10, atol=1e-12)
        np.testing.assert_array_equal(km, full_k)
        np.testing.assert_array_equal(vm, full_v)


def pin_refresh_partial_budget(o):
    """A partial selection attends over the mixed fresh/stale prefix."""
    rng = np.random.default_rng(10)
    img_pos, img_off, k, v, P, ks, vs, qs = _refresh_case(rng, 6, 2, n_img=3)
    sel = np.sort(rng.choice(len(P), size=max(1, len(P) // 3), replace=False))
    pos = P[sel]
    km, vm, out, lse = o.refresh_layer(k, v, pos, ks[sel], vs[sel], qs[sel])
    tk = torch.from_numpy(k.copy())
    tv = torch.from_numpy(v.copy())
    tk[torch.from_numpy(pos)] = torch.from_numpy(ks[sel])
    tv[torch.from_numpy(pos)] = torch.from_numpy(vs[sel])
    mask = np.arange(len(k))[None, :] <= pos[:, None]
    ref = _sdpa_out(qs[sel], tk.numpy(), tv.numpy(), mask)
    np.testing.assert_allclose(out, ref, rtol=1e-10, atol=1e-12)
    np.testing.assert_array_equal(km, tk.numpy())
    np.testing.assert_array_equal(vm, tv.numpy())


def pin_refresh_closed_forms(o):
    rng = np.random.default_rng(11)
    n_ctx, hkv, hq, d = 9, 2, 4, 5
    k = np.tile(rng.standard_normal((1, hkv, d)), (n_ctx, 1, 1))
    v = rng.standard_normal((n_ctx, hkv, d))
    pos = np.array([2, 5])
    q = rng.standard_normal((2, hq, d))
    out, lse = o.refresh_attention(q, k, v, pos)
    for i, p in enumerate(pos):
        for h in range(hq):
            np.testing.assert_allclose(out[i, h], v[: p + 1, h // 2].mean(axis=0), rtol=1e-12)
            z = q[i, h] @ k[0, h // 2] / math.sqrt(d)
            np.testing.assert_allclose(lse[i, h], z + math.log(p + 1), rtol=1e-12, atol=1e-12)
    u = rng.standard_normal((hkv, d))
    v = np.tile(u[None], (n_ctx, 1, 1))
    out, _ = o.refresh_attention(q, rng.standard_normal((n_ctx, hkv, d)), v, pos)
    for h in range(hq):
        np.testing.assert_allclose(out[:, h], np.tile(u[h // 2], (2, 1)), rtol=1e-12)


def pin_zero_budget(o):
    """0% budget: nothing is selected or scored and the cache is untouched."""
    rng = np.random.default_rng(12)
    img_pos, img_off, k, v, P, ks, vs, qs = _refresh_case(rng)
    layers = [{"q": rng.standard_normal((2, 4, 8)), "k": k, "v": v}]
    res = o.select(layers, len(k) - 2, img_pos, img_off, 0)
    assert len(res["idx"]) == 0 and len(res["pos"]) == 0
    assert res["mask"].dtype == np.uint8 and not res["mask"].any() and len(res["mask"]) == len(P)
    assert "s_hat" not in res
    km, vm, out, _ = o.refresh_layer(k, v, res["pos"], ks[:0], vs[:0], qs[:0])
    np.testing.assert_array_equal(km, k)
    np.testing.assert_array_equal(vm, v)
    assert out.size == 0


def pin_single_image_reduction(o):
    """K = 1: the composite rule is the intra-image throughput top-k."""
    rng = np.random.default_rng(13)
    n_ctx, n_q = 14, 2
    img_pos, img_off = np.array([3]), np.array([0, 9])
    layers = [{"q": rng.standard_normal((n_q, 4, 8)), "k": rng.standard_normal((n_ctx, 2, 8)),
               "v": rng.standard_normal((n_ctx, 2, 8))} for _ in range(2)]
    for lam in (0.0, 0.5, 1.0):
        res = o.select(layers, n_ctx - n_q, img_pos, img_off, 3, lam=lam)
        np.testing.assert_allclose(res["c"], [1.0], rtol=1e-15)
        np.testing.assert_allclose(res["s_hat"], res["s"], rtol=1e-15)
        assert list(res["idx"]) == sorted(np.argsort(-res["s"], kind="stable")[:3])


def pin_end_to_end_sdpa(o):
    """Algorithm 1 on random layers: s_hat rebuilt from SDPA weights and norms."""
    rng = np.random.default_rng(14)
    hq, hkv, d, n_q = 4, 2, 8, 3
    img_pos, img_off, cur = _rand_layout(rng, 3, prefix=2, sep=1)
    n_ctx = cur + n_q
    P = _p_vis(img_pos, img_off)
    layers = [{"q": rng.standard_normal((n_q, hq, d)), "k": rng.standard_normal((n_ctx, hkv, d)),
               "v": rng.standard_normal((n_ctx, hkv, d))} for _ in range(3)]
    causal = np.arange(n_ctx)[None, :] <= (cur + np.arange(n_q))[:, None]
    s = np.zeros(len(P))
    A = np.zeros(len(P))
    for L in layers:
        w = _sdpa_weights(L["q"], L["k"], causal)[:, :, P].sum(axis=(0, 1)) / (n_q * hq)
        s += w * np.linalg.norm(L["v"][P].reshape(len(P), -1), axis=1)
        A += w
    s /= 3
    g = np.array([A[img_off[j]:img_off[j + 1]].mean() / 3 for j in range(3)])
    c = g / g.mean()
    s_hat = s * np.repeat(c, np.diff(img_off))
    res = o.select(layers, cur, img_pos, img_off, 4, lam=1.0)
    np.testing.assert_allclose(res["s_hat"], s_hat, rtol=1e-10)
    np.testing.assert_allclose(res["c"], c, rtol=1e-10)


def pin_scoring_rms(o):
    """Eq. 4's root-mean-square aggregation: SDPA weights squared, averaged over
    (span token, query head) and rooted; equal keys give a closed form."""
    rng = np.random.default_rng(11)
    for trial, (hq, hkv, d, n_q, n_img) in enumerate([(4, 2, 8, 3, 2), (3, 1, 4, 2, 3)]):
        img_pos, img_off, cur = _rand_layout(rng, n_img, prefix=2, sep=trial)
        n_ctx = cur + n_q
        q = rng.standard_normal((n_q, hq, d))
        k = rng.standard_normal((n_ctx, hkv, d))
        v = rng.standard_normal((n_ctx, hkv, d))
        P = _p_vis(img_pos, img_off)
        causal = np.arange(n_ctx)[None, :] <= (cur + np.arange(n_q))[:, None]
        w = _sdpa_weights(q, k, causal)[:, :, P]
        a, _, _ = o.score_layer(q, k, v, cur, img_pos, img_off, agg=o.AGG_RMS)
        np.testing.assert_allclose(a, np.sqrt((w ** 2).sum(axis=(0, 1)) / (n_q * hq)), rtol=1e-10)
    # equal keys: row i (position q_pos0 + i) is uniform over q_pos0 + i + 1 keys
    q_pos0, n_q = 5, 3
    img_pos, img_off = np.array([1]), np.array([0, 3])
    k = np.ones((q_pos0 + n_q, 1, 2))
    a, _, _ = o.score_layer(np.ones((n_q, 2, 2)), k, np.zeros_like(k), q_pos0, img_pos, img_off,
                            agg=o.AGG_RMS)
    expect = math.sqrt(sum((1.0 / (q_pos0 + i + 1)) ** 2 for i in range(n_q)) / n_q)
    np.testing.assert_allclose(a, [expect] * 3, rtol=1e-12)


def pin_value_norm_table(o):
    """The precomputed table equals the norms of the cached rows, and scoring
    with it leaves every score unchanged (Sec. 4.3: exact)."""
    rng = np.random.default_rng(12)
    img_pos, img_off, cur = _rand_layout(rng, 3, prefix=2, sep=1)
    n_q = 2
    layers = [{"q": rng.standard_normal((n_q, 4, 4)), "k": rng.standard_normal((cur + n_q, 2, 4)),
               "v": rng.standard_normal((cur + n_q, 2, 4))} for _ in range(2)]
    P = _p_vis(img_pos, img_off)
    tables = [o.value_norms(L["v"], img_pos, img_off) for L in layers]
    for L, t in zip(layers, tables):
        np.testing.assert_allclose(t, np.linalg.norm(L["v"][P].reshape(len(P), -1), axis=1),
                                   rtol=1e-13)
    k = max(1, len(P) // 3)
    r1 = o.select(layers, cur, img_pos, img_off, k)
    r2 = o.select(layers, cur, img_pos, img_off, k, v_tables=tables)
    np.testing.assert_array_equal(r1["s"], r2["s"])
    np.testing.assert_array_equal(r1["idx"], r2["idx"])


def _bruteforce_topk(x, k):
    order = sorted(range(len(x)), key=lambda t: (-x[t], t))
    return sorted(order[:k])


def pin_attention_rule(o):
    """Value norm dropped: s_hat = (A / |L|) c_pi(t), rebuilt from SDPA weights;
    the selection is the brute-force top-k of it."""
    rng = np.random.default_rng(13)
    img_pos, img_off, cur = _rand_layout(rng, 3, prefix=3, sep=1)
    n_q, hq, hkv, d = 2, 4, 2, 4
    n_ctx = cur + n_q
    layers = [{"q": rng.standard_normal((n_q, hq, d)), "k": rng.standard_normal((n_ctx, hkv, d)),
               "v": rng.standard_normal((n_ctx, hkv, d))} for _ in range(2)]
    P = _p_vis(img_pos, img_off)
    causal = np.arange(n_ctx)[None, :] <= (cur + np.arange(n_q))[:, None]
    A = sum(_sdpa_weights(L["q"], L["k"], causal)[:, :, P].sum(axis=(0, 1)) / (n_q * hq)
            for L in layers)
    n = np.diff(img_off)
    g = np.array([A[img_off[j]:img_off[j + 1]].sum() / (2 * n[j]) for j in range(len(n))])
    lam = 0.7
    c = (1 - lam) + lam * g / g.mean()
    pi = np.repeat(np.arange(len(n)), n)
    s_hat = (A / 2) * c[pi]
    for k in (1, len(P) // 2, len(P)):
        r = o.select(layers, cur, img_pos, img_off, k, lam=lam, rule=o.RANK_ATTENTION)
        np.testing.assert_allclose(r["s_hat"], s_hat, rtol=1e-10)
        assert list(r["idx"]) == _bruteforce_topk(s_hat, k)


def _exact_quotas(c, n, k):
    """Largest remainder with caps, in exact rational arithmetic."""
    c = [Fraction(float(np.float32(x))) for x in c]
    K = len(n)
    quota, live, left = [0] * K, [True] * K, k
    while True:
        w = [c[j] * n[j] for j in range(K)]
        total = sum(w[j] for j in range(K) if live[j])
        if total == 0:
            w = [Fraction(n[j]) for j in range(K)]
            total = sum(w[j] for j in range(K) if live[j])
        share = [left * w[j] / total if live[j] else Fraction(0) for j in range(K)]
        capped = [j for j in range(K) if live[j] and share[j] >= n[j]]
        if not capped:
            break
        for j in capped:
            quota[j], live[j] = n[j], False
            left -= n[j]
    for j in range(K):
        if live[j]:
            quota[j] = min(math.floor(share[j]), n[j])
    rest = left - sum(quota[j] for j in range(K) if live[j])
    cand = sorted((j for j in range(K) if live[j] and quota[j] < n[j]),
                  key=lambda j: (-(share[j] - math.floor(share[j])), j))
    for j in cand[:rest]:
        quota[j] += 1
    return quota, share


def pin_explicit_quotas(o):
    """R26: hand-worked apportionments, an exact rational reference on random
    cases away from ties, and brute-force top-k inside each image."""
    eq = lambda c, n, k: list(o.explicit_quotas(np.array(c), np.array(n), k))
    assert eq([1, 2], [3, 3], 4) == [1, 3]            # shares 4/3, 8/3
    assert eq([1, 1, 1], [4, 4, 4], 5) == [2, 2, 1]   # equal fractions: lower images first
    assert eq([10, 1, 1], [2, 10, 10], 9) == [2, 4, 3]  # image 0 capped, 7 left
    assert eq([0, 0], [2, 3], 4) == [2, 2]            # no weight: by size (shares 8/5, 12/5)
    assert eq([3.0], [7], 5) == [5]                   # one image
    rng = np.random.default_rng(14)
    checked = 0
    for _ in range(300):
        K = int(rng.integers(1, 7))
        n = [int(x) for x in rng.integers(1, 12, size=K)]
        c = [float(x) for x in rng.uniform(0.0, 2.0, size=K)]
        k = int(rng.integers(0, sum(n) + 1))
        ref, share = _exact_quotas(c, n, k)
        fr = sorted(float(x - math.floor(x)) for x in share if x > 0)
        live = [float(x) for x in share if x > 0]
        near = any(abs(x - round(x)) < 1e-4 for x in live) or \
            any(b - a < 1e-4 for a, b in zip(fr, fr[1:]))
        got = eq(c, n, k)
        assert sum(got) == k and all(0 <= g_ <= m for g_, m in zip(got, n)), (c, n, k, got)
        if not near:
            assert got == ref, (c, n, k, got, ref)
            checked += 1
    assert checked > 150
    # in-image top-k of s with those quotas
    img_off = np.array([0, 4, 9, 11])
    s = rng.random(11)
    s[5] = s[6]  # a tie inside image 1
    for k in (0, 3, 7, 11):
        quota, idx = o.select_explicit(s, np.array([1.3, 0.6, 1.1]), img_off, k)
        expect = []
        for j in range(3):
            lo, hi = img_off[j], img_off[j + 1]
            expect += [lo + t for t in _bruteforce_topk(list(s[lo:hi]), int(quota[j]))]
        assert list(idx) == sorted(expect)
        assert sum(quota) == k


def pin_text_positions(o):
    rng = np.random.default_rng(15)
    for _ in range(20):
        img_pos, img_off, cur = _rand_layout(rng, int(rng.integers(1, 5)), prefix=int(rng.integers(0, 3)),
                                             sep=int(rng.integers(0, 3)))
        n_ctx = cur + int(rng.integers(0, 4))
        P = set(_p_vis(img_pos, img_off).tolist())
        expect = [t for t in range(n_ctx) if t not in P]
        got = o.text_positions(n_ctx, img_pos, img_off)
        assert list(got) == expect
        assert len(got) == n_ctx - int(img_off[-1])
    # hand-worked: images at 2..3 and 6..8 of 10 positions
    assert list(o.text_positions(10, np.array([2, 6]), np.array([0, 2, 5]))) == [0, 1, 4, 5, 9]


def pin_refresh_text_rows(o):
    """Every visual row plus the text rows recomputed = full prefill at every
    position; a partial selection plus the text rows = SDPA over the merged
    cache whose text rows are fresh too."""
    rng = np.random.default_rng(16)
    hq, hkv, d = 4, 2, 8
    img_pos, img_off, cur = _rand_layout(rng, 3, prefix=3, sep=2)
    n_ctx = cur + 3
    k = rng.standard_normal((n_ctx, hkv, d))
    v = rng.standard_normal((n_ctx, hkv, d))
    k_f = rng.standard_normal((n_ctx, hkv, d))   # fresh rows of every position
    v_f = rng.standard_normal((n_ctx, hkv, d))
    q_f = rng.standard_normal((n_ctx, hq, d))
    P = _p_vis(img_pos, img_off)
    T = o.text_positions(n_ctx, img_pos, img_off)
    causal = np.arange(n_ctx)[None, :] <= np.arange(n_ctx)[:, None]
    full = _sdpa_out(q_f, k_f, v_f, causal)
    rows = o.recompute_rows(P, T)
    assert sorted(rows.tolist()) == list(range(n_ctx))
    km, vm, out, _ = o.refresh_layer(k, v, rows, k_f[rows], v_f[rows], q_f[rows])
    np.testing.assert_allclose(out, full[rows], rtol=1e-10, atol=1e-12)
    np.testing.assert_array_equal(km, k_f)
    sel = P[np.sort(rng.choice(len(P), size=len(P) // 2, replace=False))]
    rows = o.recompute_rows(sel, T)
    km, vm, out, _ = o.refresh_layer(k, v, rows, k_f[rows], v_f[rows], q_f[rows])
    mk, mv = k.copy(), v.copy()
    mk[rows], mv[rows] = k_f[rows], v_f[rows]
    mask = np.arange(n_ctx)[None, :] <= rows[:, None]
    np.testing.assert_allclose(out, _sdpa_out(q_f[rows], mk, mv, mask), rtol=1e-10, atol=1e-12)


def pin_paged_cache(o):
    pages = np.arange(8, dtype=np.float64).reshape(4, 2, 1, 1)
    got = o.paged_to_contiguous(pages, np.array([2, 0, 3]), 5)
    assert got.ravel().tolist() == [4, 5, 0, 1, 6]
    rng = np.random.default_rng(17)
    for P, n_ctx in ((4, 13), (8, 16), (2, 1)):
        cache = rng.standard_normal((n_ctx, 2, 3))
        n_log = -(-n_ctx // P)
        n_pages = n_log + 3
        perm = rng.permutation(n_pages)[:n_log]
        pool = rng.standard_normal((n_pages, P, 2, 3))
        for i in range(n_log):
            blk = cache[i * P:(i + 1) * P]
            pool[perm[i], :len(blk)] = blk
        np.testing.assert_array_equal(o.paged_to_contiguous(pool, perm, n_ctx), cache)


def _residual_case(rng, hq=4, hkv=2, d=8, n_q=3):
    img_pos, img_off, cur = _rand_layout(rng, 3, prefix=2, sep=1)
    n_ctx = cur + n_q
    q = rng.standard_normal((n_q, hq, d))
    k = rng.standard_normal((n_ctx, hkv, d))
    v = rng.standard_normal((n_ctx, hkv, d))
    return img_pos, img_off, cur, n_ctx, q, k, v


def pin_residual_sdpa(o):
    """The residual of every row and head is SDPA's output when the values are
    the displacements on the non-refreshed visual keys and zero elsewhere."""
    rng = np.random.default_rng(18)
    for norm in (o.NORM_CAUSAL_ROW, o.NORM_VISUAL_ONLY):
        img_pos, img_off, cur, n_ctx, q, k, v = _residual_case(rng)
        P = _p_vis(img_pos, img_off)
        refreshed = (rng.random(len(P)) < 0.4).astype(np.uint8)
        xi = rng.standard_normal((2, len(P), 2, 8))
        err = o.residual_error(q, k, cur, img_pos, img_off, refreshed, xi, norm=norm)
        mask = np.arange(n_ctx)[None, :] <= (cur + np.arange(3))[:, None]
        if norm == o.NORM_VISUAL_ONLY:
            vis = np.zeros(n_ctx, dtype=bool)
            vis[P] = True
            mask = mask & vis[None, :]
        for m in range(2):
            vals = np.zeros((n_ctx, 2, 8))
            vals[P] = xi[m] * (refreshed == 0)[:, None, None]
            y = _sdpa_out(q, k, vals, mask)
            np.testing.assert_allclose(err[m], (y * y).sum(axis=2), rtol=1e-10, atol=1e-14)
        every = np.ones(len(P), dtype=np.uint8)
        assert not o.residual_error(q, k, cur, img_pos, img_off, every, xi, norm=norm).any()


def pin_projected_error(o):
    """App. D.3: stale values zeroed, so the displacement is V itself; with an
    empty refresh set the residual is SDPA over the visual values."""
    rng = np.random.default_rng(19)
    img_pos, img_off, cur, n_ctx, q, k, v = _residual_case(rng)
    P = _p_vis(img_pos, img_off)
    xi = o.projected_displacements(v, img_pos, img_off)
    assert xi.shape == (1, len(P), 2, 8)
    err = o.residual_error(q, k, cur, img_pos, img_off, np.zeros(len(P), np.uint8), xi)
    vals = np.zeros_like(v)
    vals[P] = v[P]
    mask = np.arange(n_ctx)[None, :] <= (cur + np.arange(3))[:, None]
    y = _sdpa_out(q, k, vals, mask)
    np.testing.assert_allclose(err[0], (y * y).sum(axis=2), rtol=1e-10)


def pin_iso_moments(o):
    """App. D.1: the samples have mean 0 and E||xi_t||^2 = kappa^2 ||V_t||^2."""
    rng = np.random.default_rng(20)
    img_pos, img_off = np.array([1, 6]), np.array([0, 3, 5])
    v = rng.standard_normal((9, 2, 4)) * rng.lognormal(0, 0.5, (9, 1, 1))
    M, kappa = 20000, 0.7
    z = rng.standard_normal((M, 5, 2, 4))
    xi = o.iso_displacements(v, img_pos, img_off, z, kappa)
    P = _p_vis(img_pos, img_off)
    target = kappa ** 2 * np.linalg.norm(v[P].reshape(5, -1), axis=1) ** 2
    sq = (xi.reshape(M, 5, -1) ** 2).sum(axis=2)        # ||xi_t||^2 per sample
    se = sq.std(axis=0) / math.sqrt(M)
    assert np.all(np.abs(sq.mean(axis=0) - target) < 5 * se), (sq.mean(axis=0), target)
    mean = xi.mean(axis=0)
    assert np.all(np.abs(mean) < 5 * xi.std(axis=0) / math.sqrt(M))
    # scaling: doubling kappa quadruples every sampled residual term
    xi2 = o.iso_displacements(v, img_pos, img_off, z[:3], 2 * kappa)
    np.testing.assert_allclose(xi2, 2 * o.iso_displacements(v, img_pos, img_off, z[:3], kappa), rtol=1e-14)


def pin_iso_unbiased(o):
    """The estimate's expectation is the isotropic closed form
    sum over non-refreshed t of alpha^2 kappa^2 ||V_t||^2 / H_kv (cross-token
    terms vanish), averaged over rows and heads; alpha from SDPA weights."""
    rng = np.random.default_rng(21)
    img_pos, img_off, cur, n_ctx, q, k, v = _residual_case(rng, hq=4, hkv=2, d=4, n_q=2)
    P = _p_vis(img_pos, img_off)
    refreshed = np.zeros(len(P), np.uint8)
    refreshed[::3] = 1
    M, kappa = 6000, 0.5
    z = rng.standard_normal((M, len(P), 2, 4))
    err = o.residual_error(q, k, cur, img_pos, img_off, refreshed,
                           o.iso_displacements(v, img_pos, img_off, z, kappa))
    mask = np.arange(n_ctx)[None, :] <= (cur + np.arange(2))[:, None]
    w = _sdpa_weights(q, k, mask)[:, :, P] * (refreshed == 0)        # [n_q, H_q, N_vis]
    vn2 = np.linalg.norm(v[P].reshape(len(P), -1), axis=1) ** 2
    expect = float(np.mean((w ** 2 * vn2).sum(axis=2))) * kappa ** 2 / 2   # H_kv = 2
    per_sample = err.mean(axis=(1, 2))
    se = per_sample.std() / math.sqrt(M)
    assert abs(o.iso_estimate(err) - expect) < 5 * se, (o.iso_estimate(err), expect, se)


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
