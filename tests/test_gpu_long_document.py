"""The long-document workload at full size on the GPU: 64 page images x 1,024
visual tokens (65,536) after a 1,024-token prefix, 256 span queries, GQA 28/4,
head_dim 128, bf16, one layer, 10% budget (6,553 refreshed rows).

The largest shapes the library is run at.  The oracle computes sampled outputs
one by one (row log-sum-exps of the scoring softmax, refreshed rows); the
column sums, which depend on every row, are held to properties that hold at
any size (non-negative; the visual share of each row's attention mass is at
most 1, exactly 1 with visual-only normalisation).  Fresh rows for the refresh
come from a seeded generator of the test.
"""
import numpy as np
import pytest
import torch

from oracle import conduit_oracle as O
from paper_2609_05821_amd import api, workloads as W
from tests.gpu_helpers import DEV, assert_attention, assert_scores, to_dev, to_f64
from tests.test_gpu_score import Layer, score_one

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def workload():
    w = W.config(5, n_layers=1)
    return w, Layer(w, 0)


@pytest.mark.parametrize("norm", [O.NORM_CAUSAL_ROW, O.NORM_VISUAL_ONLY], ids=["causal", "visual"])
def test_long_document_scoring(workload, norm):
    w, L = workload
    got = score_one(w, L, norm)
    P = w.vis_positions()
    q, k = O.to_f64(L.np["q"]), O.to_f64(L.np["k"])
    scale = 1.0 / np.sqrt(w.head_dim)
    rng = np.random.default_rng(51 + norm)
    rows = sorted(set([0, w.n_q - 1] + rng.choice(w.n_q, size=2, replace=False).tolist()))
    lse = to_f64(got["lse"])
    for kvh in range(w.n_kv_heads):
        kc = np.ascontiguousarray(k[:, kvh, :]) if norm == O.NORM_CAUSAL_ROW else \
            np.ascontiguousarray(k[P, kvh, :])
        for i in rows:
            keys = kc[: w.q_pos0 + i + 1] if norm == O.NORM_CAUSAL_ROW else kc
            for h in range(kvh * w.group, (kvh + 1) * w.group):
                _, ref = O.attention_row(q[i, h], keys, scale)
                assert_scores(lse[i, h:h + 1], np.array([ref]), what=f"row lse ({i}, {h})")
    a = to_f64(got["a"])
    assert (a >= 0).all()
    total = a.sum()
    if norm == O.NORM_VISUAL_ONLY:
        assert abs(total - 1.0) <= 1e-4, total
    else:
        assert 0.0 < total <= 1.0 + 1e-4, total
    assert_scores(to_f64(got["v"]), O.value_norms(L.np["v"], w.img_pos, w.img_off), what="||V_t||")
    # s = a * ||V|| in float32, as the finalisation computes it
    s32 = got["a"].cpu().numpy() * got["v"].cpu().numpy()
    np.testing.assert_array_equal(got["s_acc"].cpu().numpy(), s32)


def test_long_document_refresh(workload):
    w, L = workload
    k = w.budgets["10%"]
    assert k == 6553
    rng = np.random.default_rng(52)
    # selection shaped like the method's: half in the relevant pages
    rel = w.shared()["relevant"]
    pool = np.concatenate([np.arange(w.img_off[j], w.img_off[j + 1]) for j in rel])
    sel = np.sort(np.concatenate([rng.choice(pool, size=k // 2, replace=False),
                                  rng.choice(np.setdiff1d(np.arange(w.n_vis), pool), size=k - k // 2,
                                             replace=False)]))
    P = w.vis_positions()
    pos_np = P[sel]
    k_new = w._cast(rng.standard_normal((k, w.n_kv_heads, w.head_dim)).astype(np.float32))
    v_new = w._cast(rng.standard_normal((k, w.n_kv_heads, w.head_dim)).astype(np.float32))
    q_sel = w._cast(rng.standard_normal((k, w.n_q_heads, w.head_dim)).astype(np.float32))
    kc, vc = to_dev(L.np["k"]), to_dev(L.np["v"])
    kv = api.kv_desc(kc, vc, w.n_q_heads)
    pos = torch.from_numpy(pos_np.astype(np.int32)).to(DEV)
    api.conduit_scatter_kv(kv, pos, to_dev(k_new), to_dev(v_new))
    qd = to_dev(q_sel)
    out = torch.empty((k, w.n_q_heads, w.head_dim), dtype=qd.dtype, device=DEV)
    lse = torch.empty((k, w.n_q_heads), dtype=torch.float32, device=DEV)
    api.conduit_refresh_attn(kv, qd, pos, out, lse_out=lse)
    torch.cuda.synchronize()
    rows = sorted(set([0, k - 1] + rng.choice(k, size=4, replace=False).tolist()))
    km, vm, o_ref, lse_ref = O.refresh_layer(L.np["k"], L.np["v"], pos_np, k_new, v_new, q_sel, rows=rows)
    r = np.asarray(rows)
    assert_attention(to_f64(out)[r], o_ref[r], w.dtype, what="O")
    assert_scores(to_f64(lse)[r], lse_ref[r], what="lse")
    np.testing.assert_array_equal(to_f64(kc), km)
    np.testing.assert_array_equal(to_f64(vc), vm)
    assert torch.isfinite(out.float()).all()
