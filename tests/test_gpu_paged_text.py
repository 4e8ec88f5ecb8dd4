"""Text rows and paged caches on the GPU.

One refresh launch over the selected visual rows plus the request's text rows
(Sec. 3.1: text is processed normally) is checked against the oracle, and every
entry point on a paged cache (block table, Sec. 4.3 serving engine) must give
results bit-identical to the same cache stored contiguously.  Pool rows that
no table entry maps hold NaN, so a stray read shows up in the results.
"""
import numpy as np
import pytest
import torch

from oracle import conduit_oracle as O
from paper_2609_05821_amd import api, workloads as W
from tests.gpu_helpers import DEV, assert_attention, assert_scores, bits, to_dev, to_f64

pytestmark = pytest.mark.gpu

CASES = {
    "cfg1_fp32_mha": lambda: W.config(1),
    "cfg2_bf16_gqa": lambda: W.config(2),
    "ragged_bf16_gqa7": lambda: W.custom(1, 28, 4, 128, 19, 13, [37, 250, 301], 5, "bf16", n_sinks=6,
                                         n_relevant=1, seed=3),
    "ragged_bf16_d64_gqa4": lambda: W.custom(1, 8, 2, 64, 40, 7, [100, 33], 3, "bf16", seed=4),
    "ragged_fp32_d128_gqa2": lambda: W.custom(1, 4, 2, 128, 5, 3, [20, 45, 11], 2, "f32", seed=6),
}


def recompute_inputs(w, L, sel):
    """Rows of one layer's recompute (selected visual rows, then text rows) and
    their fresh K, V and queries, in that order."""
    P, T = w.vis_positions(), w.text_positions()
    rows = np.concatenate([P[sel], T]).astype(np.int64)
    cat = lambda a, b: np.ascontiguousarray(np.concatenate([a[sel], b]))
    return rows, cat(L["k_star"], L["k_text_star"]), cat(L["v_star"], L["v_text_star"]), \
        cat(L["q_star"], L["q_text_star"])


def run_recompute(w, kv, rows, kn, vn, qn):
    pos = torch.from_numpy(rows.astype(np.int32)).to(DEV)
    n = len(rows)
    k_old = torch.empty((n, w.n_kv_heads, w.head_dim), dtype=torch.float32 if w.dtype == "f32"
                        else torch.bfloat16, device=DEV)
    v_old = torch.empty_like(k_old)
    api.conduit_scatter_kv(kv, pos, to_dev(kn), to_dev(vn), k_old_out=k_old, v_old_out=v_old)
    q = to_dev(qn)
    out = torch.empty((n, w.n_q_heads, w.head_dim), dtype=q.dtype, device=DEV)
    lse = torch.empty((n, w.n_q_heads), dtype=torch.float32, device=DEV)
    api.conduit_refresh_attn(kv, q, pos, out, lse_out=lse)
    torch.cuda.synchronize()
    return {"o": out, "lse": lse, "k_old": k_old, "v_old": v_old}


def selection(w, seed):
    rng = np.random.default_rng(seed)
    k = max(1, w.n_vis // 10)
    return np.sort(rng.choice(w.n_vis, size=k, replace=False))


@pytest.mark.parametrize("case", sorted(CASES))
def test_text_rows_refresh_matches_oracle(case):
    w = CASES[case]()
    L = w.layer(0, text=True)
    T = w.text_positions()
    np.testing.assert_array_equal(T, O.text_positions(w.n_ctx, w.img_pos, w.img_off))
    sel = selection(w, len(case))
    rows, kn, vn, qn = recompute_inputs(w, L, sel)
    np.testing.assert_array_equal(rows, O.recompute_rows(w.vis_positions()[sel], T))
    kc, vc = to_dev(L["k"]), to_dev(L["v"])
    got = run_recompute(w, api.kv_desc(kc, vc, w.n_q_heads), rows, kn, vn, qn)
    km, vm, o_ref, lse_ref = O.refresh_layer(L["k"], L["v"], rows, kn, vn, qn)
    assert_attention(to_f64(got["o"]), o_ref, w.dtype, what="O")
    assert_scores(to_f64(got["lse"]), lse_ref, what="lse")
    np.testing.assert_array_equal(to_f64(kc), km)
    np.testing.assert_array_equal(to_f64(vc), vm)
    np.testing.assert_array_equal(to_f64(got["k_old"]), O.to_f64(L["k"])[rows])


def test_full_recompute_with_text_rows_equals_full_prefill():
    """Every visual row and every text row recomputed: each output row is the
    dense causal attention row of a prefill over the fully fresh cache."""
    w = CASES["ragged_bf16_gqa7"]()
    L = w.layer(0, text=True)
    sel = np.arange(w.n_vis)
    rows, kn, vn, qn = recompute_inputs(w, L, sel)
    kc, vc = to_dev(L["k"]), to_dev(L["v"])
    got = run_recompute(w, api.kv_desc(kc, vc, w.n_q_heads), rows, kn, vn, qn)
    fk = np.zeros((w.n_ctx, w.n_kv_heads, w.head_dim))
    fv, fq = np.zeros_like(fk), np.zeros((w.n_ctx, w.n_q_heads, w.head_dim))
    fk[rows], fv[rows], fq[rows] = O.to_f64(kn), O.to_f64(vn), O.to_f64(qn)
    dense, _ = O.refresh_attention(fq, fk, fv, np.arange(w.n_ctx))
    assert_attention(to_f64(got["o"]), dense[rows], w.dtype, what="O vs full prefill")
    np.testing.assert_array_equal(to_f64(kc), fk)


def test_text_rows_16k_workload_sampled_rows():
    """The 16,384-visual-token layer at 10% plus its 896 text rows in one
    launch; rows checked one by one on a sample that includes text rows."""
    w = W.config(4)
    L = w.layer(0, text=True)
    sel = selection(w, 45)
    rows, kn, vn, qn = recompute_inputs(w, L, sel)
    kc, vc = to_dev(L["k"]), to_dev(L["v"])
    got = run_recompute(w, api.kv_desc(kc, vc, w.n_q_heads), rows, kn, vn, qn)
    k = len(sel)
    rng = np.random.default_rng(46)
    check = sorted(set([0, k - 1, k, k + 1, len(rows) - 1] + rng.choice(len(rows), 24, replace=False).tolist()))
    km, vm, o_ref, lse_ref = O.refresh_layer(L["k"], L["v"], rows, kn, vn, qn, rows=check)
    assert_attention(to_f64(got["o"])[check], o_ref[check], w.dtype, what="O")
    assert_scores(to_f64(got["lse"])[check], lse_ref[check], what="lse")
    np.testing.assert_array_equal(to_f64(kc), km)


# ---------------------------------------------------------------------------
# Paged caches
# ---------------------------------------------------------------------------

def page_table(n_ctx, page, rng, spare=3):
    """A shuffled block table over a pool with `spare` unmapped pages."""
    n_log = -(-n_ctx // page)
    return rng.permutation(n_log + spare)[:n_log].astype(np.int32), n_log + spare


def page_pool(x, page, table, n_pages):
    """Scatter a [n_ctx, H, d] cache into pages by `table`; unmapped rows hold NaN."""
    nan = np.uint16(0x7FC0) if x.dtype == np.uint16 else np.float32(np.nan)
    pool = np.full((n_pages, page) + x.shape[1:], nan, dtype=x.dtype)
    for i, pg in enumerate(table):
        blk = x[i * page:(i + 1) * page]
        pool[pg, :len(blk)] = blk
    return pool


class Paged:
    """One layer's cache as a paged pool, with its descriptor."""

    def __init__(self, w, L, page, seed):
        table, n_pages = page_table(w.n_ctx, page, np.random.default_rng(seed))
        self.k = to_dev(page_pool(L["k"], page, table, n_pages))
        self.v = to_dev(page_pool(L["v"], page, table, n_pages))
        self.table = torch.from_numpy(table).to(DEV)
        self.kv = api.kv_desc_paged(self.k, self.v, self.table, w.n_ctx, w.n_q_heads)
        t = np.arange(w.n_ctx)
        self.rows = torch.from_numpy(table[t // page].astype(np.int64) * page + t % page).to(DEV)

    def logical(self, pool):
        """The logical [n_ctx, H, d] cache a pool holds."""
        return pool.reshape((-1,) + tuple(pool.shape[2:]))[self.rows]


def score_all(w, kv, q, img, norm, vnorm_in=None):
    nv = w.n_vis
    f32 = dict(dtype=torch.float32, device=DEV)
    out = {x: torch.zeros(nv, **f32) for x in ("a", "v", "s", "A")}
    out["lse"] = torch.zeros((w.n_q, w.n_q_heads), **f32)
    api.conduit_score(kv, q, w.q_pos0, img, out["s"], out["A"], norm=norm, row_lse_out=out["lse"],
                      a_out=out["a"], vnorm_out=out["v"], vnorm_in=vnorm_in)
    torch.cuda.synchronize()
    return out


PAGED = [(c, p) for c in sorted(CASES) for p in (64, 256, 1024)] + [("cfg4_16k", 256)]


@pytest.mark.parametrize("case,page", PAGED, ids=[f"{c}-p{p}" for c, p in PAGED])
def test_paged_cache_bit_identical_to_contiguous(case, page):
    w = W.config(4) if case == "cfg4_16k" else CASES[case]()
    L = w.layer(0, text=True)
    img = api.ImageTable(w.img_pos, w.img_off)
    q = to_dev(L["q"])
    kc, vc = to_dev(L["k"]), to_dev(L["v"])
    flat = api.kv_desc(kc, vc, w.n_q_heads)
    pg = Paged(w, L, page, seed=page + len(case))
    # scoring (both normalisations), value-norm table
    for norm in (api.NORM_CAUSAL_ROW, api.NORM_VISUAL_ONLY):
        a = score_all(w, flat, q, img, norm)
        b = score_all(w, pg.kv, q, img, norm)
        for key in a:
            assert np.array_equal(bits(a[key]), bits(b[key])), f"score {key} (norm {norm})"
    ta = torch.empty(w.n_vis, dtype=torch.float32, device=DEV)
    tb = torch.empty_like(ta)
    api.conduit_value_norms(flat, img, ta)
    api.conduit_value_norms(pg.kv, img, tb)
    torch.cuda.synchronize()
    assert np.array_equal(bits(ta), bits(tb)), "value norms"
    # merge + refresh over selected and text rows
    sel = selection(w, page)
    rows, kn, vn, qn = recompute_inputs(w, L, sel)
    ra = run_recompute(w, flat, rows, kn, vn, qn)
    rb = run_recompute(w, pg.kv, rows, kn, vn, qn)
    for key in ra:
        assert np.array_equal(bits(ra[key]), bits(rb[key])), f"recompute {key}"
    assert np.array_equal(bits(pg.logical(pg.k)), bits(kc)), "merged K"
    assert np.array_equal(bits(pg.logical(pg.v)), bits(vc)), "merged V"
