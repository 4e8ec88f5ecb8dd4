"""Refresh attention on the GPU (conduit_refresh_attn) over the merged cache,
against the CPU oracle."""
import numpy as np
import pytest
import torch

from oracle import conduit_oracle as O
from paper_2609_05821_amd import api, workloads as W
from tests.gpu_helpers import (DEV, assert_attention, assert_scores, bits, oracle_refresh_rows, to_dev,
                               to_f64)

pytestmark = pytest.mark.gpu


def run_refresh(w, L, sel):
    P = w.vis_positions()
    kc, vc = to_dev(L["k"]), to_dev(L["v"])
    kv = api.kv_desc(kc, vc, w.n_q_heads)
    pos = torch.from_numpy(P[sel].astype(np.int32)).to(DEV)
    k = len(sel)
    api.conduit_scatter_kv(kv, pos, to_dev(L["k_star"][sel]), to_dev(L["v_star"][sel]))
    q_sel = to_dev(L["q_star"][sel])
    out = torch.empty((k, w.n_q_heads, w.head_dim), dtype=q_sel.dtype, device=DEV)
    lse = torch.empty((k, w.n_q_heads), dtype=torch.float32, device=DEV)
    api.conduit_refresh_attn(kv, q_sel, pos, out, lse_out=lse)
    torch.cuda.synchronize()
    return out, lse, kc, vc


def check(w, L, sel, rows=None):
    out, lse, kc, vc = run_refresh(w, L, sel)
    P = w.vis_positions()
    km, vm, o_ref, lse_ref = oracle_refresh_rows(L["k"], L["v"], P[sel], L["k_star"][sel], L["v_star"][sel],
                                                 L["q_star"][sel], range(len(sel)) if rows is None else rows)
    r = slice(None) if rows is None else np.asarray(rows)
    assert_attention(to_f64(out)[r], o_ref[r], w.dtype, what="O")
    assert_scores(to_f64(lse)[r], lse_ref[r], what="lse")
    np.testing.assert_array_equal(to_f64(kc), km)
    np.testing.assert_array_equal(to_f64(vc), vm)
    return out


CASES = {
    "cfg1_fp32_mha": lambda: W.config(1),
    "cfg2_bf16_gqa": lambda: W.config(2),
    "ragged_bf16_gqa7": lambda: W.custom(1, 28, 4, 128, 19, 13, [37, 250, 301], 5, "bf16", n_sinks=6,
                                         n_relevant=1, seed=3),
    "ragged_bf16_d64_gqa4": lambda: W.custom(1, 8, 2, 64, 40, 7, [100, 33], 3, "bf16", seed=4),
    "ragged_bf16_mha": lambda: W.custom(1, 4, 4, 128, 9, 1, [70], 0, "bf16", seed=5),
    "ragged_fp32_d128_gqa2": lambda: W.custom(1, 4, 2, 128, 5, 3, [20, 45, 11], 2, "f32", seed=6),
}


@pytest.mark.parametrize("pattern", ["random", "clustered", "tail"])
@pytest.mark.parametrize("case", sorted(CASES))
def test_refresh_matches_oracle(case, pattern):
    w = CASES[case]()
    L = w.layer(0)
    rng = np.random.default_rng(len(case) * 7 + len(pattern))
    nv = w.n_vis
    k = max(1, nv // 10)
    if pattern == "random":
        sel = np.sort(rng.choice(nv, size=k, replace=False))
    elif pattern == "clustered":
        start = int(rng.integers(0, nv - k + 1))
        sel = np.arange(start, start + k)
    else:
        sel = np.arange(nv - k, nv)
    check(w, L, sel)


@pytest.mark.parametrize("case", ["ragged_bf16_gqa7", "cfg1_fp32_mha", "ragged_bf16_d64_gqa4"])
def test_full_budget_equals_full_prefill(case):
    """100% budget: every visual row is fresh, so each refreshed row equals the
    dense causal attention row of a full prefill of the layer."""
    w = CASES[case]()
    L = w.layer(0)
    sel = np.arange(w.n_vis)
    out, _, kc, vc = run_refresh(w, L, sel)
    P = w.vis_positions()
    full_k, full_v = O.to_f64(L["k"]), O.to_f64(L["v"])
    full_k[P] = O.to_f64(L["k_star"])
    full_v[P] = O.to_f64(L["v_star"])
    q_full = np.zeros((w.n_ctx, w.n_q_heads, w.head_dim))
    q_full[P] = O.to_f64(L["q_star"])
    dense, _ = O.refresh_attention(q_full, full_k, full_v, np.arange(w.n_ctx), rows=list(P))
    assert_attention(to_f64(out), dense[P], w.dtype, what="O vs full prefill")


def test_refresh_16k_workload_every_row():
    """The 16,384-visual-token layer at a 10% budget in the benchmark's launch
    shape; every one of the 1,638 rows checked by the oracle."""
    w = W.config(4)
    L = w.layer(0)
    rng = np.random.default_rng(44)
    k = w.budgets["10%"]
    # selection shaped like the method's: concentrated in three relevant images
    rel = w.shared()["relevant"]
    pool = np.concatenate([np.arange(w.img_off[j], w.img_off[j + 1]) for j in rel])
    sel = np.sort(np.concatenate([rng.choice(pool, size=k // 2, replace=False),
                                  rng.choice(np.setdiff1d(np.arange(w.n_vis), pool), size=k - k // 2,
                                             replace=False)]))
    check(w, L, sel)


@pytest.mark.parametrize("k", [2400, 3000])
def test_refresh_many_blocks_short_context(k):
    """More pair blocks than the persistent grid takes per round (k * 7 / 256 >
    64 blocks per KV head): the plan then aims at two items per block and KV
    head, so even short causal ranges are cut into splits and merged.  Every
    row is checked by the oracle."""
    w = W.custom(1, 28, 4, 128, 8, 96, [1024, 1024, 1024, 1024], 16, "bf16", n_relevant=1, seed=71)
    L = w.layer(0)
    rng = np.random.default_rng(k)
    sel = np.sort(rng.choice(w.n_vis, size=k, replace=False))
    check(w, L, sel)


def test_refresh_is_deterministic():
    w = CASES["ragged_bf16_gqa7"]()
    L = w.layer(0)
    sel = np.arange(0, w.n_vis, 7)
    o1, l1, _, _ = run_refresh(w, L, sel)
    o2, l2, _, _ = run_refresh(w, L, sel)
    np.testing.assert_array_equal(bits(o1), bits(o2))
    np.testing.assert_array_equal(bits(l1), bits(l2))


def test_split_merge_is_deterministic_at_16k():
    """The 16k-token multi-image workload at its 10% budget: nearly every pair
    block is cut into several key splits.  Three calls give the same bits (the
    split merge sums in split order, no atomics), and a few merged rows match
    the oracle."""
    w = W.config(4, n_layers=1)
    L = w.layer(0)
    k = w.budgets["10%"]
    rng = np.random.default_rng(61)
    sel = np.sort(rng.choice(w.n_vis, size=k, replace=False))
    runs = [run_refresh(w, L, sel) for _ in range(3)]
    for o, l, _, _ in runs[1:]:
        np.testing.assert_array_equal(bits(o), bits(runs[0][0]))
        np.testing.assert_array_equal(bits(l), bits(runs[0][1]))
    check(w, L, sel, rows=[0, k // 3, k - 1])


def test_zero_budget_refresh_enqueues_nothing():
    w = W.config(2)
    L = w.layer(0, fresh=False)
    kc, vc = to_dev(L["k"]), to_dev(L["v"])
    kv = api.kv_desc(kc, vc, w.n_q_heads)
    empty = torch.zeros(0, dtype=torch.int32, device=DEV)
    out = torch.full((1, w.n_q_heads, w.head_dim), 3.0, dtype=torch.bfloat16, device=DEV)
    api.conduit_refresh_attn(kv, kc[:0].view(0, 1, 1), empty, out)
    torch.cuda.synchronize()
    assert (to_f64(out) == 3.0).all()


def test_kernel_timing_records_each_launch():
    """conduit_profile_*: while enabled, the refresh call's three bf16 launches
    (plan, attention, split merge) are recorded with positive durations, and
    the result equals the untimed call's bit for bit."""
    w = CASES["ragged_bf16_gqa7"]()
    L = w.layer(0)
    sel = np.arange(0, w.n_vis, 3)
    out_plain, _, _, _ = run_refresh(w, L, sel)
    api.profile_enable(True)
    out_timed, _, _, _ = run_refresh(w, L, sel)
    api.profile_enable(False)
    recs = api.profile_records()
    names = [n for n, _ in recs]
    assert names[-3:] == ["attn_plan", "attn_values", "attn_merge"], names
    assert "scatter" in names
    assert all(ms > 0 for _, ms in recs)
    assert np.array_equal(bits(out_plain), bits(out_timed))
    api.profile_enable(True)  # enabling clears the record
    assert api.lib().conduit_profile_count() == 0
    api.profile_enable(False)


@pytest.mark.parametrize("norms", [(300.0,), (300.0, 3000.0)], ids=["one_jump", "two_jumps"])
def test_refresh_large_logit_jumps(norms):
    """Keys far larger than the rest, placed at separator positions after the
    first images: for rows that see them, a later key tile's maximum exceeds
    the reference maximum taken from the split's first keys by far more than
    2^32, so the attention restarts those items (twice for two jumps).  Every
    row is checked by the oracle."""
    w = W.custom(1, 28, 4, 128, 8, 64, [512, 512, 512, 512], 16, "bf16", seed=81)
    L = w.layer(0)
    text = O.text_positions(w.n_ctx, w.img_pos, w.img_off)
    rng = np.random.default_rng(82)
    for j, nrm in enumerate(norms):
        p = int(w.img_pos[1 + j]) - 1  # the separator token just before image 1 + j
        assert p in set(text.tolist())
        u = rng.standard_normal((w.n_kv_heads, w.head_dim))
        u /= np.linalg.norm(u, axis=1, keepdims=True)
        L["k"][p] = w._cast((nrm * u).astype(np.float32))
    sel = np.sort(rng.choice(w.n_vis, size=240, replace=False))
    check(w, L, sel)


@pytest.mark.parametrize("case", ["ragged_bf16_gqa7", "ragged_bf16_d64_gqa4", "cfg1_fp32_mha", "cfg4_16k"])
def test_merge_refresh_equals_separate_calls(case):
    """conduit_merge_refresh_attn (the plan and the merge in one launch for
    bf16) gives the merged cache, O and the LSE of conduit_scatter_kv followed
    by conduit_refresh_attn, bit for bit; and O matches the oracle."""
    w = W.config(4) if case == "cfg4_16k" else CASES[case]()
    L = w.layer(0)
    rng = np.random.default_rng(len(case))
    k = max(1, w.n_vis // 10)
    sel = np.sort(rng.choice(w.n_vis, size=k, replace=False))
    out_s, lse_s, kc_s, vc_s = run_refresh(w, L, sel)
    P = w.vis_positions()
    kc, vc = to_dev(L["k"]), to_dev(L["v"])
    kv = api.kv_desc(kc, vc, w.n_q_heads)
    pos = torch.from_numpy(P[sel].astype(np.int32)).to(DEV)
    q_sel = to_dev(L["q_star"][sel])
    out = torch.empty_like(out_s)
    lse = torch.empty_like(lse_s)
    api.conduit_merge_refresh_attn(kv, pos, to_dev(L["k_star"][sel]), to_dev(L["v_star"][sel]), q_sel, out,
                                   lse_out=lse)
    torch.cuda.synchronize()
    for a, b in ((out, out_s), (lse, lse_s), (kc, kc_s), (vc, vc_s)):
        np.testing.assert_array_equal(bits(a), bits(b))
    rows = range(k) if case != "cfg4_16k" else range(0, k, 13)
    _, _, o_ref, _ = oracle_refresh_rows(L["k"], L["v"], P[sel], L["k_star"][sel], L["v_star"][sel],
                                         L["q_star"][sel], rows)
    r = np.asarray(list(rows))
    assert_attention(to_f64(out)[r], o_ref[r], w.dtype, what="O")
