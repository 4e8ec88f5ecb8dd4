"""Cache merge on the GPU (conduit_scatter_kv): a bit copy, checked bitwise."""
import numpy as np
import pytest
import torch

from paper_2609_05821_amd import api, workloads as W
from tests.gpu_helpers import DEV, bits, to_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg", [1, 2, 4])
def test_scatter_bitwise(cfg):
    w = W.config(cfg)
    L = w.layer(0)
    P = w.vis_positions()
    k = w.budgets["10%"]
    rng = np.random.default_rng(cfg)
    sel = np.sort(rng.choice(w.n_vis, size=k, replace=False))
    kc, vc = to_dev(L["k"]), to_dev(L["v"])
    kv = api.kv_desc(kc, vc, w.n_q_heads)
    pos = torch.from_numpy(P[sel].astype(np.int32)).to(DEV)
    k_new, v_new = to_dev(L["k_star"][sel]), to_dev(L["v_star"][sel])
    k_old, v_old = torch.empty_like(k_new), torch.empty_like(v_new)
    api.conduit_scatter_kv(kv, pos, k_new, v_new, k_old, v_old)
    torch.cuda.synchronize()
    ek, ev = L["k"].copy(), L["v"].copy()
    ek[P[sel]] = L["k_star"][sel]
    ev[P[sel]] = L["v_star"][sel]
    np.testing.assert_array_equal(bits(kc), ek.view(bits(kc).dtype))
    np.testing.assert_array_equal(bits(vc), ev.view(bits(vc).dtype))
    np.testing.assert_array_equal(bits(k_old), L["k"][P[sel]].view(bits(k_old).dtype))
    np.testing.assert_array_equal(bits(v_old), L["v"][P[sel]].view(bits(v_old).dtype))
    # undo with the gathered rows: the cache returns to its original bytes
    api.conduit_scatter_kv(kv, pos, k_old, v_old)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bits(kc), L["k"].view(bits(kc).dtype))
    np.testing.assert_array_equal(bits(vc), L["v"].view(bits(vc).dtype))


def test_zero_budget_leaves_cache_untouched():
    w = W.config(2)
    L = w.layer(0, fresh=False)
    kc, vc = to_dev(L["k"]), to_dev(L["v"])
    before = (bits(kc).tobytes(), bits(vc).tobytes())
    kv = api.kv_desc(kc, vc, w.n_q_heads)
    empty = torch.zeros(0, dtype=torch.int32, device=DEV)
    api.conduit_scatter_kv(kv, empty, kc[:0], vc[:0])
    torch.cuda.synchronize()
    assert (bits(kc).tobytes(), bits(vc).tobytes()) == before


def test_strided_cache_scatter():
    w = W.custom(1, 8, 2, 64, 4, 3, [50], 0, "bf16", seed=2)
    L = w.layer(0)
    n_ctx = w.n_ctx
    big = torch.zeros((n_ctx, 3, 2, 64), dtype=torch.bfloat16, device=DEV)  # [tok][k|v|pad][h][d]
    big[:, 0] = to_dev(L["k"])
    big[:, 1] = to_dev(L["v"])
    kv = api.kv_desc(big[:, 0], big[:, 1], w.n_q_heads)
    P = w.vis_positions()
    sel = np.array([0, 7, 49])
    api.conduit_scatter_kv(kv, torch.from_numpy(P[sel].astype(np.int32)).to(DEV),
                           to_dev(L["k_star"][sel]), to_dev(L["v_star"][sel]))
    torch.cuda.synchronize()
    ek = L["k"].copy()
    ek[P[sel]] = L["k_star"][sel]
    np.testing.assert_array_equal(bits(big[:, 0]), ek)
    assert not bits(big[:, 2]).any()
