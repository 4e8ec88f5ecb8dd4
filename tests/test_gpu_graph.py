"""The refresh step captured in a HIP graph: every replay, with eager steps
run between the replays, reproduces the eager outputs bit for bit (no call on
the path records anything a replay would not repeat)."""
import numpy as np
import pytest
import torch

from paper_2609_05821_amd import api, workloads as W
from tests.gpu_helpers import DEV, to_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg", [2, 4])
def test_graph_replays_equal_eager(cfg):
    w = W.config(cfg)
    L = w.layer(0)
    kc, vc, q = to_dev(L["k"]), to_dev(L["v"]), to_dev(L["q"])
    k_pristine, v_pristine = kc.clone(), vc.clone()
    img = api.ImageTable(w.img_pos, w.img_off)
    k = list(w.budgets.values())[0]
    step = api.RefreshStep([{"k": kc, "v": vc, "q": q}], w.n_q_heads, w.q_pos0, img, k, lam=1.0,
                           device=DEV)
    kv = step.kvs[0]
    step.score_and_select()
    torch.cuda.synchronize()
    idx = step.idx[:k].cpu().numpy()
    k_new, v_new = to_dev(np.ascontiguousarray(L["k_star"][idx])), to_dev(np.ascontiguousarray(L["v_star"][idx]))
    q_sel = to_dev(np.ascontiguousarray(L["q_star"][idx]))
    pos, out, lse = step.pos[:k], step.out[0][:k], step.lse[0][:k]

    def one_step():
        api.conduit_score(kv, q, w.q_pos0, img, step.s_acc, step.a_acc, ws=step.ws_score)
        api.conduit_select_topk(step.s_acc, step.a_acc, 1, img, 1.0, k, step.idx, step.pos,
                                mask_out=step.mask, shat_out=step.shat, c_out=step.c)
        api.conduit_scatter_kv(kv, pos, k_new, v_new)
        api.conduit_refresh_attn(kv, q_sel, pos, out, lse_out=lse, ws=step.ws_refresh)

    def restore():
        kc.copy_(k_pristine)
        vc.copy_(v_pristine)

    one_step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (out, lse, step.idx, step.mask, step.shat, kc, vc)]
    restore()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        one_step()
    torch.cuda.synchronize()
    for _ in range(3):
        restore()
        graph.replay()
        torch.cuda.synchronize()
        got = (out, lse, step.idx, step.mask, step.shat, kc, vc)
        for name, a, b in zip(("out", "lse", "idx", "mask", "shat", "k", "v"), got, ref):
            assert torch.equal(a, b), name
        restore()
        one_step()  # eager work between replays
        torch.cuda.synchronize()
