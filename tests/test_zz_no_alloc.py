"""conduit_score_noalloc (the scoring pass on the library's fixed device
scratch) against conduit_score with a caller workspace, through the C ABI:
two calls in a row, the second on a smaller input, then an accumulating call.
The two entry points run the same kernels, so their outputs must agree bit for
bit; the smaller case is also held to the oracle's score bar (1e-4 relative)."""
import numpy as np
import pytest
import torch

from oracle import conduit_oracle as O
from paper_2609_05821_amd import api, workloads as W
from tests.gpu_helpers import DEV, assert_scores, bits, to_dev, to_f64

pytestmark = pytest.mark.gpu


def _outputs(w):
    f32 = dict(dtype=torch.float32, device=DEV)
    return {"s": torch.full((w.n_vis,), 7.0, **f32), "a": torch.full((w.n_vis,), 7.0, **f32),
            "a_out": torch.zeros(w.n_vis, **f32), "v_out": torch.zeros(w.n_vis, **f32),
            "lse": torch.zeros((w.n_q, w.n_q_heads), **f32)}


def _run(fn, w, kv, q, img, out, accumulate=False, norm=O.NORM_CAUSAL_ROW):
    fn(kv, q, w.q_pos0, img, out["s"], out["a"], accumulate=accumulate, norm=norm,
       row_lse_out=out["lse"], a_out=out["a_out"], vnorm_out=out["v_out"])


def _case(w):
    L = w.layer(0, fresh=False)
    k, v, q = (to_dev(L[x]) for x in ("k", "v", "q"))
    return L, k, v, q, api.kv_desc(k, v, w.n_q_heads), api.ImageTable(w.img_pos, w.img_off)


@pytest.mark.parametrize("norm", [O.NORM_CAUSAL_ROW, O.NORM_VISUAL_ONLY], ids=["causal", "visual"])
def test_noalloc_matches_workspace_entry_point(norm):
    big = W.config(4)        # 16 images x 1,024 visual tokens, 128 span rows
    small = W.config(2)      # one image of 1,024 visual tokens, 64 span rows
    for w in (big, small):   # the second call runs on a smaller input
        print(f"noalloc case n_vis={w.n_vis} n_q={w.n_q} norm={norm}", flush=True)
        Lnp, k, v, q, kv, img = _case(w)
        ref, got = _outputs(w), _outputs(w)
        _run(api.conduit_score, w, kv, q, img, ref, norm=norm)
        _run(api.conduit_score_noalloc, w, kv, q, img, got, norm=norm)
        torch.cuda.synchronize()
        for name in ref:
            assert np.array_equal(bits(got[name]), bits(ref[name])), f"{name} differs (n_vis {w.n_vis})"
        if w is small:
            a, vn, lse = O.score_layer(Lnp["q"], Lnp["k"], Lnp["v"], w.q_pos0, w.img_pos, w.img_off,
                                       norm=norm)
            assert_scores(to_f64(got["a_out"]), a, what="a")
            assert_scores(to_f64(got["v_out"]), vn, what="vnorm")
            assert_scores(to_f64(got["s"]), a * vn, what="s")
            assert_scores(to_f64(got["lse"]), lse, what="row lse")
        # layer accumulation on top of the previous call's sums
        _run(api.conduit_score, w, kv, q, img, ref, accumulate=True, norm=norm)
        _run(api.conduit_score_noalloc, w, kv, q, img, got, accumulate=True, norm=norm)
        torch.cuda.synchronize()
        for name in ("s", "a"):
            assert np.array_equal(bits(got[name]), bits(ref[name])), f"accumulated {name} differs"
