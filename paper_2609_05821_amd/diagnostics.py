"""Synthetic diagnostic harness for selection rules (Eq. 3; App. D.1, D.3).

For a generated layer it compares refresh sets chosen by several rules at a
series of refresh ratios, by the residual value-write error they leave:

  * projected error (App. D.3): stale visual values set to zero, residual at
    the final span query, summed over query heads (the concatenated layer
    output with the identity output map);
  * isotropic Monte Carlo estimate (App. D.1): mean over M samples, every
    span row and query head.

Rules: random (seeded), TopK(||V||), TopK(RMS attention), TopK(RMS attention
x ||V||) and the deployed composite rule (mean attention x ||V||, image
reweighting with lambda).  Scores, selections and residuals all come from the
library's kernels; the host draws the random baseline, picks the rule inputs
and forms the ratios error(baseline) / error(rule).
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np
import torch

from . import api

RATIOS = ((5, 100), (10, 100), (20, 100), (30, 100), (50, 100))
RULES = ("random", "vnorm", "rms_attention", "rms_attention_x_vnorm", "composite")


def rule_masks(kv: api.KV, q: torch.Tensor, q_pos0: int, img: api.ImageTable, k: int,
               scores: Dict[str, torch.Tensor], seed: int, lam: float = 1.0) -> Dict[str, torch.Tensor]:
    """Refresh masks [N_vis] uint8 of every rule for budget k."""
    n_vis = img.n_vis
    dev = q.device
    out = {}
    rng = np.random.default_rng(seed)
    rnd = np.zeros(n_vis, np.uint8)
    rnd[rng.choice(n_vis, size=k, replace=False)] = 1
    out["random"] = torch.from_numpy(rnd).to(dev)
    idx = torch.empty(max(k, 1), dtype=torch.int32, device=dev)
    pos = torch.empty_like(idx)
    shat = torch.empty(n_vis, dtype=torch.float32, device=dev)
    plan = {
        "vnorm": (scores["vnorm"], scores["vnorm"], 0.0, api.RANK_COMPOSITE),
        "rms_attention": (scores["s_rms"], scores["a_rms"], 0.0, api.RANK_ATTENTION),
        "rms_attention_x_vnorm": (scores["s_rms"], scores["a_rms"], 0.0, api.RANK_COMPOSITE),
        "composite": (scores["s_mean"], scores["a_mean"], lam, api.RANK_COMPOSITE),
    }
    for name, (s, a, lm, rule) in plan.items():
        mask = torch.empty(n_vis, dtype=torch.uint8, device=dev)
        api.conduit_select_topk(s, a, 1, img, lm, k, idx, pos, mask_out=mask, shat_out=shat, rule=rule)
        out[name] = mask
    return out


def layer_scores(kv: api.KV, q: torch.Tensor, q_pos0: int, img: api.ImageTable) -> Dict[str, torch.Tensor]:
    """RMS and mean scoring passes of one layer (the rules' inputs) and the
    row log-sum-exp."""
    n_vis, dev = img.n_vis, q.device
    f = lambda *shape: torch.zeros(shape, dtype=torch.float32, device=dev)
    sc = {"s_rms": f(n_vis), "a_rms": f(n_vis), "vnorm": f(n_vis), "s_mean": f(n_vis),
          "a_mean": f(n_vis), "lse": f(q.shape[0], kv.n_q_heads)}
    api.conduit_score(kv, q, q_pos0, img, sc["s_rms"], sc["a_rms"], agg=api.AGG_RMS,
                      row_lse_out=sc["lse"], vnorm_out=sc["vnorm"])
    api.conduit_score(kv, q, q_pos0, img, sc["s_mean"], sc["a_mean"], agg=api.AGG_MEAN)
    return sc


def rule_errors(kv: api.KV, q: torch.Tensor, q_pos0: int, img: api.ImageTable,
                z: Optional[torch.Tensor], ratios: Sequence = RATIOS, kappa: float = 0.5,
                lam: float = 1.0, seed: int = 0) -> dict:
    """Projected error and isotropic estimate of every rule at every ratio,
    and the reductions against random and TopK(||V||) selection.

    The library returns one residual per (sample, span row, query head).  The
    two reductions over those entries are harness arithmetic on the host, in
    float64 after the copy back: the projected error of App. D.3 sums the
    final span row's heads, and the isotropic estimate of App. D.1 is the mean
    over samples, rows and heads.  They are a few thousand additions per rule
    and ratio and are not part of the refresh step."""
    n_q = q.shape[0]
    sc = layer_scores(kv, q, q_pos0, img)
    q_last = q[n_q - 1:].contiguous()
    lse_last = sc["lse"][n_q - 1:].contiguous()
    dev = q.device
    res = {"ratios": [n / d for n, d in ratios], "budgets": [], "projected": {r: [] for r in RULES},
           "iso": {r: [] for r in RULES}}
    err_p = torch.empty((1, 1, kv.n_q_heads), dtype=torch.float32, device=dev)
    err_i = None if z is None else torch.empty((z.shape[0], n_q, kv.n_q_heads), dtype=torch.float32,
                                               device=dev)
    for ri, (num, den) in enumerate(ratios):
        k = api.conduit_budget(img.n_vis, num, den)
        res["budgets"].append(k)
        masks = rule_masks(kv, q, q_pos0, img, k, sc, seed=seed * 1000 + ri, lam=lam)
        for name in RULES:
            api.conduit_residual_error(kv, q_last, q_pos0 + n_q - 1, img, lse_last, masks[name], err_p)
            # host-side harness reduction (App. D.3): sum over the final row's heads
            res["projected"][name].append(float(err_p.cpu().numpy().astype(np.float64).sum()))
            if err_i is not None:
                api.conduit_residual_error(kv, q, q_pos0, img, sc["lse"], masks[name], err_i, z=z,
                                           kappa=kappa)
                # host-side harness reduction (App. D.1): mean over samples, rows, heads
                res["iso"][name].append(float(err_i.cpu().numpy().astype(np.float64).mean()))
    for est in ("projected", "iso"):
        e = res[est]
        if not e["random"]:
            continue
        res[f"{est}_reduction_vs_random"] = {
            r: [b / x if x > 0 else float("inf") for b, x in zip(e["random"], e[r])] for r in RULES}
        res[f"{est}_reduction_vs_vnorm"] = {
            r: [b / x if x > 0 else float("inf") for b, x in zip(e["vnorm"], e[r])] for r in RULES}
    return res
