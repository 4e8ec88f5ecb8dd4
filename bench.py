"""Refresh-step benchmark on one MI355X.

    python bench.py [--steps K] [--warmup W] [--cfg 4] [--no-cpu]

One step is the whole refresh step of one layer: the scoring pass
(conduit_score), reweighting and global top-k (conduit_select_topk), then the
cache merge and the refresh attention of the selected rows in one call
(conduit_merge_refresh_attn; the per-call breakdown pass calls
conduit_scatter_kv and conduit_refresh_attn separately), all through the C
ABI.  Inputs are synthetic (seeded
generator), already resident in HBM.  Before each timed step a 512 MB scrub
buffer is written so the caches start cold; after it, the merged cache is
restored from a pristine copy.  Both happen outside the per-step HIP events.

Prints one JSON line.  `value` is visual tokens scored and refreshed per
second for the layer (N_vis / step time).  `roofline` covers the refresh
attention (the dominant call): algorithmic FLOPs 4 * H_q * d * sum_i (p_i + 1)
over its event-timed duration, against the bf16 dense MFMA peak; beside it the
rate a reference loop of independent MFMAs on random operands sustains on this
device in the same run (`sustained_mfma`).
`cpu_baseline` times the float64 CPU oracle on a bounded sample of the same
step on this host's cores.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "visual tokens scored+refreshed/s per layer; refresh-step ms @16k tokens, 10%"
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0


def sustained_mfma(dev):
    """Sustained bf16 matrix-core rate of this device on random operands: a
    loop of independent v_mfma_f32_32x32x16_bf16 at two waves per SIMD
    (paper_2609_05821_amd/csrc/ceiling.hip, built as libconduit_ceiling.so).
    A reference for the attention kernel's rate: under matrix-core load the
    shader clock drops below the one the nominal peak assumes."""
    import ctypes
    import torch
    path = os.path.join(ROOT, "paper_2609_05821_amd", "libconduit_ceiling.so")
    if not os.path.exists(path):
        return {"error": "libconduit_ceiling.so is not built"}
    lib = ctypes.CDLL(path)
    lib.conduit_ceiling_ops_bytes.restype = ctypes.c_int64
    lib.conduit_ceiling_ops_bytes.argtypes = [ctypes.c_int32]
    lib.conduit_ceiling_flop.restype = ctypes.c_double
    lib.conduit_ceiling_flop.argtypes = [ctypes.c_int32, ctypes.c_int32]
    lib.conduit_ceiling_mfma_bf16.restype = ctypes.c_int
    lib.conduit_ceiling_mfma_bf16.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                              ctypes.c_int32, ctypes.c_void_p]
    blocks, iters = 512, 20000
    gen = torch.Generator(device=dev).manual_seed(7)
    ops = torch.randn(lib.conduit_ceiling_ops_bytes(blocks) // 2, generator=gen, device=dev).to(torch.bfloat16)
    out = torch.empty(blocks * 256, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def launch():
        rc = lib.conduit_ceiling_mfma_bf16(ops.data_ptr(), out.data_ptr(), blocks, iters, stream.cuda_stream)
        if rc != 0:
            raise RuntimeError(f"ceiling kernel launch failed ({rc})")

    launch()
    torch.cuda.synchronize()
    times = []
    for _ in range(3):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        launch()
        b.record(stream)
        b.synchronize()
        times.append(a.elapsed_time(b))
    t = statistics.median(times)
    tflops = lib.conduit_ceiling_flop(blocks, iters) / (t * 1e-3) / 1e12
    return {"tflops": tflops, "ms": t, "frac_of_nominal": tflops / PEAK_BF16_TFLOPS,
            "what": "independent v_mfma_f32_32x32x16_bf16 on random bf16 operands, two waves per "
                    f"SIMD, median of 3 launches of {lib.conduit_ceiling_flop(blocks, iters) / 1e12:.1f} "
                    "TFLOP each (csrc/ceiling.hip)"}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--cfg", type=int, default=4, help="workload id (4 = 16k tokens, 10%%)")
    ap.add_argument("--budget", default="10%")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-scrub", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the supplementary measurements (variants, paged cache, text rows, "
                         "residual diagnostic): only the step kernels run, e.g. under a kernel trace")
    ap.add_argument("--cpu-row-stride", type=int, default=1,
                    help="CPU baseline refreshes every n-th selected row and scales by n")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the other workloads (single image, 28-layer multi-image, long document)")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "the benchmark measures one GPU (one process, one device); --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    from paper_2609_05821_amd import api, workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = W.config(args.cfg, n_layers=1)
    k = w.budgets[args.budget]
    t_gen = time.time()
    L = w.layer(0, text=True)
    t_gen = time.time() - t_gen

    def up(x):
        if x.dtype == np.uint16:
            return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(x).to(dev)

    kc, vc, q = up(L["k"]), up(L["v"]), up(L["q"])
    k_pristine, v_pristine = kc.clone(), vc.clone()
    img = api.ImageTable(w.img_pos, w.img_off)
    step = api.RefreshStep([{"k": kc, "v": vc, "q": q}], w.n_q_heads, w.q_pos0, img, k, lam=1.0,
                           device=dev)
    kv = step.kvs[0]

    # Selection once (untimed) to gather the fresh rows the recompute would produce.
    step.score_and_select()
    torch.cuda.synchronize()
    idx0 = step.idx[:k].clone()
    idx_np = idx0.cpu().numpy()
    fresh = {"k_new": up(np.ascontiguousarray(L["k_star"][idx_np])),
             "v_new": up(np.ascontiguousarray(L["v_star"][idx_np])),
             "q_sel": up(np.ascontiguousarray(L["q_star"][idx_np]))}
    pos_np = step.pos[:k].cpu().numpy().astype(np.int64)
    q_sel_np = np.ascontiguousarray(L["q_star"][idx_np])
    del L["q_star"]

    scrub = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    pos = step.pos[:k]
    out, lse = step.out[0][:k], step.lse[0][:k]

    def one_step(ev=None, split=False):
        # ev: 5 events; the step's two bracket it.  The step merges and
        # refreshes in one call (conduit_merge_refresh_attn: the refresh plan
        # and the merge in one launch); with split, the per-call breakdown
        # pass calls conduit_scatter_kv and conduit_refresh_attn instead, with
        # the three inner events separating the calls.
        if ev:
            ev[0].record(stream)
        api.conduit_score(kv, q, w.q_pos0, img, step.s_acc, step.a_acc, ws=step.ws_score)
        if ev and split:
            ev[1].record(stream)
        api.conduit_select_topk(step.s_acc, step.a_acc, 1, img, 1.0, k, step.idx, step.pos,
                                mask_out=step.mask, shat_out=step.shat, c_out=step.c, ws=step.ws_select)
        if ev and split:
            ev[2].record(stream)
        if split:
            api.conduit_scatter_kv(kv, pos, fresh["k_new"], fresh["v_new"])
            if ev:
                ev[3].record(stream)
            api.conduit_refresh_attn(kv, fresh["q_sel"], pos, out, lse_out=lse, ws=step.ws_refresh)
        else:
            api.conduit_merge_refresh_attn(kv, pos, fresh["k_new"], fresh["v_new"], fresh["q_sel"], out, lse_out=lse,
                                           ws=step.ws_refresh)
        if ev:
            ev[4].record(stream)

    def restore():
        kc.copy_(k_pristine)
        vc.copy_(v_pristine)

    for _ in range(args.warmup):
        one_step()
        restore()
    torch.cuda.synchronize()

    # Timed steps: events only around each step.
    step_events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    for i in range(args.steps):
        if not args.no_scrub:
            scrub.fill_(i & 0xFF)
        one_step(step_events[i])
        restore()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall

    # The same steps again with events between the calls (per-call times;
    # the extra events lengthen these steps slightly).
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    for i in range(args.steps):
        if not args.no_scrub:
            scrub.fill_(i & 0xFF)
        one_step(events[i], split=True)
        restore()
    torch.cuda.synchronize()

    # Second timed pass of the same steps with per-launch kernel timing (HIP
    # events recorded by the library around each launch, on this stream).
    api.profile_enable(True)
    for i in range(args.steps):
        if not args.no_scrub:
            scrub.fill_(i & 0xFF)
        one_step()
        restore()
    torch.cuda.synchronize()
    api.profile_enable(False)
    kern = {}
    for name, t in api.profile_records():
        kern.setdefault(name, []).append(t)
    kernels_ms = {name: {"calls_per_step": len(v) / args.steps, "mean": statistics.mean(v),
                         "p10": pct(v, 10), "p90": pct(v, 90)} for name, v in kern.items()}

    per = {"score": [], "select": [], "scatter": [], "refresh": [], "step": [], "step_with_call_events": []}
    for ev in events:
        per["score"].append(ev[0].elapsed_time(ev[1]))
        per["select"].append(ev[1].elapsed_time(ev[2]))
        per["scatter"].append(ev[2].elapsed_time(ev[3]))
        per["refresh"].append(ev[3].elapsed_time(ev[4]))
        per["step_with_call_events"].append(ev[0].elapsed_time(ev[4]))
    for ev in step_events:
        per["step"].append(ev[0].elapsed_time(ev[4]))
    ms_step = statistics.mean(per["step"])
    ms = {key: statistics.mean(v) for key, v in per.items()}
    med = {key: statistics.median(v) for key, v in per.items()}
    p10 = {key: pct(v, 10) for key, v in per.items()}
    p90 = {key: pct(v, 90) for key, v in per.items()}

    # Scoring with the row log-sum-exp supplied (the row-statistics pass is
    # skipped), and the same pass at n_q = 8 (bandwidth probe: far below the
    # MFMA ridge, so HBM-bound).
    lse_rows = torch.empty(w.n_q * w.n_q_heads, dtype=torch.float32, device=dev)
    api.conduit_score(kv, q, w.q_pos0, img, step.s_acc, step.a_acc, row_lse_out=lse_rows,
                      ws=step.ws_score)
    q8 = q[:8].contiguous()
    ws8 = torch.empty(api.score_workspace_bytes(kv, 8, img), dtype=torch.uint8, device=dev)

    def timed(fn):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * args.steps)]
        for _ in range(args.warmup):
            fn()
        out_ms = []
        for i in range(args.steps):
            if not args.no_scrub:
                scrub.fill_(i & 0xFF)
            ev[2 * i].record(stream)
            fn()
            ev[2 * i + 1].record(stream)
        torch.cuda.synchronize()
        out_ms = [ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(args.steps)]
        return {"mean": statistics.mean(out_ms), "p10": pct(out_ms, 10), "p90": pct(out_ms, 90)}

    score_lse_in = timed(lambda: api.conduit_score(kv, q, w.q_pos0, img, step.s_acc, step.a_acc,
                                                   row_lse_in=lse_rows, ws=step.ws_score))

    def one_step_lse_in():
        api.conduit_score(kv, q, w.q_pos0, img, step.s_acc, step.a_acc, row_lse_in=lse_rows,
                          ws=step.ws_score)
        api.conduit_select_topk(step.s_acc, step.a_acc, 1, img, 1.0, k, step.idx, step.pos,
                                mask_out=step.mask, shat_out=step.shat, c_out=step.c, ws=step.ws_select)
        api.conduit_merge_refresh_attn(kv, pos, fresh["k_new"], fresh["v_new"], fresh["q_sel"], out, lse_out=lse,
                                       ws=step.ws_refresh)

    def timed_restored(fn):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * args.steps)]
        for _ in range(args.warmup):
            fn()
            restore()
        for i in range(args.steps):
            if not args.no_scrub:
                scrub.fill_(i & 0xFF)
            ev[2 * i].record(stream)
            fn()
            ev[2 * i + 1].record(stream)
            restore()
        torch.cuda.synchronize()
        out_ms = [ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(args.steps)]
        return {"mean": statistics.mean(out_ms), "p10": pct(out_ms, 10), "p90": pct(out_ms, 90)}

    step_lse_in = timed_restored(one_step_lse_in)
    probe = timed(lambda: api.conduit_score(kv, q8, w.q_pos0, img, step.s_acc, step.a_acc, ws=ws8))
    tiny = torch.empty(1, dtype=torch.float32, device=dev)
    launch_floor = timed(lambda: tiny.fill_(0.0))

    # Selection must be the same every step (deterministic).
    assert torch.equal(step.idx[:k], idx0), "selection changed between steps"

    # Algorithmic work.
    H, d, hkv = w.n_q_heads, w.head_dim, w.n_kv_heads
    refresh_flops = 4.0 * H * d * float(np.sum(pos_np + 1))
    refresh_exps = H * float(np.sum(pos_np + 1))
    e = 2  # bf16 bytes
    score_bytes = (w.n_q * H * d * e + w.n_ctx * hkv * d * e + w.n_vis * hkv * d * e
                   + w.n_vis * 4 * 4)
    score_flops = 2.0 * d * H * sum(w.q_pos0 + i + 1 for i in range(w.n_q)) + \
        2.0 * d * H * w.n_q * w.n_vis
    scatter_bytes = 2 * 2 * k * hkv * d * e
    refresh_tflops = refresh_flops / (ms["refresh"] * 1e-3) / 1e12
    attn_ms = kernels_ms["attn_values"]["mean"]
    attn_tflops = refresh_flops / (attn_ms * 1e-3) / 1e12
    probe_bytes = (8 * H * d * e + w.n_ctx * hkv * d * e + w.n_vis * hkv * d * e + w.n_vis * 4 * 4)
    ceiling = sustained_mfma(dev)  # after the timed passes

    result = {
        "metric": METRIC,
        "value": w.n_vis / (ms_step * 1e-3),
        "unit": "visual tokens/s per layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic (seeded generator; no dataset or weights)",
        "config": {
            "workload": w.name + f", budget {args.budget} (k={k}), one layer",
            "cfg": args.cfg, "n_vis": w.n_vis, "n_ctx": w.n_ctx, "n_images": w.n_images,
            "n_q": w.n_q, "n_q_heads": H, "n_kv_heads": hkv, "head_dim": d, "k": k,
            "lambda": 1.0, "norm": "causal_row", "cold_cache_scrub": not args.no_scrub,
        },
        "roofline": {
            "kernel": "attn_bf16_kernel<128, true, 8, false> (refresh attention of conduit_refresh_attn)",
            "bound": "mfma",
            "achieved": attn_tflops,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": attn_tflops / PEAK_BF16_TFLOPS,
            "traffic": traffic_from_profile(),
            "algorithmic_flops_per_launch": refresh_flops,
            "avg_launch_ms": attn_ms,
            "timing": "HIP events around the kernel launch on its stream (library per-launch "
                      "timing), same steps as the timed region, second pass",
            "whole_call": {"ms": ms["refresh"], "tflops": refresh_tflops,
                           "note": "conduit_refresh_attn = plan + attention + split merge"},
            "sustained_mfma": ceiling,
            "frac_of_sustained": attn_tflops / ceiling["tflops"] if "tflops" in ceiling else None,
        },
        "per_call_ms_mean": ms,
        "per_call_ms_median": med,
        "per_call_ms_p10": p10,
        "per_call_ms_p90": p90,
        "kernels_ms": kernels_ms,
        "score_row_lse_in_ms": score_lse_in,
        "step_row_lse_in": {
            "ms": step_lse_in, "value": w.n_vis / (step_lse_in["mean"] * 1e-3),
            "note": "the same step with the span rows' log-sum-exp supplied to conduit_score (e.g. "
                    "from the model's own attention of the span): the row-statistics pass is skipped"},
        "bandwidth_probe": {
            "what": "conduit_score at n_q = 8 on the same cache (supplementary; not a benchmark "
                    "config): HBM-bound",
            "ms": probe, "algorithmic_bytes": probe_bytes,
            "gbs": probe_bytes / (probe["mean"] * 1e-3) / 1e9,
            "hbm_frac": probe_bytes / (probe["mean"] * 1e-3) / 1e9 / PEAK_HBM_GBS,
        },
        "launch_floor_ms": launch_floor,
        "provenance": provenance(),
        "score": {
            "algorithmic_bytes": score_bytes, "algorithmic_flops": score_flops,
            "gbs": score_bytes / (ms["score"] * 1e-3) / 1e9,
            "hbm_frac": score_bytes / (ms["score"] * 1e-3) / 1e9 / PEAK_HBM_GBS,
            "mfma_frac": score_flops / (ms["score"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
        },
        "scatter_gbs": scatter_bytes / (ms["scatter"] * 1e-3) / 1e9,
        "refresh_exps_per_s": refresh_exps / (ms["refresh"] * 1e-3),
        "wall_ms_per_step_incl_scrub_restore": t_wall / args.steps * 1e3,
        "gen_s": t_gen,
    }

    if not args.no_extras:
        # Variants on the same workload: the value-norm table (built once per
        # cache), scoring that reads the table instead of V, RMS aggregation, and
        # the attention-only and explicit-quota selection rules.
        table = torch.empty(w.n_vis, dtype=torch.float32, device=dev)
        quota = torch.empty(w.n_images, dtype=torch.int32, device=dev)
        variants_ms = {
            "value_norms": timed(lambda: api.conduit_value_norms(kv, img, table)),
            "score_vnorm_table": timed(lambda: api.conduit_score(kv, q, w.q_pos0, img, step.s_acc,
                                                                 step.a_acc, ws=step.ws_score,
                                                                 vnorm_in=table)),
            "score_rms": timed(lambda: api.conduit_score(kv, q, w.q_pos0, img, step.s_acc, step.a_acc,
                                                         ws=step.ws_score, agg=api.AGG_RMS)),
        }
        api.conduit_score(kv, q, w.q_pos0, img, step.s_acc, step.a_acc, ws=step.ws_score)
        for name, rule in (("select_attention", api.RANK_ATTENTION), ("select_explicit", api.RANK_EXPLICIT)):
            variants_ms[name] = timed(lambda rule=rule: api.conduit_select_topk(
                step.s_acc, step.a_acc, 1, img, 1.0, k, step.idx, step.pos, mask_out=step.mask,
                shat_out=step.shat, c_out=step.c, ws=step.ws_select, rule=rule, quota_out=quota))

        # Paged cache (256-token pages, shuffled pool) and the recompute with the
        # request's text rows in the same merge and attention launch.
        page = 256
        n_log = -(-w.n_ctx // page)
        table_np = np.random.default_rng(7).permutation(n_log + 8)[:n_log].astype(np.int32)
        table = torch.from_numpy(table_np).to(dev)
        tok = np.arange(w.n_ctx)
        rows_idx = torch.from_numpy(table_np[tok // page].astype(np.int64) * page + tok % page).to(dev)
        k_pool = torch.zeros(((n_log + 8) * page, w.n_kv_heads, w.head_dim), dtype=kc.dtype, device=dev)
        v_pool = torch.zeros_like(k_pool)
        k_pool[rows_idx] = k_pristine
        v_pool[rows_idx] = v_pristine
        kv_paged = api.kv_desc_paged(k_pool.view(n_log + 8, page, w.n_kv_heads, w.head_dim),
                                     v_pool.view(n_log + 8, page, w.n_kv_heads, w.head_dim), table,
                                     w.n_ctx, w.n_q_heads)
        text_np = w.text_positions()
        rows_all = torch.cat([pos, torch.from_numpy(text_np.astype(np.int32)).to(dev)])
        k_all = torch.cat([fresh["k_new"], up(L["k_text_star"])])
        v_all = torch.cat([fresh["v_new"], up(L["v_text_star"])])
        q_all = torch.cat([fresh["q_sel"], up(L["q_text_star"])])
        n_all = rows_all.numel()
        out_all = torch.empty((n_all, w.n_q_heads, w.head_dim), dtype=q_all.dtype, device=dev)
        ws_all = torch.empty(api.refresh_workspace_bytes(kv, n_all), dtype=torch.uint8, device=dev)
        variants_ms["score_paged256"] = timed(lambda: api.conduit_score(
            kv_paged, q, w.q_pos0, img, step.s_acc, step.a_acc, ws=step.ws_score))
        api.conduit_scatter_kv(kv_paged, pos, fresh["k_new"], fresh["v_new"])
        variants_ms["refresh_paged256"] = timed(lambda: api.conduit_refresh_attn(
            kv_paged, fresh["q_sel"], pos, out, lse_out=lse, ws=step.ws_refresh))
        variants_ms["recompute_with_text_rows"] = timed(lambda: (
            api.conduit_scatter_kv(kv, rows_all, k_all, v_all),
            api.conduit_refresh_attn(kv, q_all, rows_all, out_all, ws=ws_all)))
        restore()

        # The step captured once in a HIP graph and replayed (same kernels, same
        # buffers); replays, with eager steps between them, must reproduce the
        # eager outputs bit for bit before their time is reported.
        try:
            restore()
            one_step()
            torch.cuda.synchronize()
            ref = (out.clone(), lse.clone(), step.idx.clone(), kc.clone())
            restore()
            gstream = torch.cuda.Stream()
            gstream.wait_stream(stream)
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=gstream):
                one_step()
            torch.cuda.synchronize()
            restore()
            same = True
            for _ in range(3):
                graph.replay()
                torch.cuda.synchronize()
                same = same and all(torch.equal(a, b) for a, b in zip((out, lse, step.idx, kc), ref))
                restore()
                one_step()
                restore()
            torch.cuda.synchronize()
            graph_info = {"ms_per_step": timed(graph.replay), "replays_equal_eager": bool(same),
                          "note": "the timed step captured in a HIP graph (supplementary; value is eager)"}
            restore()
        except Exception as ex:  # noqa: BLE001 - reported, the eager figures stand
            graph_info = {"error": repr(ex)}

        # Residual-error diagnostic: the isotropic estimate (M = 5) of the step's
        # own 10% refresh set, timed, and the rule comparison table.
        from paper_2609_05821_amd import diagnostics as D
        n_samples = 5
        z_dev = up(W.iso_directions(w, 0, n_samples))
        err_iso = torch.empty((n_samples, w.n_q, w.n_q_heads), dtype=torch.float32, device=dev)
        ws_res = torch.empty(api.residual_workspace_bytes(kv, w.n_q, img, n_samples, True), dtype=torch.uint8,
                             device=dev)
        variants_ms["residual_iso_m5"] = timed(lambda: api.conduit_residual_error(
            kv, q, w.q_pos0, img, lse_rows, step.mask, err_iso, z=z_dev, ws=ws_res))
        diag = D.rule_errors(kv, q, w.q_pos0, img, z_dev, seed=0)
        del z_dev
        text_flops = refresh_flops + 4.0 * H * d * float(np.sum(text_np + 1))
        res_flops = 2.0 * w.n_q * H * w.n_vis * d * (1 + n_samples)   # S once, then one product per sample
        res_bytes = (n_samples + 2) * w.n_vis * hkv * d * e + w.n_q * H * d * e  # z, K and V rows, Q
        vnorm_bytes = w.n_vis * hkv * d * e + w.n_vis * 4
        score_table_bytes = score_bytes - w.n_vis * hkv * d * e + w.n_vis * 4
        result.update({
            "graph_replay": graph_info,
            "variants_ms": variants_ms,
            "recompute_with_text_rows": {
                "rows": n_all, "text_rows": int(len(text_np)),
                "algorithmic_flops": text_flops,
                "tflops_whole_call": text_flops / (variants_ms["recompute_with_text_rows"]["mean"] * 1e-3) / 1e12,
                "note": "merge + refresh attention of the selected rows and every text row, one launch each",
            },
            "residual_iso_m5": {
                "algorithmic_flops": res_flops, "algorithmic_bytes": res_bytes,
                "tflops": res_flops / (variants_ms["residual_iso_m5"]["mean"] * 1e-3) / 1e12,
                "gbs": res_bytes / (variants_ms["residual_iso_m5"]["mean"] * 1e-3) / 1e9,
                "note": "conduit_residual_error, isotropic estimator, M = 5, the step's 10% set, all span rows",
            },
            "diagnostics": diag,
            "paged": {"page_size": page, "pages": n_log + 8,
                      "note": "same workload with K/V in a shuffled pool of 256-token pages"},
            "variants_bytes": {
                "value_norms": vnorm_bytes,
                "value_norms_gbs": vnorm_bytes / (variants_ms["value_norms"]["mean"] * 1e-3) / 1e9,
                "score_vnorm_table": score_table_bytes,
                "score_vnorm_table_gbs": score_table_bytes /
                (variants_ms["score_vnorm_table"]["mean"] * 1e-3) / 1e9,
            },
        })

    del scrub, step, fresh
    torch.cuda.empty_cache()
    if not args.no_workloads:
        result["workloads"] = other_workloads(args, dev)
    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline(w, L, q_sel_np, idx_np, pos_np, k,
                                              args.cpu_row_stride)
    print(json.dumps(result))


def pct(v, q):
    """q-th percentile (nearest rank) of a list."""
    xs = sorted(v)
    return xs[min(len(xs) - 1, max(0, int(round(q / 100.0 * (len(xs) - 1)))))]


def source_digest(paths):
    """First 16 hex digits of the SHA-256 of the files' bytes, in order."""
    import hashlib
    h = hashlib.sha256()
    for path in paths:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


# Sources that decide the refresh kernel's code and tiling.
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2609_05821_amd", "csrc", f) for f in ("attn.hip", "common.h")]


def traffic_from_profile():
    """Bytes per launch of the refresh attention kernel between its L2s and the
    memory fabric, from the committed counter summary (read requests counted
    by size, 128 x RDREQ_128B + 64 x RDREQ_64B + 32 x RDREQ_32B, plus the
    WRITE_SIZE bytes); None when the summary is missing or was taken on another
    version of the kernel source."""
    path = os.path.join(ROOT, "profiles", "attn_values_16k_traffic.md")
    try:
        text = open(path).read()
    except OSError:
        return None
    import re
    m = re.search(r"```json\n(.*?)\n```", text, re.S)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("kernel_sources_sha256_16") != source_digest(KERNEL_SOURCES):
        return None
    return rec.get("traffic_bytes_per_launch")


def other_workloads(args, dev):
    """The other workloads, each step timed on this GPU (HIP events around
    the whole step, cold caches) beside its CPU oracle timing.

    A step is the refresh step of the workload: the scoring of every scored
    layer (conduit_score_layers: layer sums accumulated, up to 16 layers per
    launch), one conduit_select_topk, then the merge and refresh of every
    layer (conduit_scatter_kv_layers + conduit_refresh_attn_layers: up to 16
    layers per launch, one plan).  The 28-layer
    workloads hold 28 per-layer caches, span queries and fresh rows in device
    memory; their contents are one generated layer copied into each (so the
    selection is that of one layer; every layer still reads and writes its own
    buffers).  Throughput is visual tokens per second per layer:
    N_vis / (step time / layers)."""
    import torch

    from paper_2609_05821_amd import api, workloads as W

    stream = torch.cuda.current_stream()
    scrub = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    out = {}
    plan = [(1, ["10%", "10%-stated"], 1), (2, ["10%"], 1), (3, ["5%", "10%", "20%"], 28),
            (5, ["10%", "10%-stated"], 28)]
    for cfg, labels, n_layers in plan:
        w = W.config(cfg, n_layers=1)
        L = w.layer(0)

        def up(x):
            if x.dtype == np.uint16:
                return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)
            return torch.from_numpy(np.ascontiguousarray(x)).to(dev)

        k0, v0, q0 = up(L["k"]), up(L["v"]), up(L["q"])
        caches = [(k0, v0)] + [(k0.clone(), v0.clone()) for _ in range(n_layers - 1)]
        qs = [q0] + [q0.clone() for _ in range(n_layers - 1)]
        kvs = [api.kv_desc(kc, vc, w.n_q_heads) for kc, vc in caches]
        img = api.ImageTable(w.img_pos, w.img_off)
        f32 = dict(dtype=torch.float32, device=dev)
        s_acc, a_acc = torch.zeros(w.n_vis, **f32), torch.zeros(w.n_vis, **f32)
        shat, cj = torch.zeros(w.n_vis, **f32), torch.zeros(w.n_images, **f32)
        mask = torch.zeros(w.n_vis, dtype=torch.uint8, device=dev)
        ws_score = torch.empty(api.score_layers_workspace_bytes(kvs[0], w.n_q, img, n_layers), dtype=torch.uint8,
                               device=dev)
        ws_sel = torch.empty(max(1, int(api.lib().conduit_select_workspace_bytes(w.n_vis, w.n_images))),
                             dtype=torch.uint8, device=dev)
        entry = {"workload": w.name, "layers": n_layers, "n_vis": w.n_vis, "n_ctx": w.n_ctx,
                 "dtype": w.dtype, "budgets": {}}
        for label in labels:
            k = w.budgets[label]
            idx = torch.zeros(k, dtype=torch.int32, device=dev)
            pos = torch.zeros(k, dtype=torch.int32, device=dev)

            def score_select():
                # every layer's scoring in two launches per 16 layers, summed in layer order
                api.conduit_score_layers(kvs, qs, w.q_pos0, img, s_acc, a_acc, ws=ws_score)
                api.conduit_select_topk(s_acc, a_acc, n_layers, img, 1.0, k, idx, pos, mask_out=mask,
                                        shat_out=shat, c_out=cj, ws=ws_sel)

            score_select()
            torch.cuda.synchronize()
            idx_np = idx.cpu().numpy()
            pos_np = pos.cpu().numpy().astype(np.int64)
            kn, vn, qn = (up(L[x][idx_np]) for x in ("k_star", "v_star", "q_star"))
            k_new = [kn] + [kn.clone() for _ in range(n_layers - 1)]
            v_new = [vn] + [vn.clone() for _ in range(n_layers - 1)]
            q_sel = [qn] + [qn.clone() for _ in range(n_layers - 1)]
            pos_l = pos.long()
            stale = [(kc[pos_l].clone(), vc[pos_l].clone()) for kc, vc in caches]
            outs = [torch.empty((k, w.n_q_heads, w.head_dim), dtype=k0.dtype, device=dev) for _ in range(n_layers)]
            ws_ref = torch.empty(max(1, api.refresh_layers_workspace_bytes(kvs[0], k, n_layers)), dtype=torch.uint8,
                                 device=dev)

            def step_fn():
                score_select()
                if n_layers > 1:  # every layer's merge and refresh in a few launches
                    api.conduit_scatter_kv_layers(kvs, pos, k_new, v_new)
                    api.conduit_refresh_attn_layers(kvs, q_sel, pos, outs, ws=ws_ref)
                else:
                    api.conduit_scatter_kv(kvs[0], pos, k_new[0], v_new[0])
                    api.conduit_refresh_attn(kvs[0], q_sel[0], pos, outs[0], ws=ws_ref)

            def restore():
                for (kc, vc), (ks, vs) in zip(caches, stale):
                    kc[pos_l] = ks
                    vc[pos_l] = vs

            n_steps, n_warm = max(3, args.steps // 4), 2
            for _ in range(n_warm):
                step_fn()
                restore()
            torch.cuda.synchronize()
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * n_steps)]
            for i in range(n_steps):
                if not args.no_scrub:
                    scrub.fill_(i & 0xFF)
                ev[2 * i].record(stream)
                step_fn()
                ev[2 * i + 1].record(stream)
                restore()
            torch.cuda.synchronize()
            ms = [ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(n_steps)]
            assert torch.equal(pos[:k].long(), pos_l), "selection changed between steps"
            api.profile_enable(True)
            step_fn()
            torch.cuda.synchronize()
            api.profile_enable(False)
            restore()
            kern = {}
            for name, t in api.profile_records():
                kern.setdefault(name, []).append(t)
            ms_step = statistics.mean(ms)
            rec = {"k": k, "ms_per_step": ms_step, "p10": pct(ms, 10), "p90": pct(ms, 90), "steps": n_steps,
                   "value": w.n_vis / (ms_step * 1e-3 / n_layers),
                   "kernels_ms_per_step": {n: sum(v) for n, v in kern.items()}}
            if "attn_values" in kern:
                # one launch covers up to 16 layers: rate over the step's launches
                fl = 4.0 * w.n_q_heads * w.head_dim * float(np.sum(pos_np + 1))
                t_att = sum(kern["attn_values"])
                rec["refresh_kernel"] = {"algorithmic_flops_per_layer": fl, "launches": len(kern["attn_values"]),
                                         "ms_per_layer": t_att / n_layers,
                                         "tflops": fl * n_layers / (t_att * 1e-3) / 1e12,
                                         "frac_of_bf16_peak": fl * n_layers / (t_att * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}
            if not args.no_cpu and not (cfg == 5 and label != labels[0]):
                # (the long document's two budgets differ by one row: its CPU leg runs once)
                rec["cpu_baseline"] = cpu_workload(w, L, idx_np, pos_np, k, n_layers)
            entry["budgets"][label] = rec
            del k_new, v_new, q_sel, stale, outs, ws_ref, kn, vn, qn
        out[f"cfg{cfg}"] = entry
        del caches, qs, kvs, k0, v0, q0, L
        torch.cuda.empty_cache()
    return out


def cpu_workload(w, L, idx, pos, k, n_layers):
    """The float64 oracle on this host for one workload: scoring, reweighting,
    top-k and merge of one layer plus the refresh attention of its selected
    rows.  The single-image workloads run in full, with all host threads and
    again single-threaded; the 28-layer ones time one layer (the long
    document on a sample of span rows and refreshed rows, scaled) and report
    the step as 28 such layers, labelled as an extrapolation."""
    import threadpoolctl

    from oracle import conduit_oracle as O

    def run(score_rows, ref_stride):
        layer = {"q": L["q"][:score_rows], "k": L["k"], "v": L["v"]}
        t0 = time.perf_counter()
        O.select([layer], w.q_pos0, w.img_pos, w.img_off, k, lam=1.0)
        t1 = time.perf_counter()
        rows = list(range(0, k, ref_stride))
        O.refresh_layer(L["k"], L["v"], pos, L["k_star"][idx], L["v_star"][idx], L["q_star"][idx], rows=rows)
        t2 = time.perf_counter()
        return (t1 - t0) * (w.n_q / score_rows) + (t2 - t1) * (k / len(rows)), t1 - t0, t2 - t1, len(rows)

    info = threadpoolctl.threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info] or [1])
    if w.cfg_id == 5:
        score_rows, stride = 16, 64
    else:
        score_rows, stride = w.n_q, 1
    t_layer, ts, tr, nr = run(score_rows, stride)
    rec = {"value": w.n_vis / t_layer, "unit": "visual tokens/s per layer", "cores": threads,
           "kind": "oracle", "seconds_per_layer": t_layer,
           "sample": (f"one layer: scoring of {score_rows} of {w.n_q} span rows ({ts:.2f} s"
                      + (f", scaled x{w.n_q / score_rows:.0f}" if score_rows < w.n_q else "")
                      + f"), reweighting, top-k and merge, refresh attention of {nr} of {k} rows "
                      f"({tr:.2f} s" + (f", scaled x{k / nr:.1f}" if nr < k else "") + "); float64 numpy")}
    if n_layers > 1:
        rec["seconds_per_step_extrapolated"] = t_layer * n_layers
        rec["note"] = f"per-layer rate; the {n_layers}-layer step is extrapolated as {n_layers} x one layer"
    if w.n_vis <= 1024:
        with threadpoolctl.threadpool_limits(1):
            t1, _, _, _ = run(score_rows, stride)
        rec["single_thread"] = {"value": w.n_vis / t1, "seconds_per_layer": t1, "cores": 1}
    return rec


def provenance():
    import torch

    from paper_2609_05821_amd import build as B
    rocm = ""
    try:
        rocm = open("/opt/rocm/.info/version").read().strip()
    except OSError:
        pass
    flags, skip = [], False
    for f in B.FLAGS:  # drop include paths (machine-specific)
        if skip or f.startswith("/"):
            skip = False
            continue
        if f == "-I":
            skip = True
            continue
        flags.append(f)
    return {"rocm": rocm, "torch": torch.__version__,
            "device": torch.cuda.get_device_name(0),
            "arch": getattr(torch.cuda.get_device_properties(0), "gcnArchName", ""),
            "hipcc_flags": " ".join(flags)}


def cpu_baseline(w, L, q_sel, idx, pos, k, stride):
    """The float64 oracle on this host: full scoring, reweighting, top-k and
    merge of the layer, and the refresh attention of every `stride`-th selected
    row, scaled by `stride` (rows are spread evenly over the positions)."""
    import threadpoolctl

    from oracle import conduit_oracle as O

    info = threadpoolctl.threadpool_info()
    blas_threads = max([i.get("num_threads", 1) for i in info] or [1])
    cores = len(os.sched_getaffinity(0))
    layer = {"q": L["q"], "k": L["k"], "v": L["v"]}
    t0 = time.perf_counter()
    O.select([layer], w.q_pos0, w.img_pos, w.img_off, k, lam=1.0)
    t1 = time.perf_counter()
    rows = list(range(0, k, stride))
    t2 = time.perf_counter()
    O.refresh_layer(L["k"], L["v"], pos, L["k_star"][idx], L["v_star"][idx], q_sel, rows=rows)
    t3 = time.perf_counter()
    t_step = (t1 - t0) + (t3 - t2) * (k / len(rows))
    cpu_model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": w.n_vis / t_step, "unit": "visual tokens/s per layer", "cores": blas_threads,
            "kind": "oracle",
            "sample": f"one layer of the same workload: full scoring pass, reweighting, top-k and "
                      f"merge ({t1 - t0:.2f} s), refresh attention of {len(rows)} of {k} selected "
                      f"rows (every {stride}th, {t3 - t2:.2f} s) scaled x{k / len(rows):.2f}; "
                      f"float64 numpy",
            "seconds_per_step": t_step, "host_cpus": cores, "blas_threads": blas_threads,
            "cpu_model": cpu_model}


if __name__ == "__main__":
    main()
