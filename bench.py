#!/usr/bin/env python3
"""Benchmark of the OSCAR INT2 decode path on one MI355X.

One step = one decode step of one attention layer for B sequences
(oscar_decode_step): kv_append of each sequence's newest token (rotate, clip,
INT2, pack) and the query rotation q~ = q R_k in one launch, then split (paged
split-K attention over the INT2 cache) and reduce (log-sum-exp merge,
o = o~ R_v^T), all on one HIP stream with the inputs already resident in HBM.  The default
workload is the Qwen3-8B-shaped layer: 32 query / 8 KV heads, head dim 128,
batch 64, per-sequence context lengths uniform in [16384, 32768], page size 64,
shuffled non-contiguous pages.

Prints one JSON line.  `value` is the step's algorithmic HBM bytes divided by
the step time (GB/s): K eager steps bracketed by torch.cuda.synchronize(), wall
clock.  `roofline` is the split kernel (the dominant kernel), timed with HIP
events on the library's stream around K back-to-back launches; `kernels_us`
breaks one step down with events between the stages (a separate pass, since
those events add launch gaps).
`cpu_baseline` is the CPU oracle timed on a bounded sample of the same
workload.  `bf16_baseline` is the bf16 paged-decode kernel on the same
sequences.  `mixed_cache_step` is oscar_decode_step_mixed on the same sequences
with a bf16 sink of 64 and a bf16 window of 256 tokens around the INT2 history.
`variants` times the same step with the cache in other quantizer formats: the
paper's stated one (128-channel groups, bf16 scale/zero, per-token quantile
clip), the same at 64-channel groups, identity R_V, and one rotation per KV head.
`prefill_128k_tokens` times one 131072-token prompt written by
oscar_mixed_append.  `calibration` times the offline calibration of one layer
(oscar_calibrate_layer on 8878 synthetic calibration tokens) and its stages.
`c3_qwen3_32b_b128` and `c4_longctx_b16` time the same step on the Qwen3-32B
shaped layer (64/8 heads, batch 128, 32768 tokens; with its bf16 baseline) and
the long-context layer (96/8 heads, batch 16, 131072 tokens, Student-t keys,
64 splits), each with its split kernel's roofline and the pieces per sequence
the split produces; `c3_tp8_share` is one GPU's share of the Qwen3-32B-shaped
layer under 8-way KV-head sharding (one KV head, 8 query heads, batch 128, 32768
tokens).  `small_configs` times the cache-resident workloads (tiny
4/1 x 256, Qwen3-4B 8192, Qwen3-8B batch 1) warm and cold (a 1 GiB buffer
written between the calls, outside the events), with the oracle on one host
thread and on all of them.  `read_probe_ex` is the streaming-read probe over
access patterns (loads in flight, non-temporal loads, per-wave chunks).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("INT2 paged decode attn: µs/step, HBM GB/s & % of peak "
          "(Qwen3-8B shape, 32k ctx)")
HBM_PEAK_GBS = 8000.0
INT2_BYTES_PER_TOKEN_HEAD = 96          # 32 B K codes + 32 B V codes + 16 B K (s,z) + 16 B V (s,z)
BF16_BYTES_PER_TOKEN_HEAD = 512


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=2, help="workload index 0..5 (default 2)")
    ap.add_argument("--batch", type=int, default=None, help="batch override (config 2: 64)")
    ap.add_argument("--num-splits", type=int, default=0, help="0 = library default")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-bf16-baseline", action="store_true")
    ap.add_argument("--settle-ms", type=float, default=50.0,
                    help="untimed steps run for this long before the warm-up steps")
    ap.add_argument("--graph", action="store_true",
                    help="also time HIP-graph replays of the step (reported under timing; "
                         "slower than eager launches on ROCm 7.x, so never used for value)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target CPU time for the oracle baseline sample")
    ap.add_argument("--no-prefill", action="store_true",
                    help="skip the prefill-scale cache write (one 131072-token prompt)")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the quantizer-variant steps (paper format at G = 128 and 64, identity R_V, per-head R)")
    ap.add_argument("--no-calib", action="store_true",
                    help="skip the offline calibration of one layer (8878 tokens)")
    ap.add_argument("--no-mixed", action="store_true",
                    help="skip the mixed-precision cache step (bf16 sink + window)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the Qwen3-32B (config 3) and long-context (config 4) rows")
    ap.add_argument("--no-small", action="store_true",
                    help="skip the warm/cold rows of the cache-resident configs 0, 1, 2 (B=1)")
    ap.add_argument("--sink", type=int, default=64, help="mixed cache: bf16 sink tokens S0")
    ap.add_argument("--window", type=int, default=256, help="mixed cache: bf16 window tokens W")
    return ap.parse_args()


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: liboscar runs the decode path on a single "
              "MI355X (no multi-GPU path); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2605_17757_amd as ok
    import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    dev = "cuda"
    cfg = W.config(args.config, batch=args.batch if args.batch else (64 if args.config == 2 else None))
    B, Hq, Hkv, d = cfg.B, cfg.Hq, cfg.Hkv, cfg.d
    lens = cfg.lens.astype(np.int64)
    table, num_pages = W.block_table(cfg)
    lay = ok.Layout(num_kv_heads=Hkv, num_pages=num_pages)
    Rk_np, Rv_np = W.rotations(cfg)
    Rk = torch.from_numpy(Rk_np).to(dev)
    Rv = torch.from_numpy(Rv_np).to(dev)
    bt = torch.from_numpy(table).to(dev)
    sl = torch.from_numpy(cfg.lens).to(dev)
    q = W.queries(cfg, device=dev)
    S = args.num_splits or ok.default_num_splits(lay, B, Hq, int(table.shape[1]) * 64)
    if cfg.min_splits and S < cfg.min_splits:
        S = cfg.min_splits

    # ---- setup (untimed): build the INT2 and bf16 caches from the same rows ----
    t0 = time.time()
    pool = ok.alloc_pool(lay)
    bf_pool = None
    if not args.no_bf16_baseline:
        bf_pool = torch.zeros(ok.bf16_pool_bytes(lay) // 2, dtype=torch.bfloat16, device=dev)
    new_k = torch.empty(B, Hkv, d, dtype=torch.bfloat16, device=dev)
    new_v = torch.empty_like(new_k)
    new_slots = np.zeros(B, np.int64)
    # mixed cache: the same pool serves as its INT2 history (its history tokens are
    # quantized from the same rows); the sink and window rows go to a segment store
    S0m, Wm = args.sink, args.window
    seg_store = None if args.no_mixed else ok.alloc_seg(lay, B, S0m, Wm)
    pre = torch.from_numpy(cfg.lens - 1).to(dev)
    for b in range(B):
        k, v = W.cache_kv(cfg, b, device=dev)
        n = int(lens[b])
        slots = torch.from_numpy(W.slots_for(table, b, np.arange(n))).to(dev)
        # the cache holds tokens 0 .. n-2; token n-1 is the step's new token
        ok.kv_append(lay, pool, k[:n - 1], v[:n - 1], slots[:n - 1], Rk, Rv, cfg.clip_k,
                     cfg.clip_v)
        if bf_pool is not None:
            ok.bf16_kv_append(lay, bf_pool, k, v, slots)
        if seg_store is not None:  # sink and window tokens of the cache of length n - 1
            lo = min(S0m, n - 1)
            keep = torch.from_numpy(np.r_[0:lo, max(lo, n - 1 - Wm):n - 1].astype(np.int64)).to(dev)
            if keep.numel():
                ok.mixed_append(lay, pool, seg_store, S0m, Wm, k[keep], v[keep],
                                torch.full((keep.numel(),), b, dtype=torch.int32, device=dev),
                                keep, bt, pre, Rk, Rv, cfg.clip_k, cfg.clip_v)
        new_k[b] = k[n - 1]
        new_v[b] = v[n - 1]
        new_slots[b] = int(W.slots_for(table, b, [n - 1])[0])
        del k, v
    new_slots_t = torch.from_numpy(new_slots).to(dev)
    ws = ok.alloc_workspace(lay, B, Hq, S)
    out = torch.empty(B, Hq, d, dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    setup_s = time.time() - t0
    print("setup %.1fs: %s B=%d Hq=%d Hkv=%d splits=%d mean_len=%.0f" %
          (setup_s, cfg.name, B, Hq, Hkv, S, lens.mean()), file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream()

    def step_fused():
        """The timed step: oscar_decode_step (cache update + query rotation in one
        launch, then split, then reduce)."""
        ok.decode_step(lay, pool, new_k, new_v, new_slots_t, cfg.clip_k, cfg.clip_v, q, bt, sl,
                       Rk, Rv, cfg.sm_scale, S, ws, out)

    def step(ev=None):
        """The same step as four separate stage calls, for the per-stage breakdown."""
        if ev: ev[0].record(stream)
        ok.kv_append(lay, pool, new_k, new_v, new_slots_t, Rk, Rv, cfg.clip_k, cfg.clip_v)
        if ev: ev[1].record(stream)
        ok.decode_prepare(lay, q, Rk, cfg.sm_scale, S, ws)
        if ev: ev[2].record(stream)
        ok.decode_split(lay, pool, B, Hq, bt, sl, S, ws)
        if ev: ev[3].record(stream)
        ok.decode_reduce(lay, B, Hq, Rv, S, ws, out)
        if ev: ev[4].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ref_out = out.clone()
    for _ in range(args.warmup):
        step_fused()
    torch.cuda.synchronize()
    if not torch.equal(out, ref_out):
        raise SystemExit("oscar_decode_step output differs from the four stage calls")
    # Settle: after any pause of the GPU (here the output check above) the next
    # ~60 steps run 5-20% slower while it ramps back up, whatever ran before the
    # pause; untimed blocks of steps run back to back for --settle-ms right
    # before the timed region.
    t_settle = time.perf_counter()
    while (time.perf_counter() - t_settle) * 1e3 < args.settle_ms:
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record(stream)
        for _ in range(20):
            step_fused()
        s1.record(stream)
        torch.cuda.synchronize()

    def timed(run_one):
        """K steps bracketed by synchronize; HIP events around the whole region."""
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        e0.record(stream)
        for _ in range(args.steps):
            run_one()
        e1.record(stream)
        torch.cuda.synchronize()
        wall_us = (time.perf_counter() - w0) / args.steps * 1e6
        return wall_us, e0.elapsed_time(e1) * 1e3 / args.steps

    eager_wall_us, eager_ev_us = timed(step_fused)

    # Optional: the step captured once as a HIP graph and replayed; reported only
    # when every replay reproduces the eager output bit for bit.
    graph_note = "not timed (pass --graph)"
    graph_wall_us = graph_ev_us = None
    if args.graph:
        try:
            g = torch.cuda.CUDAGraph()
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                step_fused()  # warm the side stream
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            with torch.cuda.graph(g):
                step_fused()
            torch.cuda.synchronize()
            ok_replays = True
            for _ in range(3):
                out.zero_()
                g.replay()
                torch.cuda.synchronize()
                ok_replays &= bool(torch.equal(out, ref_out))
            if ok_replays:
                graph_wall_us, graph_ev_us = timed(g.replay)
                ok_replays = bool(torch.equal(out, ref_out))
            graph_note = "timed" if ok_replays else "replay output differs from eager: not timed"
            if not ok_replays:
                graph_wall_us = graph_ev_us = None
        except Exception as exc:  # capture unsupported: report and time eagerly
            graph_note = "capture failed: %s" % (type(exc).__name__,)
    us_step = eager_wall_us

    # per-stage breakdown: a separate pass with events between the stages
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    seg = np.array([[evs[i][j].elapsed_time(evs[i][j + 1]) for j in range(4)]
                    for i in range(args.steps)]) * 1e3               # us
    step_us = np.array([evs[i][0].elapsed_time(evs[i][4]) for i in range(args.steps)]) * 1e3

    # ---- algorithmic bytes ----
    pages_used = int(np.sum((lens + 63) // 64))
    kv_bytes = int(lens.sum()) * Hkv * INT2_BYTES_PER_TOKEN_HEAD
    table_bytes = pages_used * 4 + B * 4
    split_bytes = kv_bytes + table_bytes
    qo_bytes = 2 * B * Hq * d * 2
    append_bytes = 2 * B * Hkv * d * 2 + B * Hkv * INT2_BYTES_PER_TOKEN_HEAD + B * 8 + 2 * d * d * 4
    step_bytes = split_bytes + qo_bytes + append_bytes + 2 * d * d * 4
    # the dominant kernel alone: K back-to-back launches between two events on its stream
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        ok.decode_split(lay, pool, B, Hq, bt, sl, S, ws)
    e1.record(stream)
    torch.cuda.synchronize()
    split_us = e0.elapsed_time(e1) * 1e3 / args.steps
    achieved = split_bytes / (split_us * 1e-6) / 1e9
    pieces_main = pieces_per_sequence(ws, B, Hq, S)

    # ---- the 64-token-per-sequence cache update (4096 tokens x 8 KV heads) ----
    # into each sequence's spare slots len_b .. len_b + 63 (never read by the
    # decode above, whose lengths stay len_b); rotation-bound: 2 * 128 * 128 FLOP
    # per row (token, KV head, K or V), accumulated in fp64
    n_new = 64
    ak = torch.randn(B * n_new, Hkv, d, device=dev).to(torch.bfloat16)
    av = torch.randn(B * n_new, Hkv, d, device=dev).to(torch.bfloat16)
    aslots = torch.from_numpy(np.concatenate(
        [W.slots_for(table, b, np.arange(int(lens[b]), int(lens[b]) + n_new)) for b in range(B)])).to(dev)
    for _ in range(3):
        ok.kv_append(lay, pool, ak, av, aslots, Rk, Rv, cfg.clip_k, cfg.clip_v)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        ok.kv_append(lay, pool, ak, av, aslots, Rk, Rv, cfg.clip_k, cfg.clip_v)
    e1.record(stream)
    torch.cuda.synchronize()
    app_us = e0.elapsed_time(e1) * 1e3 / args.steps
    app_rows = 2 * B * n_new * Hkv
    app_flop = app_rows * 2 * d * d
    del ak, av

    # ---- prefill-scale cache write: one 131072-token prompt x 8 KV heads routed by
    # oscar_mixed_append (bf16 sink 64 + window 256, the rest INT2), into a pool of
    # its own; rotation-bound like the 64-token update ----
    pf = None
    if not args.no_prefill:
        pf_tok = 131072
        pf_pages = (pf_tok + 63) // 64
        pf_lay = ok.Layout(num_kv_heads=Hkv, num_pages=pf_pages)
        pf_pool = ok.alloc_pool(pf_lay)
        pf_seg = ok.alloc_seg(pf_lay, 1, S0m, Wm)
        pk = torch.randn(pf_tok, Hkv, d, device=dev).to(torch.bfloat16)
        pv = torch.randn(pf_tok, Hkv, d, device=dev).to(torch.bfloat16)
        pidx = torch.zeros(pf_tok, dtype=torch.int32, device=dev)
        ppos = torch.arange(pf_tok, dtype=torch.int64, device=dev)
        pbt = torch.arange(pf_pages, dtype=torch.int32, device=dev).view(1, pf_pages)
        plen = torch.tensor([pf_tok], dtype=torch.int32, device=dev)

        def prefill():
            ok.mixed_append(pf_lay, pf_pool, pf_seg, S0m, Wm, pk, pv, pidx, ppos, pbt, plen, Rk,
                            Rv, cfg.clip_k, cfg.clip_v)

        prefill()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        n_pf = 5
        e0.record(stream)
        for _ in range(n_pf):
            prefill()
        e1.record(stream)
        torch.cuda.synchronize()
        pf_us = e0.elapsed_time(e1) * 1e3 / n_pf
        pf_rows = 2 * (pf_tok - S0m - Wm) * Hkv                   # quantized rows (K and V)
        pf_flop = pf_rows * 2 * d * d                              # their rotations
        pf = {"tokens": pf_tok, "kv_heads": Hkv, "S0": S0m, "W": Wm, "us": round(pf_us, 1),
              "tokens_per_s": round(pf_tok / (pf_us * 1e-6), 1), "bound": "alu",
              "achieved_tflops_fp64": round(pf_flop / (pf_us * 1e-6) / 1e12, 2),
              "peak_tflops_fp64": 78.6,
              "frac": round(pf_flop / (pf_us * 1e-6) / 1e12 / 78.6, 4),
              "int2_rows": pf_rows}
        del pf_pool, pf_seg, pk, pv

    res = {
        "metric": METRIC,
        "value": round(step_bytes / (us_step * 1e-6) / 1e9, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(us_step / 1e3, 4),
        "us_per_step": round(us_step, 2),
        "frac_of_peak": round(step_bytes / (us_step * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
        "tokens_per_s": round(B / (us_step * 1e-6), 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": cfg.name, "batch": B, "q_heads": Hq, "kv_heads": Hkv, "head_dim": d,
            "page_size": 64, "group_size": 32, "clip": cfg.clip_k,
            "seq_len_mean": float(lens.mean()), "seq_len_min": int(lens.min()),
            "seq_len_max": int(lens.max()), "num_splits": S, "new_tokens_per_step": B,
        },
        "timing": {
            "us_per_step_eager_wall": round(eager_wall_us, 2),
            "us_per_step_eager_events": round(eager_ev_us, 2),
            "us_per_step_graph_wall": None if graph_wall_us is None else round(graph_wall_us, 2),
            "us_per_step_graph_events": None if graph_ev_us is None else round(graph_ev_us, 2),
            "graph_replay": graph_note,
        },
        "kernels_us": {
            "kv_append": round(float(np.mean(seg[:, 0])), 2),
            "decode_prepare": round(float(np.mean(seg[:, 1])), 2),
            "decode_split": round(float(np.mean(seg[:, 2])), 2),
            "decode_split_back_to_back": round(split_us, 2),
            "decode_reduce": round(float(np.mean(seg[:, 3])), 2),
            "step_events_median": round(float(np.median(step_us)), 2),
            "step_events_p10": round(float(np.percentile(step_us, 10)), 2),
            "step_events_p90": round(float(np.percentile(step_us, 90)), 2),
        },
        "roofline": {
            "kernel": "decode_split", "bound": "hbm", "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": split_traffic(cfg.name), "bytes_per_launch": split_bytes,
        },
        "append_64_tokens_per_seq": {
            "tokens": B * n_new, "rows": app_rows, "us": round(app_us, 2),
            "bound": "alu", "achieved_tflops_fp64": round(app_flop / (app_us * 1e-6) / 1e12, 2),
            "peak_tflops_fp64": 78.6,
            "frac": round(app_flop / (app_us * 1e-6) / 1e12 / 78.6, 4),
            "bytes": 2 * B * n_new * Hkv * d * 2 + B * n_new * Hkv * INT2_BYTES_PER_TOKEN_HEAD,
        },
        "prefill_128k_tokens": pf,
        "bytes": {"int2_kv": kv_bytes, "block_table": table_bytes, "q_and_out": qo_bytes,
                  "append": append_bytes, "step_total": step_bytes,
                  "bf16_kv_equivalent": int(lens.sum()) * Hkv * BF16_BYTES_PER_TOKEN_HEAD},
    }

    # ---- the mixed-precision cache (bf16 sink S0 + INT2 history + bf16 window W) ----
    # one oscar_decode_step_mixed per step: update (new token into the window,
    # the window's oldest token demoted to INT2) + query rotation, INT2 split over
    # the history, bf16 partial over sink and window, merge.  Run after the
    # measurements above: its demotions rewrite pool slots they do not read.
    if seg_store is not None:
        mws = ok.alloc_mixed_workspace(lay, B, Hq, S)
        mout = torch.empty_like(out)

        def step_mixed():
            ok.decode_step_mixed(lay, pool, seg_store, S0m, Wm, new_k, new_v, cfg.clip_k,
                                 cfg.clip_v, q, bt, sl, Rk, Rv, cfg.sm_scale, S, mws, mout)

        for _ in range(args.warmup):
            step_mixed()
        t_settle = time.perf_counter()
        while (time.perf_counter() - t_settle) * 1e3 < args.settle_ms:
            for _ in range(20):
                step_mixed()
            torch.cuda.synchronize()
        m_wall_us, m_ev_us = timed(step_mixed)
        lo_m = np.minimum(S0m, lens)
        hi_m = np.maximum(lo_m, lens - Wm)
        n_bf = lo_m + (lens - hi_m)
        hist_pages = np.where(hi_m > lo_m, (hi_m + 63) // 64 - lo_m // 64, 0)
        m_hist = int(np.sum(hi_m - lo_m)) * Hkv * INT2_BYTES_PER_TOKEN_HEAD
        m_bf16 = int(np.sum(n_bf)) * Hkv * BF16_BYTES_PER_TOKEN_HEAD
        n_dem = int(np.sum((lens - 1 - Wm >= S0m) & (Wm > 0)))
        m_update = (2 * B * Hkv * d * 2          # new rows read
                    + 2 * B * Hkv * d * 2        # new rows written to the window
                    + 2 * n_dem * Hkv * d * 2    # demoted rows read
                    + n_dem * Hkv * INT2_BYTES_PER_TOKEN_HEAD + 2 * d * d * 4)
        m_bytes = (m_hist + m_bf16 + int(np.sum(hist_pages)) * 4 + B * 4 + qo_bytes + m_update
                   + 2 * d * d * 4)
        res["mixed_cache_step"] = {
            "S0": S0m, "W": Wm, "us_per_step": round(m_wall_us, 2),
            "us_per_step_events": round(m_ev_us, 2),
            "GBps": round(m_bytes / (m_wall_us * 1e-6) / 1e9, 1),
            "frac_of_peak": round(m_bytes / (m_wall_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "bytes": {"int2_history": m_hist, "bf16_sink_window": m_bf16, "update": m_update,
                      "step_total": m_bytes},
        }
        del mws, seg_store

    # ---- quantizer variants on the same sequences: a cache of tokens 0..n-2 in the
    # variant's format, then the same timed oscar_decode_step ----
    if not args.no_variants:
        del pool  # the INT2 pool of the main step is no longer needed
        torch.cuda.empty_cache()
        res["variants"] = {}
        # per-head rotations: one seeded matrix per KV head for K and V
        Rk_ph = torch.from_numpy(np.stack([W.rotation(cfg.seed + W.S_RK + 7919 * h)
                                           for h in range(Hkv)])).to(dev)
        Rv_ph = torch.from_numpy(np.stack([W.rotation(cfg.seed + W.S_RV + 7919 * h)
                                           for h in range(Hkv)])).to(dev)
        for vname, (clip_mode, meta, use_rv, G, rph) in {
                "paper_format": (ok.CLIP_TOKEN_QUANTILE, ok.META_BF16, True, 128, 0),
                "paper_format_g64": (ok.CLIP_TOKEN_QUANTILE, ok.META_BF16, True, 64, 0),
                "identity_v": (ok.CLIP_GROUP_ABSMAX, ok.META_F16, False, 32, 0),
                "per_head_r": (ok.CLIP_GROUP_ABSMAX, ok.META_F16, True, 32, 1)}.items():
            vlay = ok.Layout(num_kv_heads=Hkv, num_pages=num_pages, group_size=G,
                             clip_mode=clip_mode, meta_dtype=meta, rot_per_head=rph)
            vRk = Rk_ph if rph else Rk
            vRv = (Rv_ph if rph else Rv) if use_rv else None
            vpool = ok.alloc_pool(vlay)
            t0 = time.time()
            for b in range(B):
                k, v = W.cache_kv(cfg, b, device=dev)
                n = int(lens[b])
                slots = torch.from_numpy(W.slots_for(table, b, np.arange(n - 1))).to(dev)
                ok.kv_append(vlay, vpool, k[:n - 1], v[:n - 1], slots, vRk, vRv, cfg.clip_k,
                             cfg.clip_v)
                del k, v
            torch.cuda.synchronize()
            build_s = time.time() - t0

            def step_v():
                ok.decode_step(vlay, vpool, new_k, new_v, new_slots_t, cfg.clip_k, cfg.clip_v, q,
                               bt, sl, vRk, vRv, cfg.sm_scale, S, ws, out)

            for _ in range(args.warmup):
                step_v()
            t_settle = time.perf_counter()
            while (time.perf_counter() - t_settle) * 1e3 < args.settle_ms:
                for _ in range(20):
                    step_v()
                torch.cuda.synchronize()
            v_wall_us, v_ev_us = timed(step_v)
            # per token-head: 64 B of codes + 2 (128 / G) (s, z) entries of 4 B; no R_v
            # reads (update, reduce) without R_v
            tok_b = 64 + 2 * (d // G) * 4
            vbytes = (step_bytes - kv_bytes + int(lens.sum()) * Hkv * tok_b
                      - B * Hkv * (INT2_BYTES_PER_TOKEN_HEAD - tok_b)
                      - (0 if use_rv else 2 * d * d * 4)
                      + (2 * (Hkv - 1) * 2 * d * d * 4 if rph else 0))  # R_k, R_v read per head
            res["variants"][vname] = {
                "clip_mode": "token_quantile" if clip_mode else "group_absmax",
                "meta_dtype": "bf16" if meta else "f16", "R_v": "given" if use_rv else "identity",
                "rotation_per_kv_head": bool(rph),
                "group_size": G, "bytes_per_token_head": tok_b, "step_bytes": vbytes,
                "us_per_step": round(v_wall_us, 2), "us_per_step_events": round(v_ev_us, 2),
                "GBps": round(vbytes / (v_wall_us * 1e-6) / 1e9, 1),
                "frac_of_peak": round(vbytes / (v_wall_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                "cache_build_s": round(build_s, 2),
            }
            del vpool
            torch.cuda.empty_cache()

    # ---- bf16 paged-decode baseline on the same sequences ----
    if bf_pool is not None:
        bf_out = torch.empty_like(out)
        bws = torch.empty(ok.decode_workspace_bytes(lay, B, Hq, S), dtype=torch.uint8,
                          device=dev)
        for _ in range(args.warmup):
            ok.bf16_decode_attn(lay, bf_pool, q, bt, sl, cfg.sm_scale, S, bws, bf_out)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.steps):
            ok.bf16_decode_attn(lay, bf_pool, q, bt, sl, cfg.sm_scale, S, bws, bf_out)
        e1.record(stream)
        torch.cuda.synchronize()
        bus = e0.elapsed_time(e1) * 1e3 / args.steps
        bbytes = int(lens.sum()) * Hkv * BF16_BYTES_PER_TOKEN_HEAD + table_bytes + qo_bytes
        int2_decode_us = float(np.mean(seg[:, 1] + seg[:, 2] + seg[:, 3]))
        res["bf16_baseline"] = {
            "us_per_decode": round(bus, 2), "GBps": round(bbytes / (bus * 1e-6) / 1e9, 1),
            "frac_of_peak": round(bbytes / (bus * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "int2_decode_us": round(int2_decode_us, 2),
            "int2_speedup": round(bus / int2_decode_us, 3),
            "kv_footprint_ratio": round(BF16_BYTES_PER_TOKEN_HEAD / INT2_BYTES_PER_TOKEN_HEAD, 3),
        }
        del bf_pool

    # ---- offline calibration of one layer (Alg. 1 Calibrate): 8878 calibration
    # tokens of this layer shape, the paper's quantizer format for the clip ratios ----
    if not args.no_calib:
        torch.cuda.empty_cache()
        Tc = W.CALIB_TOKENS
        cq, ck, cv = (t.to(dev) for t in W.calib_activations(Tc, Hq, Hkv, 4242))
        clay = ok.Layout(num_kv_heads=Hkv, num_pages=1, group_size=128,
                         clip_mode=ok.CLIP_TOKEN_QUANTILE, meta_dtype=ok.META_BF16)
        cands = torch.tensor([round(0.80 + 0.01 * n, 2) for n in range(21)],
                             dtype=torch.float32, device=dev)
        cws = torch.empty(ok.calibrate_layer_workspace_bytes(clay, Tc, Hq, cands.numel()),
                          dtype=torch.uint8, device=dev)
        cal = ok.calibrate_layer(clay, cq, ck, cv, cands, workspace=cws)
        torch.cuda.synchronize()

        def ev_time(fn, n):
            for _ in range(2):
                fn()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record(stream)
            for _ in range(n):
                fn()
            b.record(stream)
            torch.cuda.synchronize()
            return a.elapsed_time(b) * 1e3 / n

        layer_us = ev_time(lambda: ok.calibrate_layer(clay, cq, ck, cv, cands, workspace=cws), 5)
        obuf = torch.empty(Tc, Hq, d, dtype=torch.float32, device=dev)
        attn_us = ev_time(lambda: ok.calib_attn(cq, ck, cv, out=obuf), 10)
        sws = torch.empty(ok.calib_workspace_bytes(Tc, Hq, Hkv), dtype=torch.uint8, device=dev)
        cq_us = ev_time(lambda: ok.calib_query_cov(cq, Hkv, workspace=sws), 10)
        cs_us = ev_time(lambda: ok.calib_score_cov(cq, ck, cv, workspace=sws), 5)
        Cst = torch.stack([ok.calib_query_cov(cq, Hkv, workspace=sws),
                           ok.calib_score_cov(cq, ck, cv, workspace=sws)])
        rot_us = ev_time(lambda: ok.calib_rotation(Cst), 3)
        C72 = Cst.repeat(36, 1, 1).contiguous()   # a 36-layer model's K and V matrices
        rot72_us = ev_time(lambda: ok.calib_rotation(C72), 2)
        clip_us = ev_time(lambda: ok.calib_clip(clay, ck, cal["R_K"], cands), 5)
        pairs = Tc * (Tc + 1) // 2                 # causal (query, key) pairs per head
        attn_flop = pairs * Hq * 4 * d             # q k^T and p v, 2 d each
        res["calibration"] = {
            "tokens": Tc, "q_heads": Hq, "kv_heads": Hkv, "causal": True,
            "clip_format": "G=128, bf16 scale/zero, token quantile", "candidates": cands.numel(),
            "us_per_layer": round(layer_us, 1),
            "stages_us": {"query_cov": round(cq_us, 1), "score_cov": round(cs_us, 1),
                          "attn": round(attn_us, 1), "rotation_2_matrices": round(rot_us, 1),
                          "rotation_72_matrices": round(rot72_us, 1),
                          "clip_one_tensor": round(clip_us, 1)},
            "attn_roofline": {"bound": "mfma", "flop": attn_flop,
                              "achieved_tflops": round(attn_flop / (attn_us * 1e-6) / 1e12, 1),
                              "peak_tflops_bf16": 2500.0,
                              "frac": round(attn_flop / (attn_us * 1e-6) / 1e12 / 2500.0, 4)},
            "sweeps": [int(x) for x in cal["info"].tolist()],
            "clip": [round(float(x), 2) for x in cal["clip"].tolist()],
        }
        del cq, ck, cv, cws, obuf, sws, Cst, C72
        torch.cuda.empty_cache()

    # ---- device copy probe (achievable HBM bandwidth) ----
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(10):
        dst.copy_(src)
    e1.record(stream)
    torch.cuda.synchronize()
    res["copy_probe_GBps"] = round(2 * src.numel() * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)
    del dst
    # ---- streaming reads of 2 GiB (the reference for the split kernel's reads):
    # the plain probe at four grid sizes, then the access-pattern sweep ----
    src = torch.empty(2 << 30, dtype=torch.uint8, device=dev)
    src.fill_(1)
    cus = torch.cuda.get_device_properties(0).multi_processor_count

    def probe_rate(nb, loads=None, flags=0):
        sink = torch.empty(nb * 256, dtype=torch.int32, device=dev)
        for _ in range(2):
            ok.hbm_read_probe(src, nb, sink, loads=loads, flags=flags)
        ts = []
        for _ in range(10):
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            ok.hbm_read_probe(src, nb, sink, loads=loads, flags=flags)
            z.record(stream)
            z.synchronize()
            ts.append(a.elapsed_time(z))
        return round(src.numel() / (sorted(ts)[5] * 1e-3) / 1e9, 1)

    rp = {"%d_blocks" % (m * cus): probe_rate(m * cus) for m in (4, 8, 16, 32)}
    res["read_probe_GBps"] = rp
    sweep = {}
    for loads in (4, 8, 16):
        for flags, fname in ((0, "plain"), (ok.PROBE_NONTEMPORAL, "nt"),
                             (ok.PROBE_WAVE_CHUNKS, "chunks"),
                             (ok.PROBE_NONTEMPORAL | ok.PROBE_WAVE_CHUNKS, "nt_chunks")):
            for m in (8, 16, 32):
                sweep["%s_x%d_%dpercu" % (fname, loads, m)] = probe_rate(m * cus, loads, flags)
    best = max(sweep, key=sweep.get)
    res["read_probe_ex"] = {"best": best, "best_GBps": sweep[best], "GBps": sweep}
    res["read_probe_best_GBps"] = max(max(rp.values()), sweep[best])
    res["roofline"]["frac_of_read_probe"] = round(achieved / res["read_probe_best_GBps"], 4)
    del src

    # ---- the Qwen3-32B-shaped and long-context layers, and the cache-resident
    # workloads warm and cold ----
    res["pieces_per_sequence"] = pieces_main
    if not args.no_configs:
        torch.cuda.empty_cache()
        res["c3_qwen3_32b_b128"] = config_row(args, 3, not args.no_bf16_baseline)
        torch.cuda.empty_cache()
        res["c4_longctx_b16"] = config_row(args, 4, not args.no_bf16_baseline)
        torch.cuda.empty_cache()
        res["c3_tp8_share"] = config_row(args, 5, False)
        torch.cuda.empty_cache()
    if not args.no_small:
        res["small_configs"] = small_config_rows(args, not args.no_cpu_baseline)
        torch.cuda.empty_cache()

    # ---- CPU oracle baseline on a bounded sample ----
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(cfg, table, Rk_np, Rv_np, q, args.cpu_seconds)

    print(json.dumps(res), flush=True)


def _a256(x: int) -> int:
    return (x + 255) & ~255


def pieces_per_sequence(ws, B: int, Hq: int, S: int) -> dict:
    """Partial states the split wrote per sequence after a decode, read from the
    workspace's (m, l) slots (q~ fp32 [B*Hq, 128], o~ fp32 [B*Hq*S, 128], (m, l)
    fp32 [B*Hq*S, 2], 256-byte aligned regions; an unused slot holds m = -inf)."""
    import torch
    off = _a256(B * Hq * 128 * 4)
    off += _a256(B * Hq * S * 128 * 4)
    ml = ws[off:off + B * Hq * S * 8].view(torch.float32).view(B, Hq, S, 2)
    live = (ml[..., 0] > float("-inf")).sum(-1)[:, 0].cpu().numpy()  # head 0 of each sequence
    return {"min": int(live.min()), "mean": round(float(live.mean()), 2), "max": int(live.max()),
            "slots": S}


def _events(n):
    import torch
    return [torch.cuda.Event(enable_timing=True) for _ in range(n)]


def _back_to_back_us(fn, n, stream):
    """n calls of fn between two HIP events on `stream`; mean microseconds per call."""
    import torch
    e0, e1 = _events(2)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(n):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / n


def _build_cache(ok, W, cfg, dev, with_bf16: bool):
    """INT2 pool with tokens 0..n-2 of every sequence (token n-1 is the step's new
    token), the optional bf16 pool with all n tokens, and the new rows/slots."""
    import torch
    B, Hkv, d = cfg.B, cfg.Hkv, cfg.d
    table, num_pages = W.block_table(cfg)
    lay = ok.Layout(num_kv_heads=Hkv, num_pages=num_pages)
    Rk_np, Rv_np = W.rotations(cfg)
    Rk, Rv = torch.from_numpy(Rk_np).to(dev), torch.from_numpy(Rv_np).to(dev)
    pool = ok.alloc_pool(lay)
    bf_pool = (torch.zeros(ok.bf16_pool_bytes(lay) // 2, dtype=torch.bfloat16, device=dev)
               if with_bf16 else None)
    new_k = torch.empty(B, Hkv, d, dtype=torch.bfloat16, device=dev)
    new_v = torch.empty_like(new_k)
    new_slots = np.zeros(B, np.int64)
    for b in range(B):
        k, v = W.cache_kv(cfg, b, device=dev)
        n = int(cfg.lens[b])
        slots = torch.from_numpy(W.slots_for(table, b, np.arange(n))).to(dev)
        if n > 1:
            ok.kv_append(lay, pool, k[:n - 1], v[:n - 1], slots[:n - 1], Rk, Rv, cfg.clip_k,
                         cfg.clip_v)
        if bf_pool is not None:
            ok.bf16_kv_append(lay, bf_pool, k, v, slots)
        new_k[b] = k[n - 1]
        new_v[b] = v[n - 1]
        new_slots[b] = int(W.slots_for(table, b, [n - 1])[0])
        del k, v
    torch.cuda.synchronize()
    return dict(table=table, lay=lay, Rk=Rk, Rv=Rv, Rk_np=Rk_np, Rv_np=Rv_np, pool=pool,
                bf_pool=bf_pool, new_k=new_k, new_v=new_v,
                new_slots=torch.from_numpy(new_slots).to(dev),
                bt=torch.from_numpy(table).to(dev), sl=torch.from_numpy(cfg.lens).to(dev),
                q=W.queries(cfg, device=dev))


def _step_bytes(cfg):
    """Algorithmic bytes of one decode step (split, q/out, the new tokens' update,
    R_k and R_v) and of the split alone."""
    lens = cfg.lens.astype(np.int64)
    B, Hq, Hkv, d = cfg.B, cfg.Hq, cfg.Hkv, cfg.d
    split = int(lens.sum()) * Hkv * INT2_BYTES_PER_TOKEN_HEAD + int(np.sum((lens + 63) // 64)) * 4 + B * 4
    qo = 2 * B * Hq * d * 2
    app = 2 * B * Hkv * d * 2 + B * Hkv * INT2_BYTES_PER_TOKEN_HEAD + B * 8 + 2 * d * d * 4
    return split + qo + app + 2 * d * d * 4, split, qo


def config_row(args, index: int, with_bf16: bool) -> dict:
    """The decode step on workload `index` (3: Qwen3-32B shape, 4: long context):
    step time, split roofline, stage breakdown, pieces per sequence, bf16 baseline."""
    import torch

    import paper_2605_17757_amd as ok
    import workloads as W
    dev = "cuda"
    stream = torch.cuda.current_stream()
    cfg = W.config(index)
    B, Hq, Hkv, d = cfg.B, cfg.Hq, cfg.Hkv, cfg.d
    t0 = time.time()
    c = _build_cache(ok, W, cfg, dev, with_bf16)
    lay = c["lay"]
    S = args.num_splits or ok.default_num_splits(lay, B, Hq, int(c["table"].shape[1]) * 64)
    if cfg.min_splits and S < cfg.min_splits:
        S = cfg.min_splits
    ws = ok.alloc_workspace(lay, B, Hq, S)
    out = torch.empty(B, Hq, d, dtype=torch.bfloat16, device=dev)
    print("setup %.1fs: %s B=%d Hq=%d Hkv=%d splits=%d" % (time.time() - t0, cfg.name, B, Hq, Hkv,
                                                          S), file=sys.stderr, flush=True)

    def step():
        ok.decode_step(lay, c["pool"], c["new_k"], c["new_v"], c["new_slots"], cfg.clip_k,
                       cfg.clip_v, c["q"], c["bt"], c["sl"], c["Rk"], c["Rv"], cfg.sm_scale, S,
                       ws, out)

    for _ in range(args.warmup):
        step()
    t_settle = time.perf_counter()
    while (time.perf_counter() - t_settle) * 1e3 < args.settle_ms:
        for _ in range(10):
            step()
        torch.cuda.synchronize()
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    us = (time.perf_counter() - w0) / args.steps * 1e6
    step_b, split_b, qo_b = _step_bytes(cfg)
    # stage breakdown (events between the decode stages)
    ev = [_events(4) for _ in range(args.steps)]
    for i in range(args.steps):
        ev[i][0].record(stream)
        ok.decode_prepare(lay, c["q"], c["Rk"], cfg.sm_scale, S, ws)
        ev[i][1].record(stream)
        ok.decode_split(lay, c["pool"], B, Hq, c["bt"], c["sl"], S, ws)
        ev[i][2].record(stream)
        ok.decode_reduce(lay, B, Hq, c["Rv"], S, ws, out)
        ev[i][3].record(stream)
    torch.cuda.synchronize()
    seg = np.array([[ev[i][j].elapsed_time(ev[i][j + 1]) for j in range(3)]
                    for i in range(args.steps)]) * 1e3
    split_us = _back_to_back_us(lambda: ok.decode_split(lay, c["pool"], B, Hq, c["bt"], c["sl"],
                                                        S, ws), args.steps, stream)
    ach = split_b / (split_us * 1e-6) / 1e9
    row = {
        "workload": cfg.name, "batch": B, "q_heads": Hq, "kv_heads": Hkv,
        "seq_len": int(cfg.lens.max()), "k_dist": cfg.k_dist, "num_splits": S,
        "us_per_step": round(us, 2), "GBps": round(step_b / (us * 1e-6) / 1e9, 1),
        "frac_of_peak": round(step_b / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
        "tokens_per_s": round(B / (us * 1e-6), 1),
        "stages_us": {"decode_prepare": round(float(np.mean(seg[:, 0])), 2),
                      "decode_split": round(float(np.mean(seg[:, 1])), 2),
                      "decode_reduce": round(float(np.mean(seg[:, 2])), 2)},
        "roofline": {"kernel": "decode_split", "bound": "hbm", "achieved": round(ach, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(ach / HBM_PEAK_GBS, 4), "us": round(split_us, 2),
                     "bytes_per_launch": split_b, "traffic": split_traffic(cfg.name)},
        "pieces_per_sequence": pieces_per_sequence(ws, B, Hq, S),
        "bytes": {"step_total": step_b, "int2_kv": int(cfg.lens.astype(np.int64).sum()) * Hkv *
                  INT2_BYTES_PER_TOKEN_HEAD,
                  "bf16_kv_equivalent": int(cfg.lens.astype(np.int64).sum()) * Hkv *
                  BF16_BYTES_PER_TOKEN_HEAD},
    }
    if c["bf_pool"] is not None:
        bws = torch.empty(ok.decode_workspace_bytes(lay, B, Hq, S), dtype=torch.uint8,
                          device=dev)
        bout = torch.empty_like(out)

        def bf16():
            ok.bf16_decode_attn(lay, c["bf_pool"], c["q"], c["bt"], c["sl"], cfg.sm_scale, S,
                                bws, bout)

        for _ in range(3):
            bf16()
        bus = _back_to_back_us(bf16, max(5, args.steps // 4), stream)
        bbytes = row["bytes"]["bf16_kv_equivalent"] + split_b - row["bytes"]["int2_kv"] + qo_b
        int2_us = float(np.mean(seg.sum(axis=1)))
        row["bf16_baseline"] = {
            "us_per_decode": round(bus, 2), "GBps": round(bbytes / (bus * 1e-6) / 1e9, 1),
            "frac_of_peak": round(bbytes / (bus * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "int2_decode_us": round(int2_us, 2), "int2_speedup": round(bus / int2_us, 3),
            "kv_footprint_ratio": round(BF16_BYTES_PER_TOKEN_HEAD / INT2_BYTES_PER_TOKEN_HEAD, 3)}
        del bws
    del c, ws
    return row


def small_config_rows(args, with_oracle: bool) -> dict:
    """Cache-resident workloads (tiny 4/1 x 256, Qwen3-4B 8192, Qwen3-8B batch 1):
    the decode step warm (back to back, and per call between events) and cold
    (a 1 GiB buffer written between the calls, outside the events), and the
    oracle's decode of the same cache on one host thread and on all of them."""
    import torch

    import oracle
    import paper_2605_17757_amd as ok
    import workloads as W
    dev = "cuda"
    stream = torch.cuda.current_stream()
    flush = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    rows = {}
    for index, batch in ((0, None), (1, None), (2, 1)):
        cfg = W.config(index, batch=batch)
        B, Hq, Hkv, d = cfg.B, cfg.Hq, cfg.Hkv, cfg.d
        c = _build_cache(ok, W, cfg, dev, False)
        lay = c["lay"]
        S = ok.default_num_splits(lay, B, Hq, int(c["table"].shape[1]) * 64)
        ws = ok.alloc_workspace(lay, B, Hq, S)
        out = torch.empty(B, Hq, d, dtype=torch.bfloat16, device=dev)

        def step():
            ok.decode_step(lay, c["pool"], c["new_k"], c["new_v"], c["new_slots"], cfg.clip_k,
                           cfg.clip_v, c["q"], c["bt"], c["sl"], c["Rk"], c["Rv"], cfg.sm_scale,
                           S, ws, out)

        for _ in range(20):
            step()
        b2b = _back_to_back_us(step, 200, stream)
        ev = [_events(2) for _ in range(100)]
        torch.cuda.synchronize()
        for e in ev:
            e[0].record(stream)
            step()
            e[1].record(stream)
        torch.cuda.synchronize()
        warm = np.array([e[0].elapsed_time(e[1]) for e in ev]) * 1e3
        cold = []
        for i in range(30):
            flush.fill_(i & 0xff)
            e = _events(2)
            e[0].record(stream)
            step()
            e[1].record(stream)
            torch.cuda.synchronize()
            cold.append(e[0].elapsed_time(e[1]) * 1e3)
        cold = np.array(cold)
        step_b, split_b, _ = _step_bytes(cfg)

        def pct(x):
            return {"median": round(float(np.median(x)), 2), "p10": round(float(np.percentile(x, 10)), 2),
                    "p90": round(float(np.percentile(x, 90)), 2)}

        row = {"workload": cfg.name, "batch": B, "q_heads": Hq, "kv_heads": Hkv,
               "seq_len": int(cfg.lens.max()), "num_splits": S, "step_bytes": step_b,
               "int2_kv_bytes": int(cfg.lens.astype(np.int64).sum()) * Hkv * INT2_BYTES_PER_TOKEN_HEAD,
               "warm_us_back_to_back": round(b2b, 2), "warm_us_per_call": pct(warm),
               "cold_us_per_call": pct(cold),
               "cold_GBps": round(step_b / (np.median(cold) * 1e-6) / 1e9, 1),
               "cold_frac_of_peak": round(step_b / (np.median(cold) * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
               "tokens_per_s_warm": round(B / (b2b * 1e-6), 1)}
        if with_oracle:
            row["oracle"] = _oracle_small(oracle, W, cfg, c)
        rows[cfg.name] = row
        del c, ws
    del flush
    return rows


def _oracle_small(oracle, W, cfg, c) -> dict:
    """The oracle's decode of the whole workload (its own cache, built untimed),
    median of 3 runs on one thread and on all of them."""
    import torch

    def u16(t):
        return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)

    Hkv, d = cfg.Hkv, cfg.d
    table, lens = c["table"], cfg.lens
    bph = oracle.page_head_bytes(d, 64, 32)
    pool = np.zeros(table.size * Hkv * bph, np.uint8)
    for b in range(cfg.B):
        n = int(lens[b])
        k, v = W.cache_kv(cfg, b, device="cuda")
        oracle.kv_append(pool, d=d, Hkv=Hkv, P=64, G=32, k=u16(k), v=u16(v),
                         slot_mapping=W.slots_for(table, b, np.arange(n)), Rk=c["Rk_np"],
                         Rv=c["Rv_np"], clip_k=cfg.clip_k, clip_v=cfg.clip_v)
    qh = u16(c["q"])
    all_threads = oracle.num_threads()
    res = {}
    for name, nt in (("one_thread", 1), ("all_threads", all_threads)):
        oracle.set_num_threads(nt)
        ts = []
        for _ in range(3):
            t0 = time.perf_counter()
            oracle.decode(pool, d=d, Hkv=Hkv, P=64, G=32, q=qh, block_table=table,
                          seq_lens=lens, Rk=c["Rk_np"], Rv=c["Rv_np"], sm_scale=cfg.sm_scale)
            ts.append(time.perf_counter() - t0)
        t = float(np.median(ts))
        res[name] = {"threads": nt, "us_per_step": round(t * 1e6, 1),
                     "tokens_per_s": round(cfg.B / t, 3)}
    oracle.set_num_threads(all_threads)
    return res


def split_traffic(workload: str = "qwen3_8b_b64_ctx32k"):
    """HBM bytes per split launch on `workload` from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE passes (FETCH_SIZE scaled by what it reads for a 1 GiB
    copy and a 2 GiB streaming read of known size), or None when the split
    kernel's source has changed since those counters were taken or the workload
    has no record."""
    import hashlib
    rec_path = os.path.join(ROOT, "profiles", "split_mfma_kernel_traffic.json")
    try:
        rec = json.load(open(rec_path))
        src = open(os.path.join(ROOT, rec["source"]), "rb").read()
        entry = rec["workloads"][workload]
    except (OSError, ValueError, KeyError):
        return None
    if hashlib.sha256(src).hexdigest() != rec.get("source_sha256"):
        return None
    return int(entry["traffic_bytes_per_launch"])


def cpu_baseline(cfg, table, Rk_np, Rv_np, q, seconds, max_seqs=4):
    """The CPU oracle (plain C, fp64, OpenMP over (sequence, head)) decoding whole
    sequences of the same workload.  The sample is the first `max_seqs`
    sequences; the oracle builds its own cache for them with its own append
    (untimed), then decodes them repeatedly until about `seconds` of decode time.
    Reported in the metric's unit (GB/s of algorithmic INT2 bytes)."""
    import torch

    import oracle
    import workloads as W

    def u16(t):
        return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)

    qh = u16(q)
    Hkv, d = cfg.Hkv, cfg.d
    bph = oracle.page_head_bytes(d, 64, 32)
    sample = []
    for b in range(min(cfg.B, max_seqs)):
        n = int(cfg.lens[b])
        k, v = W.cache_kv(cfg, b, device="cuda")
        kb, vb = u16(k), u16(v)
        del k, v
        npg = (n + 63) // 64
        pool = np.zeros(npg * Hkv * bph, np.uint8)
        oracle.kv_append(pool, d=d, Hkv=Hkv, P=64, G=32, k=kb, v=vb,
                         slot_mapping=np.arange(n, dtype=np.int64), Rk=Rk_np, Rv=Rv_np,
                         clip_k=cfg.clip_k, clip_v=cfg.clip_v)
        sample.append((b, n, pool, np.arange(npg, dtype=np.int32)[None, :]))
    spent, nbytes, passes = 0.0, 0, 0
    while spent < seconds:
        for b, n, pool, loc in sample:
            t0 = time.perf_counter()
            oracle.decode(pool, d=d, Hkv=Hkv, P=64, G=32, q=qh[b:b + 1], block_table=loc,
                          seq_lens=np.array([n], np.int32), Rk=Rk_np, Rv=Rv_np,
                          sm_scale=cfg.sm_scale)
            spent += time.perf_counter() - t0
            nbytes += n * Hkv * INT2_BYTES_PER_TOKEN_HEAD
        passes += 1
    ntok = sum(n for _, n, _, _ in sample)
    return {
        "value": round(nbytes / spent / 1e9, 4), "unit": "GB/s",
        "cores": oracle.num_threads(), "kind": "oracle",
        "us_per_step_equiv": round(spent / (passes * len(sample)) * cfg.B * 1e6, 1),
        "sample": "decode of sequences 0-%d (%d tokens, %d q-heads each) of the same "
                  "workload, %d passes, %.1f s of oracle time" % (len(sample) - 1, ntok, cfg.Hq,
                                                                  passes, spent),
        "cpu_model": _cpu_model(),
    }


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


if __name__ == "__main__":
    main()
