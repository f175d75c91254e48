"""Benchmark of the WnW per-token decode step on one MI355X.

A step is one call of wnw_decode_step: anchor attention with chunk mass, chunk scores, top-k
and residency, recall of newly resident complements, tidal and fixed attention, merge.  The
headline run uses the paper's selection timing (the selection made after step s serves step
s+1, so the recall of step s overlaps the rest of the step); the same-step timing is measured in
the same run and reported beside it.
Inputs are seeded synthetic caches of the Voxtral-mini-3B shape at 10 minutes of audio
(30 layers, 32 query / 8 KV heads, d 128, 15 000 audio + 512 text positions, chunk 64, 20 %
on-GPU budget; 24 anchor / 120 tidal / 96 fixed KV-heads), resident in HBM before timing.

The timed steps are clip steps 16.. whatever --warmup is (the warm-up runs the steps before them).
Prints one JSON line: steps/s (value, from a timed region without timing events), per-kernel HBM
rates from HIP events bound to the launches inside the library (a second context running the
same steps), the recall rate, and the CPU oracle timed on a bounded sample of the same workload.
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

METRIC = "WnW decode steps/sec + achieved HBM GB/s (attn) at 15k audio tokens, 1 GPU"
PEAK_HBM_GBPS = 8000.0
TIMED_FROM = 16                # first clip step of the timed region (the warm-up runs the steps before it)
PEAK_BF16_TFLOPS = 2500.0      # dense bf16 MFMA
PEAK_LINK_GBPS = 64.0          # PCIe 5.0 x16, one direction
PEAK_FP64_TFLOPS = 78.6        # fp64, matrix cores (the vector rate is the same)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def overlap_sweep(W, torch, w, ctx, geo, qd, out, sc, sel, stream, args):
    """Force about N newly resident chunks per step through the selection override: k - N chunks
    stay selected, N more rotate through the remaining chunks.  For each N: step time, chunks
    copied and revived per step, and (in a context with timing events) the recall time.  The
    same schedule from the same state gives the same recall in both contexts; merge_sweep joins
    them."""
    B, S, k, nc = w.batch, w.steps, geo["k"], geo["n_chunks"]
    res = []
    for n_new in (1, 2, 4, 8, 24):
        if n_new > k or nc - (k - n_new) < n_new:
            continue
        steps, warm = 40, 8
        core = np.arange(k - n_new, dtype=np.int32)
        pool = np.arange(k - n_new, nc, dtype=np.int32)
        sched = np.empty((warm + steps, B, k), dtype=np.int32)
        for s in range(warm + steps):
            rot = pool[(s * n_new + np.arange(n_new)) % len(pool)]
            sched[s, :] = np.sort(np.concatenate([core, rot]))
        sd = torch.from_numpy(sched).cuda()
        for s in range(warm):
            W.wnw_set_selection_override(ctx, sd[s])
            W.wnw_decode_step(ctx, qd[s % S], out, sc, sel, stream)
        torch.cuda.synchronize()
        a = W.wnw_get_stats(ctx)
        t0 = time.perf_counter()
        for s in range(warm, warm + steps):
            W.wnw_set_selection_override(ctx, sd[s])
            W.wnw_decode_step(ctx, qd[s % S], out, sc, sel, stream)
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        b = W.wnw_get_stats(ctx)
        ms = el * 1e3 / steps
        nt = b["timed_steps"] - a["timed_steps"]
        rec_ms = (b["t_recall_ms"] - a["t_recall_ms"]) / nt if nt else None
        res.append({"new_per_step": n_new, "ms_per_step": ms,
                    "copied_per_step": (b["recalled_chunks"] - a["recalled_chunks"]) / steps / B,
                    "revived_per_step": (b["revived_chunks"] - a["revived_chunks"]) / steps / B,
                    "recall_ms": rec_ms})
        log(f"[bench] sweep {n_new} new/step: {1e3 / ms:.0f} steps/s" + (" (timing events)" if nt else ""))
    return res


def merge_sweep(plain, timed, ms_no_recall):
    """Steps/s from the context without timing events (plain), the recall time from the one with
    them (timed), and overlap = 1 - (T_step - T_no_recall) / T_recall: the share of the recall
    hidden behind the rest of the step."""
    rec = {r["new_per_step"]: r["recall_ms"] for r in timed}
    res = []
    for r in plain:
        ms, rec_ms = r["ms_per_step"], rec.get(r["new_per_step"])
        ov = max(0.0, min(1.0, 1.0 - (ms - ms_no_recall) / rec_ms)) if rec_ms else None
        res.append({"new_per_step": r["new_per_step"], "steps_per_s": 1e3 / ms, "ms_per_step": ms,
                    "copied_per_step": r["copied_per_step"], "revived_per_step": r["revived_per_step"],
                    "recall_ms": rec_ms, "overlap": ov})
    return res


def _steps(W, torch, ctx, qd, out, sc, sel, stream, first, n, S):
    """Run n decode steps on clip steps first.. (cyclic) and return the wall time in seconds,
    bracketed by device synchronisation."""
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(n):
        W.wnw_decode_step(ctx, qd[(first + i) % S], out, sc, sel, stream)
    torch.cuda.synchronize()
    return time.perf_counter() - t0


def run_timing(W, torch, w, timing, recall, kd, vd, qd, roles, prefill, args, chunks="disjoint", retention="uniform"):
    """One configuration (selection timing, recall path, chunk structure, retention) in two
    contexts.  The first has no timing events: its warm-up and timed steps give steps/s, and a
    second region with the selection pinned to resident chunks (no recall) gives the step time
    without recall.  The second context records HIP events around the launches (WNW_F_TIMING)
    and runs the same steps for the per-kernel breakdown.  Each runs the overlap sweep: its
    steps/s from the first, its recall time from the second.  Returns the context-independent
    numbers; both contexts are destroyed."""
    B, L, H, D, S = w.batch, w.layers, w.kv_heads, w.head_dim, w.steps
    base = ((W.WNW_F_RECALL_MEMCPY if recall == "memcpy" else 0)
            | (W.WNW_F_SELECT_NEXT_STEP if timing == "next" else 0)
            | (W.WNW_F_OVERLAP_CHUNKS if chunks == "overlap" else 0))
    stream = torch.cuda.current_stream()
    res = {}
    for timed_events in (False, True):
        if timed_events and args.no_timing:
            break
        cfg = W.make_config(B, L, w.q_heads, H, w.audio_len, w.text_len, w.chunk_len, w.budget_bp,
                            flags=base | (W.WNW_F_TIMING if timed_events else 0))
        ctx = W.wnw_init_cache(cfg, kd, vd, stream)
        try:
            if retention == "per-head":
                from synth import gen
                W.wnw_set_retention(ctx, gen.importance(w), args.lam)
            W.wnw_set_roles(ctx, roles, prefill)
            geo = W.wnw_query_geometry(ctx)
            out = torch.empty((B, L, w.q_heads, D), dtype=torch.float32, device="cuda")
            sc = torch.empty((B, geo["n_chunks"]), dtype=torch.float32, device="cuda")
            sel = torch.empty((B, max(geo["k"], 1)), dtype=torch.int32, device="cuda")
            tag = "breakdown (timing events)" if timed_events else "timed region (no events)"
            log(f"[bench] {timing}-step timing, {recall} recall, {chunks} chunks, {retention} retention, {tag}: "
                f"set-up done {geo}")
            if args.calibrate_copy and not timed_events:
                src = torch.ones(128 << 20, dtype=torch.int16, device="cuda")
                dst = torch.empty_like(src)
                for _ in range(3):
                    dst.copy_(src)
                torch.cuda.synchronize()
                del src, dst
            # the timed steps are clip steps TIMED_FROM.. whatever --warmup is (the recall's
            # churn depends on the clip position); the warm-up runs the W steps just before them
            _steps(W, torch, ctx, qd, out, sc, sel, stream, (TIMED_FROM - args.warmup) % S, args.warmup, S)
            st0 = W.wnw_get_stats(ctx)
            t_el = _steps(W, torch, ctx, qd, out, sc, sel, stream, TIMED_FROM % S, args.steps, S)
            st1 = W.wnw_get_stats(ctx)
            log(f"[bench] {timing}-step, {chunks} chunks, {tag}: {args.steps} steps in {t_el * 1e3:.1f} ms")
            # the selection pinned to the last step's chunks (all resident after one step): no
            # complement is recalled and every launch streams HBM only
            nr = max(8, args.steps // 4)
            pinned = sel.clone()         # read by every following step: kept alive here
            W.wnw_set_selection_override(ctx, pinned)
            _steps(W, torch, ctx, qd, out, sc, sel, stream, 0, 4, S)
            st2 = W.wnw_get_stats(ctx)
            t2 = _steps(W, torch, ctx, qd, out, sc, sel, stream, 0, nr, S)
            st3 = W.wnw_get_stats(ctx)
            sweep = []
            if args.sweep and timing == "next" and geo["k"] > 0:
                sweep = overlap_sweep(W, torch, w, ctx, geo, qd, out, sc, sel, stream, args)
            W.wnw_set_selection_override(ctx, None)
            del pinned
        finally:
            W.wnw_destroy(ctx)
        K = args.steps
        d = {k: st1[k] - st0[k] for k in st1 if isinstance(st1[k], (int, float))}
        d2 = {k: st3[k] - st2[k] for k in st3 if isinstance(st3[k], (int, float))}
        if not timed_events:
            res.update({"value": K / t_el, "ms_per_step": t_el * 1e3 / K, "geo": geo, "st1": st1,
                        "r_gpu": st1["r_gpu"], "r_gpu_cpu": st1["r_gpu_cpu"],
                        "clip_steps": [TIMED_FROM % S, (TIMED_FROM + K) % S or S],
                        "recall": {"copied_chunks_per_step": d["recalled_chunks"] / K / B,
                                   "revived_chunks_per_step": d["revived_chunks"] / K / B,
                                   "MB_per_step": d["recalled_bytes"] / K / 1e6,
                                   "chunk_MB": geo.get("chunk_bytes", 0) / 1e6,
                                   "step_ms_no_recall": t2 * 1e3 / nr,
                                   "host_wait_ms_per_step": d["t_host_wait_ms"] / K}})
            res["sweep_plain"] = sweep
            continue
        res["sweep"] = merge_sweep(res.pop("sweep_plain", []), sweep, res["recall"]["step_ms_no_recall"])
        n, n2 = d["timed_steps"], d2["timed_steps"]
        row_bytes = 2 * D * 2                      # K + V of one position, bf16
        # slot_rows: complement rows attended, summed over steps, sequences and tidal heads.  With
        # next-step timing the first launch carries the static tidal/fixed tiles, the tidal launch
        # every resident complement
        first = "attention" if timing == "next" else "anchor_attn"
        if timing == "next":
            first_bytes = first2_bytes = st1["anchor_bytes"] + st1["static_bytes"]
            tf_bytes = d["slot_rows"] / K * row_bytes
            tf2_bytes = d2["slot_rows"] / nr * row_bytes
        else:
            first_bytes = first2_bytes = st1["anchor_bytes"]
            tf_bytes = st1["static_bytes"] + d["slot_rows"] / K * row_bytes
            tf2_bytes = st1["static_bytes"] + d2["slot_rows"] / nr * row_bytes
        a_ms, a2_ms = d["t_anchor_ms"] / n, d2["t_anchor_ms"] / n2
        tf_ms, tf2_ms = d["t_tidal_fixed_ms"] / n, d2["t_tidal_fixed_ms"] / n2
        res["first"] = first
        res["kernels"] = {
            first: {"avg_ms": a_ms, "bytes": first_bytes, "GBps": first_bytes / a_ms / 1e6},
            first + "_pinned_selection": {"avg_ms": a2_ms, "bytes": first2_bytes, "GBps": first2_bytes / a2_ms / 1e6},
            "mass_select": {"avg_ms": d["t_select_ms"] / n},
            "recall_wait": {"avg_ms": d["t_recall_wait_ms"] / n},
            "tidal_fixed": {"avg_ms": tf_ms, "bytes": tf_bytes, "GBps": tf_bytes / tf_ms / 1e6 if tf_ms > 0 else None},
            "tidal_fixed_pinned_selection": {"avg_ms": tf2_ms, "bytes": tf2_bytes,
                                             "GBps": tf2_bytes / tf2_ms / 1e6 if tf2_ms > 0 else None},
            "combine": {"avg_ms": d["t_combine_ms"] / n},
            "step_gpu": {"avg_ms": d["t_step_ms"] / n},
        }
        if d["t_new_ms"] > 0:
            res["kernels"]["new_slots"] = {"avg_ms": d["t_new_ms"] / n}
        # the recall: the launch that carries it (same-step timing), the copy kernel on the side
        # stream (next-step timing) or the host-issued copies
        rms = d["t_recall_ms"] / n
        res["recall"]["ms"] = rms
        res["recall"]["GBps"] = (d["recalled_bytes"] / n) / rms / 1e6 if rms > 0 else None
    if "sweep_plain" in res:   # no context with timing events ran
        res["sweep"] = merge_sweep(res.pop("sweep_plain"), [], res["recall"]["step_ms_no_recall"])
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--workload", default=None, help="workload name from synth.configs (default: the 15k-audio one)")
    ap.add_argument("--recall", choices=("auto", "kernel", "memcpy"), default="auto",
                    help="recall path: copy-engine transfers issued by the host after each selection (memcpy), or "
                         "work-groups reading mapped pinned memory (kernel); auto = memcpy with next-step timing "
                         "when a segment block is at least 1 MB (the transfers leave the compute units to the "
                         "attention launch beside them), kernel otherwise and with same-step timing (the recall is "
                         "attended in the same pass, no host wait)")
    ap.add_argument("--timing", choices=("next", "same"), default="next",
                    help="selection timing of the headline run: the selection made after step s serves step s+1 "
                         "(the paper's timing; the recall overlaps the step) or step s itself")
    ap.add_argument("--no-other-timing", action="store_true", help="skip the run with the other selection timing")
    ap.add_argument("--chunks", choices=("disjoint", "overlap"), default="disjoint",
                    help="chunk structure of the headline run: disjoint chunks of chunk_len positions, or chunks of "
                         "two chunk_len/2 segments starting at every segment")
    ap.add_argument("--no-other-chunks", action="store_true", help="skip the run with the other chunk structure")
    ap.add_argument("--retention", choices=("uniform", "per-head"), default="uniform",
                    help="audio retention of the headline run: the workload's uniform budget, or min(importance * "
                         "lambda, 1) per head with seeded U(0,1) importance")
    ap.add_argument("--lam", type=float, default=0.4, help="lambda of the per-head retention (0.4: mean 20 %%)")
    ap.add_argument("--no-other-retention", action="store_true", help="skip the run with the other retention")
    ap.add_argument("--no-prefill", action="store_true",
                    help="skip the set-up measurements (prefill compression, head triage arithmetic)")
    ap.add_argument("--no-sweep", dest="sweep", action="store_false",
                    help="skip the overlap sweep (forced 1..24 newly resident chunks per step)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the CPU oracle sample (0 = skip)")
    ap.add_argument("--no-timing", action="store_true", help="no per-kernel events (for profiler runs)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run a plain 256 MiB device copy (the reference for hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: --gpus {args.gpus} is not supported "
              "(the decode step is measured on one MI355X)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2608_22704_amd import wnw as W
    from synth import configs, gen

    w = configs.BY_NAME[args.workload] if args.workload else configs.HEADLINE
    torch.cuda.set_device(0)
    B, L, H, T, D, S = w.batch, w.layers, w.kv_heads, w.total_len, w.head_dim, w.steps
    log(f"[bench] generating {w.name} (B={B}, L={L}, Hkv={H}, T={T})")
    t0 = time.time()
    roles = gen.roles(w)
    kd = torch.empty((B, L, H, T, D), dtype=torch.int16, device="cuda")
    vd = torch.empty_like(kd)
    qd = torch.empty((S, B, L, w.q_heads, D), dtype=torch.int16, device="cuda")
    prefill = np.empty((B, L, H, w.audio_len), dtype=np.float32)
    for b in range(B):
        for l, kl, vl, ql, pl in gen.iter_layers(w, b):
            kd[b, l].copy_(torch.from_numpy(kl.view(np.int16)))
            vd[b, l].copy_(torch.from_numpy(vl.view(np.int16)))
            qd[:, b, l].copy_(torch.from_numpy(ql.view(np.int16)))
            prefill[b, l] = pl
    torch.cuda.synchronize()
    log(f"[bench] inputs resident in HBM after {time.time() - t0:.1f}s")

    # one segment's complement block over all tidal heads (uniform retention): K and V rows of
    # every tidal head, bf16
    block_bytes = w.n_tidal * 2 * (w.chunk_len - w.budget_bp * w.chunk_len // 10000) * D * 2

    def recall_for(timing):
        # copy engines with next-step timing once a segment block is large enough to amortise a
        # transfer's fixed cost (measured: 3.2 MB blocks 1757 vs 1670 steps/s; 0.48 MB blocks
        # 6335 vs 6407); work-groups reading pinned memory otherwise, and with same-step timing
        if args.recall != "auto":
            return args.recall
        return "memcpy" if timing == "next" and block_bytes >= (1 << 20) else "kernel"

    main_run = run_timing(W, torch, w, args.timing, recall_for(args.timing), kd, vd, qd, roles, prefill, args,
                          args.chunks, args.retention)
    other = other_ch = None
    args_other = argparse.Namespace(**{**vars(args), "calibrate_copy": False, "sweep": False})
    if not args.no_other_timing:
        other_timing = "same" if args.timing == "next" else "next"
        other = run_timing(W, torch, w, other_timing, recall_for(other_timing), kd, vd, qd, roles, prefill, args_other,
                           args.chunks, args.retention)
    other_chunks = "overlap" if args.chunks == "disjoint" else "disjoint"
    if not args.no_other_chunks:
        other_ch = run_timing(W, torch, w, args.timing, recall_for(args.timing), kd, vd, qd, roles, prefill,
                              args_other, other_chunks, args.retention)
    other_retention = "per-head" if args.retention == "uniform" else "uniform"
    other_ret = None
    if not args.no_other_retention:
        other_ret = run_timing(W, torch, w, args.timing, recall_for(args.timing), kd, vd, qd, roles, prefill,
                               args_other, args.chunks, other_retention)
    prefill_res = None if args.no_prefill else prefill_bench(W, torch, w, kd, vd, roles)
    triage_res = None if args.no_prefill else triage_bench(W, torch, w, kd)
    del kd, vd
    torch.cuda.empty_cache()

    K = args.steps
    st1 = main_run["st1"]
    res = {
        "metric": METRIC, "value": main_run["value"], "unit": "steps/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": main_run["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name, "batch": B, "layers": L, "q_heads": w.q_heads, "kv_heads": H,
                   "head_dim": D, "audio_len": w.audio_len, "text_len": w.text_len, "chunk_len": w.chunk_len,
                   "budget_bp": w.budget_bp, "roles": [w.n_anchor, w.n_tidal, w.n_fixed], "kv_storage": "bf16",
                   "selection_timing": args.timing, "recall": recall_for(args.timing), "chunks": args.chunks,
                   "retention": args.retention if args.retention == "uniform" else f"per-head, lambda {args.lam}",
                   "clip_steps": main_run["clip_steps"],
                   "timed_region": "no timing events (per-kernel figures come from a second context that records them)"},
    }
    if "kernels" in main_run:
        k = main_run["kernels"]
        first = main_run["first"]
        res["kernels"] = k
        res["roofline"] = attention_roofline(k, first, w.name)
    res["recall"] = main_run["recall"]
    if main_run["recall"].get("GBps"):
        # the recall is bound by the host link (PCIe 5.0 x16, 64 GB/s per direction)
        gb = main_run["recall"]["GBps"]
        res["recall"]["roofline"] = {"bound": "host link", "achieved": gb, "peak": PEAK_LINK_GBPS, "unit": "GB/s",
                                     "frac": gb / PEAK_LINK_GBPS}
    if main_run.get("sweep"):
        res["overlap_sweep"] = main_run["sweep"]
        # share of the recall hidden behind the step at the workload's own recall load
        rm = main_run["recall"]
        if rm.get("ms"):
            res["recall"]["overlap"] = max(0.0, min(1.0, 1.0 - (main_run["ms_per_step"] - rm["step_ms_no_recall"]) / rm["ms"]))
    res["r_gpu"] = st1["r_gpu"]
    res["r_gpu_cpu"] = st1["r_gpu_cpu"]
    if other is not None:
        o = {"selection_timing": other_timing, "recall": recall_for(other_timing), "value": other["value"],
             "unit": "steps/s", "ms_per_step": other["ms_per_step"], "recall": other["recall"]}
        if "kernels" in other:
            o["kernels"] = other["kernels"]
        res["other_timing"] = o
    if other_ch is not None:
        o = {"chunks": other_chunks, "selection_timing": args.timing, "value": other_ch["value"], "unit": "steps/s",
             "ms_per_step": other_ch["ms_per_step"], "n_chunks": other_ch["geo"]["n_chunks"],
             "n_segments": other_ch["geo"]["n_segments"], "recall": other_ch["recall"]}
        if "kernels" in other_ch:
            o["kernels"] = other_ch["kernels"]
        res["other_chunks"] = o
    if other_ret is not None:
        o = {"retention": other_retention if other_retention == "uniform" else f"per-head, lambda {args.lam}",
             "chunks": args.chunks, "selection_timing": args.timing, "value": other_ret["value"], "unit": "steps/s",
             "ms_per_step": other_ret["ms_per_step"], "r_gpu": other_ret["r_gpu"], "r_gpu_cpu": other_ret["r_gpu_cpu"],
             "recall": other_ret["recall"]}
        if "kernels" in other_ret:
            o["kernels"] = other_ret["kernels"]
        res["other_retention"] = o

    # the paper's own runtime figures (runtime table): end-to-end decode of the whole model with
    # the recall active, on other hardware; context only, not comparable with this step alone
    res["paper_context"] = {"scope": "end-to-end decode of the whole Voxtral-mini-3B model, recall active",
                            "hardware": "1x A100, batch 1", "median_ms_per_token": [26.7, 27.8],
                            "recall_MB_per_step": [0.05, 1.04], "r_gpu": [0.197, 0.217]}
    if prefill_res is not None:
        res["prefill"] = prefill_res
    if triage_res is not None:
        res["triage"] = triage_res
    if args.cpu_seconds > 0:
        res["cpu_baseline"] = cpu_baseline(w, roles, prefill, args.cpu_seconds)
    print(json.dumps(res), flush=True)


# rocprofv3 names of the launches behind the bench's kernel keys (the headline's group of 4)
# (the tidal/fixed launch of next-step timing has two instantiations: without and with the
# chunk-mass merge and the selection inside it)
PROFILE_NAMES = {"attention": "attention_kernel<4>", "tidal_fixed": "tidal_fixed_kernel<4, 8, false, false/true>"}


def attention_roofline(k, first, workload):
    """HBM roofline of the attention launches: per launch (algorithmic bytes / its average
    duration from HIP events bound to the launch) and together (sum of bytes / sum of
    durations), over the timed steps with the recall running beside them; traffic from the
    committed counter summaries when they match the current kernels."""
    per = {}
    for name in (first, "tidal_fixed"):
        e = k[name]
        gb = e["GBps"]
        per[name] = {"kernel": PROFILE_NAMES.get(name, name), "achieved": gb, "avg_ms": e["avg_ms"],
                     "bytes": e["bytes"], "frac": gb / PEAK_HBM_GBPS if gb else None,
                     "traffic": measured_traffic(name, workload),
                     "achieved_without_recall": k[name + "_pinned_selection"]["GBps"]}
    tot_b = sum(p["bytes"] for p in per.values())
    tot_ms = sum(p["avg_ms"] for p in per.values())
    tr = [p["traffic"] for p in per.values()]
    pin_b = sum(k[n + "_pinned_selection"]["bytes"] for n in per)
    pin_ms = sum(k[n + "_pinned_selection"]["avg_ms"] for n in per)
    agg = tot_b / tot_ms / 1e6
    return {"bound": "hbm", "kernel": " + ".join(p["kernel"] for p in per.values()), "achieved": agg,
            "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": agg / PEAK_HBM_GBPS,
            "traffic": sum(tr) if all(t is not None for t in tr) else None,
            "achieved_without_recall": pin_b / pin_ms / 1e6, "per_launch": per,
            "note": "all attention launches of a step (anchor + static tiles, then the slot groups of the resident "
                    "complements): sum of algorithmic bytes / sum of launch durations (HIP events bound to each "
                    "launch) over the timed steps, recall beside them; achieved_without_recall: selection pinned"}


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter summary
    (FETCH_SIZE + WRITE_SIZE per dispatch, each scaled by what the counter reads for a plain
    copy of known size), or None when there is no summary or the kernel source has changed
    since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_pmc.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    src = os.path.join(ROOT, "paper_2608_22704_amd", "csrc", "wnw_kernels.hip")
    if vals.get("kernels_source_sha256") != hashlib.sha256(open(src, "rb").read()).hexdigest():
        return None
    try:
        fetch = float(vals["fetch_kib_per_dispatch"]) * 1024 / float(vals["fetch_copy_factor"])
        write = float(vals["write_kib_per_dispatch"]) * 1024 / float(vals["write_copy_factor"])
    except (KeyError, ValueError, ZeroDivisionError):
        return None
    return fetch + write


def prefill_bench(W, torch, w, kd, vd, roles, reps=5):
    """Prefill compression on the device for the workload: wnw_prefill_scores (text-to-audio
    attention sums over the synthetic text queries, two MFMA passes) timed with events on the
    set-up stream, then wnw_set_roles_device against wnw_set_roles (host ranking) on the same
    scores.  Algorithmic flops: 2 d per logit of the method's one causal text-to-cache QK^T
    (T_a + t + 1 keys for text token t), over every q-head; the kernels' second pass recomputes
    the audio logits (a further T_a keys per text token), which is reported beside it as
    executed work."""
    from synth import gen
    B, L, H, D, Ta, Tt, g = w.batch, w.layers, w.kv_heads, w.head_dim, w.audio_len, w.text_len, w.group
    qt = torch.empty((B, L, w.q_heads, Tt, D), dtype=torch.int16, device="cuda")
    for b in range(B):
        kb = kd[b].cpu().numpy().view(np.uint16)
        for l in range(L):
            for kv in range(H):
                qt[b, l, kv * g:(kv + 1) * g].copy_(torch.from_numpy(gen.text_queries(w, b, l, kv, kb[l, kv]).view(np.int16)))
    sc = torch.empty((B, L, H, Ta), dtype=torch.float32, device="cuda")
    cfg = W.make_config(B, L, w.q_heads, H, Ta, Tt, w.chunk_len, w.budget_bp, flags=W.WNW_F_SELECT_NEXT_STEP)
    stream = torch.cuda.current_stream()
    flop = 2.0 * D * g * L * H * B * (Tt * (Ta + 1) + Tt * (Tt - 1) / 2)
    flop_exec = flop + 2.0 * D * g * L * H * B * Tt * Ta
    ctx = W.wnw_init_cache(cfg, kd, vd, stream)
    try:
        W.wnw_prefill_scores(ctx, qt, sc)            # warm-up
        ms = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            W.wnw_prefill_scores(ctx, qt, sc)
            e1.record(stream)
            e1.synchronize()
            ms.append(e0.elapsed_time(e1))
        t0 = time.perf_counter()
        W.wnw_set_roles_device(ctx, roles, sc)
        t_dev = time.perf_counter() - t0
    finally:
        W.wnw_destroy(ctx)
    host_sc = sc.cpu().numpy()
    ctx = W.wnw_init_cache(cfg, kd, vd, stream)
    try:
        t0 = time.perf_counter()
        W.wnw_set_roles(ctx, roles, host_sc)
        t_host = time.perf_counter() - t0
    finally:
        W.wnw_destroy(ctx)
    avg = sum(ms) / len(ms)
    tf = flop / (avg * 1e-3) / 1e12
    log(f"[bench] prefill scores {avg:.3f} ms ({tf:.0f} TFLOP/s); set_roles device {t_dev:.2f} s, host {t_host:.2f} s")
    tfx = flop_exec / (avg * 1e-3) / 1e12
    return {"scores_ms": avg, "flop": flop, "achieved_tflops": tf, "peak_tflops": PEAK_BF16_TFLOPS,
            "frac": tf / PEAK_BF16_TFLOPS, "flop_executed": flop_exec, "executed_tflops": tfx,
            "executed_frac": tfx / PEAK_BF16_TFLOPS, "set_roles_device_s": t_dev, "set_roles_host_s": t_host,
            "note": "one-time set-up, outside the decode step; scores_ms over both MFMA passes (HIP events); flop "
                    "counts the causal QK^T once, flop_executed adds the second pass's recomputed audio logits"}


def triage_bench(W, torch, w, kd, n_tok=64, reps=5):
    """Head triage arithmetic at the workload's shapes (one calibration sample): voice-score hits
    of n_tok answer tokens (fp64 dot products over every audio key: 2 d flops per token, q-head
    and audio key), and the key sensitivity of one answer token (a read of its fp32 key gradients:
    L * H_kv * T_a * d * 4 bytes).  Synthetic inputs; calibration itself is offline."""
    L, Hq, H, D, Ta, T = w.layers, w.q_heads, w.kv_heads, w.head_dim, w.audio_len, w.total_len
    g = torch.Generator(device="cuda").manual_seed(5)
    q = torch.randn((n_tok, L, Hq, D), device="cuda", generator=g).to(torch.bfloat16).view(torch.int16)
    a = torch.randint(0, max(Ta - 8, 1), (n_tok,), device="cuda", generator=g)
    span = torch.stack([a, a + 8], dim=1).to(torch.int32).contiguous()
    hits = torch.empty((n_tok, L, Hq), dtype=torch.int32, device="cuda")
    k0 = kd[0].contiguous()
    grad = torch.randn((1, L, H, Ta, D), device="cuda", generator=g, dtype=torch.float32)
    sens = torch.empty((1, L, H), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    def timed(fn):
        fn()
        ms = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            e1.synchronize()
            ms.append(e0.elapsed_time(e1))
        return sum(ms) / len(ms)

    vh = timed(lambda: W.wnw_voice_hits(k0, q, span, 4, Ta, hits))
    ks = timed(lambda: W.wnw_key_sensitivity(grad, sens))
    flop = 2.0 * D * n_tok * L * Hq * Ta
    nbytes = float(L * H * Ta * D * 4)
    del grad
    log(f"[bench] triage: voice hits {vh:.3f} ms, key sensitivity {ks:.3f} ms")
    return {"voice_hits_ms": vh, "voice_hits_tokens": n_tok, "voice_hits_tflops": flop / (vh * 1e-3) / 1e12,
            "voice_hits_frac": flop / (vh * 1e-3) / 1e12 / PEAK_FP64_TFLOPS, "voice_hits_bound": "fp64 mfma",
            "key_sensitivity_ms": ks, "key_sensitivity_GBps": nbytes / (ks * 1e-3) / 1e9,
            "key_sensitivity_frac": nbytes / (ks * 1e-3) / 1e9 / PEAK_HBM_GBPS,
            "note": "offline calibration arithmetic on synthetic inputs; one sample, K = 4"}


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo), or None."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(w, roles, prefill, budget_s):
    """The CPU oracle on the first decode steps of sequence 0 of the same workload, all heads:
    steps/s over a bounded sample with every host thread (OpenMP across heads), then over a
    shorter sample with one thread."""
    from oracle import oracle as O
    from synth import gen

    log(f"[bench] CPU oracle sample (~{budget_s:.0f}s + ~{budget_s * 2 / 3:.0f}s on one thread)")
    seq = gen.sequence(w.with_(batch=1), 0) if w.batch == 1 else gen.sequence(w, 0)

    def sample(seconds):
        o = O.Oracle(O.cfg_from_workload(w, batch=1), seq["k"][None], seq["v"][None], roles, prefill[:1])
        n, t0 = 0, time.perf_counter()
        while n == 0 or (time.perf_counter() - t0 < seconds and n < w.steps):
            o.step(seq["q"][n][None])
            n += 1
        el = time.perf_counter() - t0
        o.close()
        return n, el

    cores = O.set_threads(0)
    n, el = sample(budget_s)
    O.set_threads(1)
    n1, el1 = sample(budget_s * 2 / 3)
    O.set_threads(cores)
    return {"value": n / el, "unit": "steps/s", "cores": cores, "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"first {n} decode steps of sequence 0 of {w.name}, every head, double precision, "
                      f"{cores} threads ({el:.1f}s)",
            "value_1_core": n1 / el1, "sample_1_core": f"first {n1} steps on one thread ({el1:.1f}s)"}


if __name__ == "__main__":
    main()
