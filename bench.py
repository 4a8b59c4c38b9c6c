"""Benchmark of the shared-stage hot path on one MI355X.

Headline: prefill tokens/s of the 4-layer thinker stack (hidden 3584, 28/4
heads, head_dim 128, FFN 18944) over the seeded ragged batch of 8 requests
(T = 10,515 rows), at the full 256-CU budget.  Also reported: the same stack
at CU budgets 64/128/192 (fraction of the CU-scaled bf16 MFMA peak) and the
spatial co-run of that prefill on a 128-CU mask with a 16-layer talker decode
step (batch 32) looping on the complementary 128 CUs.

Prints one JSON line.  The CPU reference is timed on a bounded sample of the
same workload (rank 0, N = 1 only).
"""
from __future__ import annotations

import argparse
import dataclasses
import gc
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16 = 2.5e15       # MI355X dense bf16/fp16 MFMA, FLOP/s, 256 CUs
PEAK_HBM = 8.0e12        # bytes/s
N_CUS = 256
SPEC_MHZ = 2400.0        # clock of the published peak


# HBM-side bytes per gate/up launch at 256 CUs from rocprofv3 FETCH_SIZE and
# WRITE_SIZE passes (KiB per dispatch), each scaled by what the counter reads for a
# 1 GiB device copy (fetch x 2.000, write x 1.000).  Valid only for the GEMM
# source these counters were taken on.
MEASURED_TRAFFIC = {
    "35c5cac0be380a8f": {"fetch_kib": 2241038.6, "fetch_scale": 2.0, "write_kib": 397954.7, "write_scale": 1.0},
    "b13966ab4f6ab1ce": {"fetch_kib": 2240940.5, "fetch_scale": 2.0, "write_kib": 400059.4, "write_scale": 1.0},
    "03c73fb21179ef2c": {"fetch_kib": 2241088.2, "fetch_scale": 2.0, "write_kib": 399894.8, "write_scale": 1.0},
    "f9d19f9ce46f207e": {"fetch_kib": 2245197.3, "fetch_scale": 2.0, "write_kib": 399491.4, "write_scale": 1.0},
    "e964d3aa53b0007d": {"fetch_kib": 2224511.9, "fetch_scale": 2.0, "write_kib": 397264.2, "write_scale": 1.0},
    "d4915bf77392150d": {"fetch_kib": 2226951.2, "fetch_scale": 2.0, "write_kib": 397023.8, "write_scale": 1.0},
    "adc65d4733f8721b": {"fetch_kib": 2315757.9, "fetch_scale": 2.0, "write_kib": 395098.1, "write_scale": 1.0},
}


def gemm_traffic_bytes():
    import hashlib
    with open(os.path.join(ROOT, "paper_2608_01785_amd", "csrc", "gemm.hip"), "rb") as f:
        key = hashlib.sha256(f.read()).hexdigest()[:16]
    m = MEASURED_TRAFFIC.get(key)
    if m is None:
        return None
    return int(1024 * (m["fetch_kib"] * m["fetch_scale"] + m["write_kib"] * m["write_scale"]))


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def thinker_flops(shape, lengths, ctx=None):
    """Algorithmic FLOPs of one layer: 2 * params per row + 4 * Hq * dh per visible (query, key) pair."""
    L = np.asarray(lengths, np.int64)
    c = np.zeros_like(L) if ctx is None else np.asarray(ctx, np.int64)
    params = shape.params_per_layer
    pairs = int(np.sum(L * c + L * (L + 1) // 2))
    return 2.0 * params * int(L.sum()), 4.0 * shape.n_q_heads * shape.head_dim * pairs


def talker_bytes(shape, n_layers, kv_lens):
    """HBM bytes of one decode step: weights once + cached K/V read + new K/V written."""
    per_tok = 2 * shape.n_kv_heads * shape.head_dim * 2  # K and V, fp16, per layer
    kv = np.asarray(kv_lens, np.int64)
    return n_layers * (shape.params_per_layer * 2 + per_tok * int(kv.sum()) + per_tok * len(kv))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--budgets", type=str, default="64,128,192")
    ap.add_argument("--no-corun", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-controller", action="store_true")
    ap.add_argument("--no-tpot", action="store_true")
    ap.add_argument("--no-mixed", action="store_true")
    ap.add_argument("--no-loop", action="store_true")
    ap.add_argument("--no-dit", action="store_true")
    # Profiling runs (under rocprofv3): one piece of work only, then exit.
    ap.add_argument("--profile-budget", type=int, default=0,
                    help="run only the thinker stack at this CU budget, --steps times")
    ap.add_argument("--profile-decode", action="store_true",
                    help="run only the talker decode step (batch 32, 16 layers) on 128 CUs, --steps times")
    ap.add_argument("--profile-ladder", action="store_true",
                    help="launch the topology probe once on every stream of the bench's ladder")
    ap.add_argument("--cpu-rows", type=int, default=0,
                    help="rows per sequence in the CPU-reference sample (0: sized to take about 15 s)")
    ap.add_argument("--quick", action="store_true", help="headline stack only (no budget sweep, co-run, CPU leg)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one device copy of this many MiB (counter calibration under a profiler)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "bench.py measures one GPU only: the path is a single-GPU spatial-sharing design "
                                   "(run with --gpus 1)"}))
        sys.exit(2)

    import torch
    from paper_2608_01785_amd import binding, workloads as W
    from paper_2608_01785_amd.device_data import DeviceCache, prepare_f16, to_device, upload_weights

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = "cuda:0"
    budgets = [int(b) for b in args.budgets.split(",") if b]
    if args.quick:
        budgets, args.no_corun, args.no_cpu_baseline, args.no_controller, args.no_tpot = [], True, True, True, True
        args.no_mixed = True
        args.no_loop = True
        args.no_dit = True
    # One context holds every level the sections below use (each level is a
    # pair of CU-masked hardware queues).
    # The timed loops issue many short library calls from Python.  A cyclic
    # garbage-collection pass over the objects that earlier sections built
    # stalled one call by ~37 ms inside a timed loop, so the collector runs
    # only between sections.
    gc.disable()
    ladder = sorted(set(budgets + [96, 128, 160, 224, 256] + ([] if args.no_tpot else TPOT_CAPS)
                        + ([] if args.no_corun else [N_CUS - c for c in DOWN_SWEEP])))
    if args.profile_budget or args.profile_decode or args.profile_ladder:
        return profile_only(args, torch, binding, W, ladder)
    ctx = binding.Context(0, budgets=ladder)

    # ---------------------------------------------------------------- thinker stack
    shape, n_layers = W.THINKER, 4
    t0 = time.time()
    layers = W.make_weights(shape, n_layers, W.SEEDS["thinker"]["weights"])
    batch = W.thinker_batch()
    log(f"[bench] generated thinker weights/batch in {time.time() - t0:.1f}s, T={batch.n_tokens}")
    wbf16 = upload_weights(layers, dev)
    # One-time weight preparation: fp16 copies of the projection matrices
    # (the MFMA operand type); the bf16 originals are timed once as well.
    wdev = prepare_f16(ctx, wbf16)
    x = to_device(batch.x, dev)
    y = torch.empty(x.shape, dtype=torch.float32, device=dev)
    T, B = batch.n_tokens, batch.n_seqs
    max_pos = int(batch.lengths.max())
    ws = torch.empty(binding.hs_workspace_size(shape, T, B, max_pos), dtype=torch.uint8, device=dev)
    lin, att = thinker_flops(shape, batch.lengths)
    flops_step = n_layers * (lin + att)
    torch.cuda.synchronize()

    def run(budget, k, weights=None):
        weights = wdev if weights is None else weights
        s = binding.hs_context_stream(ctx, budget, binding.HS_ROLE_SHARED)
        ts = torch.cuda.ExternalStream(s)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(ts)
        for _ in range(k):
            binding.hs_shared_stage_forward(ctx, shape, weights, x, y, batch.seq_offsets, None, None, budget, None, ws)
        e1.record(ts)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / k

    def instrumented(budget, k):
        """Per-kernel event times and sustained clocks over k more steps (outside the timed loops)."""
        binding.hs_timing_enable(ctx, True)
        run(budget, k)
        kern = {n: binding.hs_timing_read(ctx, n) for n in binding.KERNEL_KINDS}
        clk = {n: binding.hs_timing_read_clock(ctx, n)[0] for n in binding.KERNEL_KINDS}
        binding.hs_timing_enable(ctx, False)
        return ({n: (v[0] / v[1] if v[1] else 0.0) for n, v in kern.items()},
                {n: round(v, 1) for n, v in clk.items() if v > 0})

    for _ in range(args.warmup):
        run(256, 1)
    # The headline loop runs without per-kernel events; a separate pass
    # records them.
    ms = run(256, args.steps)
    kernel_ms, clock_mhz = instrumented(256, max(2, args.steps // 2))
    tok_s = T / (ms / 1e3)
    log(f"[bench] thinker stack @256 CUs: {ms:.3f} ms/step, {tok_s:,.0f} tok/s, "
        f"{flops_step / (ms / 1e3) / 1e12:.1f} TFLOP/s")
    for k, v in kernel_ms.items():
        if v:
            log(f"    {k:12s} {v:8.3f} ms avg" + (f", clock {clock_mhz[k]:.0f} MHz" if k in clock_mhz else ""))

    # Dominant kernel: the gate/up projection (SwiGLU epilogue), ~58 % of the FLOPs.
    gu_flops = 2.0 * T * shape.hidden * 2 * shape.ffn
    gu_ms = kernel_ms["gate_up"]
    gu_bytes = 2 * (T * shape.hidden + 2 * shape.ffn * shape.hidden + T * shape.ffn)  # A, W, a (fp16)
    achieved = gu_flops / (gu_ms / 1e3) / 1e12
    gu_mhz = clock_mhz.get("gate_up")
    roofline = {"bound": "mfma", "kernel": "gate_up_swiglu_gemm", "achieved": round(achieved, 1),
                "peak": PEAK_BF16 / 1e12, "unit": "TFLOP/s", "frac": round(achieved / (PEAK_BF16 / 1e12), 4),
                "traffic": gemm_traffic_bytes(), "algorithmic_bytes": gu_bytes, "avg_launch_ms": round(gu_ms, 4),
                # The same against the peak at the launch's measured sustained clock.
                "clock_mhz": gu_mhz,
                "frac_at_measured_clock": round(achieved / (PEAK_BF16 / 1e12 * gu_mhz / SPEC_MHZ), 4) if gu_mhz else None}

    run(256, 1, wbf16)
    ms_bf16w = run(256, max(2, args.steps // 2), wbf16)
    log(f"[bench] thinker stack @256 CUs with bf16 weights converted in the GEMM: {ms_bf16w:.3f} ms/step")

    def budget_entry(b, mb, kms, clk):
        """Stack rate at budget b, with the GEMMs' average clock (launch-time weighted) and the
        fraction of the CU-scaled peak at that clock."""
        gem = [k for k in ("qkv", "o_proj", "gate_up", "down") if k in clk and kms.get(k)]
        mhz = sum(clk[k] * kms[k] for k in gem) / sum(kms[k] for k in gem) if gem else None
        frac = flops_step / (mb / 1e3) / (PEAK_BF16 * b / N_CUS)
        return {"ms_per_step": round(mb, 3), "tok_s": round(T / (mb / 1e3)), "mfma_frac_cu_scaled": round(frac, 4),
                "gemm_clock_mhz": round(mhz, 1) if mhz else None,
                "mfma_frac_cu_scaled_at_measured_clock": round(frac * SPEC_MHZ / mhz, 4) if mhz else None,
                "kernel_ms": {k: round(v, 4) for k, v in kms.items() if v}}

    per_budget = {}
    for b in budgets:
        if b == 256:
            continue
        run(b, 1)
        mb = run(b, max(2, args.steps // 2))
        kms, clk = instrumented(b, 1)
        per_budget[str(b)] = budget_entry(b, mb, kms, clk)
        log(f"[bench] thinker stack @{b} CUs: {mb:.3f} ms/step, {T / (mb / 1e3):,.0f} tok/s, "
            f"GEMM clock {per_budget[str(b)]['gemm_clock_mhz']} MHz")
    per_budget["256"] = budget_entry(256, ms, kernel_ms, clock_mhz)

    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {args.calib_copy_mib} MiB done")
        del src, dst

    # ---------------------------------------------------------------- co-run
    gc.collect()
    corun = None
    if not args.no_corun:
        corun = corun_measure(torch, binding, W, ctx, shape, wdev, x, y, batch, ws, dev, flops_step)

    # ---------------------------------------------------------------- second downstream workload (DiT)
    gc.collect()
    dit = None
    if not args.no_dit:
        dit = dit_corun(torch, binding, W, ctx, shape, wdev, x, y, batch, ws, dev, flops_step)

    # ---------------------------------------------------------------- downstream-heavy mixed step
    gc.collect()
    mixed = None
    if not args.no_mixed:
        mixed = corun_mixed(torch, binding, W, ctx, dev)

    # ---------------------------------------------------------------- shared-stage decode TPOT vs CU cap
    gc.collect()
    tpot = None
    if not args.no_tpot:
        tpot = thinker_decode_sweep(torch, binding, W, ctx, shape, wdev, n_layers, dev)

    # ---------------------------------------------------------------- spatial controller costs
    gc.collect()
    controller = None
    if not args.no_controller:
        controller = controller_measure(torch, binding, ctx, [b for b in ladder if b < N_CUS], dev)

    # ---------------------------------------------------------------- Algorithm 1 on the GPU
    loop = None
    if not args.no_loop:
        gc.collect()
        # B_sat: the talker's traffic share where its step stops improving with more CUs
        # (the largest share over the complement sweep).
        b_sat = 0.25
        if corun is not None:
            tb = corun["decode_bytes_per_step"]
            b_sat = round(max(tb / (ms_ / 1e3) / PEAK_HBM for ms_ in corun["decode_ms_vs_cus"].values()), 4)
        # Six seeded arrival streams per policy: one 48-request stream is a small sample
        # (a stream's short-path attainment moves in steps of ~0.04), so the means and the
        # spread across streams are reported.
        loop = {"runs": [], "seeds": LOOP_SEEDS}
        for p, sb in (("baseline", 0), ("joint", 0), ("joint", 1024)):
            runs = [serving_loop(torch, binding, W, ctx, wdev, dev, p, saturation=b_sat, short_budget=sb, seed=sd)
                    for sd in LOOP_SEEDS]
            loop["runs"] += runs
            agg = {"policy": p, "short_budget": runs[0]["short_budget"], "saturation": b_sat}
            for c in ("short", "long"):
                agg[c] = {k: round(float(np.mean([r[c][k] for r in runs if r[c][k] is not None])), 4)
                          for k in ("slo_attainment", "p50_ms", "p95_ms")}
            for c in ("short", "long"):
                att = [r[c]["slo_attainment"] for r in runs if r[c]["slo_attainment"] is not None]
                agg[c]["slo_attainment_sd"] = round(float(np.std(att)), 4) if att else None
            agg["mean_shared_cus"] = round(float(np.mean([r["mean_shared_cus"] for r in runs])), 1)
            agg["makespan_ms"] = round(float(np.mean([r["makespan_ms"] for r in runs])), 2)
            loop.setdefault("mean_over_seeds", []).append(agg)
            log(f"[bench] serving loop mean over seeds {LOOP_SEEDS} ({p}, short budget {agg['short_budget']}): "
                f"short SLO {agg['short']['slo_attainment']:.3f} (sd {agg['short']['slo_attainment_sd']}) "
                f"p95 {agg['short']['p95_ms']:.1f} ms, long SLO "
                f"{agg['long']['slo_attainment']:.3f} p95 {agg['long']['p95_ms']:.1f} ms")
        for r in loop["runs"][1:]:      # one step trace is kept, to keep the line short
            r.pop("trace", None)

    # ---------------------------------------------------------------- serving-loop model on measured times
    policy = None
    if corun is not None and "unmasked" in corun:
        gc.collect()
        policy = policy_model(W, shape, batch, per_budget, corun)

    # ---------------------------------------------------------------- CPU reference sample
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(W, layers, batch, shape, args.cpu_rows)

    out = {
        "metric": "shared-stage prefill tok/s vs CU budget (% MFMA roofline); co-run decode tok/s",
        "value": round(tok_s, 1),
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic (seeded N(0,0.02) bf16 weights, N(0,1) bf16 token rows); fp16 MFMA operands, "
                "fp32 accumulation and residual stream",
        "config": {"workload": "thinker 4-layer stack prefill, hidden 3584, 28/4 heads, dh 128, ffn 18944, "
                               "8 ragged requests T=10515, 256 CUs",
                   "global_batch": B, "seq_len": int(batch.lengths.max()), "tokens": T,
                   "parallelism": "single GPU, CU-masked streams"},
        "tflops": round(flops_step / (ms / 1e3) / 1e12, 1),
        "mfma_frac": round(flops_step / (ms / 1e3) / PEAK_BF16, 4),
        "roofline": roofline,
        "kernel_ms": {k: round(v, 4) for k, v in kernel_ms.items() if v},
        "kernel_clock_mhz": clock_mhz,
        "ms_per_step_bf16_weights": round(ms_bf16w, 4),
        "budgets": per_budget,
        "corun": corun,
        "mixed_corun": mixed,
        "dit_corun": dit,
        "decode_tpot_vs_cus": tpot,
        "controller": controller,
        "policy_model": policy,
        "serving_loop": loop,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    torch.cuda.synchronize()
    ctx.close()


def profile_only(args, torch, binding, W, ladder):
    """A single piece of work for a profiler run: the thinker stack at one budget, the talker
    decode step, or one probe launch on every stream of the bench's ladder (the full ladder,
    as the default run builds it).  Prints one JSON line."""
    from paper_2608_01785_amd.device_data import DeviceCache, prepare_f16, to_device, upload_weights
    dev = "cuda:0"
    full_ladder = sorted(set([64, 128, 192, 96, 160, 224, 256] + TPOT_CAPS + [N_CUS - c for c in DOWN_SWEEP]))
    ctx = binding.Context(0, budgets=full_ladder if args.profile_ladder else
                          sorted(set([128, 256] + ([args.profile_budget] if args.profile_budget else []))))
    out = {}
    try:
        if args.profile_ladder:
            ids = torch.zeros(1024 * 4, dtype=torch.int32, device=dev)
            streams = []
            for b in full_ladder:
                for role in (binding.HS_ROLE_SHARED, binding.HS_ROLE_DOWN):
                    if role == binding.HS_ROLE_DOWN and b == N_CUS:
                        continue
                    s = binding.hs_context_stream(ctx, b, role)
                    binding.hs_probe_hw_ids(ctx, s, 1024, ids)
                    torch.cuda.synchronize()
                    streams.append((b, role))
            out = {"probe_launches": len(streams), "levels": full_ladder}
        elif args.profile_budget:
            shape, n_layers = W.THINKER, 4
            layers = W.make_weights(shape, n_layers, W.SEEDS["thinker"]["weights"])
            batch = W.thinker_batch()
            wdev = prepare_f16(ctx, upload_weights(layers, dev))
            x = to_device(batch.x, dev)
            y = torch.empty(x.shape, dtype=torch.float32, device=dev)
            ws = torch.empty(binding.hs_workspace_size(shape, batch.n_tokens, batch.n_seqs, int(batch.lengths.max())),
                             dtype=torch.uint8, device=dev)
            b = args.profile_budget
            s = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, b, binding.HS_ROLE_SHARED))
            for _ in range(args.warmup):
                binding.hs_shared_stage_forward(ctx, shape, wdev, x, y, batch.seq_offsets, None, None, b, None, ws)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            for _ in range(args.steps):
                binding.hs_shared_stage_forward(ctx, shape, wdev, x, y, batch.seq_offsets, None, None, b, None, ws)
            e1.record(s)
            torch.cuda.synchronize()
            out = {"budget": b, "ms_per_step": round(e0.elapsed_time(e1) / args.steps, 3)}
        else:
            ts, n_layers, bt = W.TALKER, 16, 32
            seeds = W.SEEDS["talker"]
            kv_lens = W.talker_kv_lens(bt, seeds["cache"])
            tl = prepare_f16(ctx, upload_weights(W.make_weights(ts, n_layers, seeds["weights"]), dev))
            max_ctx = int(np.ceil((kv_lens.max() + 1) / 64) * 64)
            cache = DeviceCache(n_layers, bt, max_ctx, ts.n_kv_heads, ts.head_dim, dev)
            gen = torch.Generator(device=dev)
            gen.manual_seed(seeds["cache"])
            for l in range(n_layers):
                for b in range(bt):
                    cache.fill_random(l, b, int(kv_lens[b]), gen)
            xt = to_device(W.talker_batch(ts, n_layers, bt, seeds, with_cache=False).x, dev)
            yt = torch.empty(xt.shape, dtype=torch.float32, device=dev)
            wst = torch.empty(binding.hs_workspace_size(ts, bt, bt, int(kv_lens.max()) + 1), dtype=torch.uint8,
                              device=dev)
            s = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, 128, binding.HS_ROLE_DOWN))
            for _ in range(args.warmup):
                binding.hs_downstream_decode_step(ctx, ts, tl, xt, yt, cache.as_arg(), kv_lens, 128, None, wst)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            for _ in range(args.steps):
                binding.hs_downstream_decode_step(ctx, ts, tl, xt, yt, cache.as_arg(), kv_lens, 128, None, wst)
            e1.record(s)
            torch.cuda.synchronize()
            out = {"decode_ms_per_step": round(e0.elapsed_time(e1) / args.steps, 4),
                   "bytes_per_step": talker_bytes(ts, n_layers, kv_lens)}
        if args.calib_copy_mib:
            n = args.calib_copy_mib * (1 << 20) // 4
            src = torch.ones(n, dtype=torch.float32, device=dev)
            dst = torch.empty_like(src)
            torch.cuda.synchronize()
            dst.copy_(src)
            torch.cuda.synchronize()
            out["calibration_copy_mib"] = args.calib_copy_mib
    finally:
        torch.cuda.synchronize()
        ctx.close()
    print(json.dumps(out), flush=True)


def corun_measure(torch, binding, W, ctx, shape, wdev, x, y, batch, ws, dev, flops_step):
    """Prefill on a 128-CU mask while talker decode steps loop on the other 128 CUs."""
    from paper_2608_01785_amd.device_data import DeviceCache, to_device, upload_weights
    ts_shape, ts_layers, bt = W.TALKER, 16, 32
    seeds = W.SEEDS["talker"]
    kv_lens = W.talker_kv_lens(bt, seeds["cache"])
    from paper_2608_01785_amd.device_data import prepare_f16
    tl = prepare_f16(ctx, upload_weights(W.make_weights(ts_shape, ts_layers, seeds["weights"]), dev))
    max_ctx = int(np.ceil((kv_lens.max() + 1) / 64) * 64)
    cache = DeviceCache(ts_layers, bt, max_ctx, ts_shape.n_kv_heads, ts_shape.head_dim, dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(seeds["cache"])
    for l in range(ts_layers):
        for b in range(bt):
            cache.fill_random(l, b, int(kv_lens[b]), gen)
    xt = to_device(W.talker_batch(ts_shape, ts_layers, bt, seeds, with_cache=False).x, dev)
    yt = torch.empty(xt.shape, dtype=torch.float32, device=dev)
    wst = torch.empty(binding.hs_workspace_size(ts_shape, bt, bt, int(kv_lens.max()) + 1), dtype=torch.uint8, device=dev)
    step_bytes = talker_bytes(ts_shape, ts_layers, kv_lens)
    s_sh = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, 128, binding.HS_ROLE_SHARED))
    s_dn = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, 128, binding.HS_ROLE_DOWN))

    # The same step captured once and replayed (the serving path for a fixed batch).
    wsg = torch.empty(binding.hs_workspace_size(ts_shape, bt, bt, max_ctx), dtype=torch.uint8, device=dev)
    tgraph = binding.DecodeGraph(ctx, ts_shape, tl, xt, yt, cache.as_arg(), bt, 128, None, wsg)

    def decode(n, cus=128, stream=None, rec=None, graph=False):
        rec = s_dn if rec is None else rec
        ev = []
        for _ in range(n):
            if graph:
                tgraph.launch(kv_lens)
            else:
                binding.hs_downstream_decode_step(ctx, ts_shape, tl, xt, yt, cache.as_arg(), kv_lens, cus, stream,
                                                  wst)
            e = torch.cuda.Event(enable_timing=True)
            e.record(rec)
            ev.append(e)
        return ev

    def corun_window(prefill_stream, prefill_cus, dec_cus, dec_stream, dec_rec):
        """Prefill forward with decode steps looping beside it: (window ms, decode ms per step, steps)."""
        torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        start.record(prefill_stream)
        dec_rec.wait_event(start)
        binding.hs_shared_stage_forward(ctx, shape, wdev, x, y, batch.seq_offsets, None, None, prefill_cus, None, ws)
        p_end = torch.cuda.Event(enable_timing=True)
        p_end.record(prefill_stream)
        dec_ev = []
        while True:
            dec_ev += decode(1, dec_cus, dec_stream, dec_rec)
            if p_end.query():
                break
            if len(dec_ev) > 4:
                dec_ev[-4].synchronize()
            if len(dec_ev) > 2000:
                break
        torch.cuda.synchronize()
        window = start.elapsed_time(p_end)
        done = [start.elapsed_time(e) for e in dec_ev]
        n_in = sum(1 for t in done if t <= window)
        t_last = max([t for t in done if t <= window], default=0.0)
        return window, (t_last / n_in if n_in else float("nan")), n_in

    # Solo decode on its 128 CUs: replayed graph, and eager launches.
    def solo(graph):
        """(GPU ms per step, host ms per issued step) over 20 back-to-back steps."""
        torch.cuda.synchronize()
        decode(3, graph=graph)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e0.record(s_dn)
        t0 = time.perf_counter()
        ev = decode(20, graph=graph)
        host = (time.perf_counter() - t0) * 1e3 / 20
        torch.cuda.synchronize()
        return e0.elapsed_time(ev[-1]) / 20, host

    solo_ms, host_eager_ms = solo(False)
    solo_graph_ms, host_graph_ms = solo(True)

    # Per-kernel averages of the solo decode step (events on the decode stream).
    binding.hs_timing_enable(ctx, True)
    decode(10)
    torch.cuda.synchronize()
    dk = {k: binding.hs_timing_read(ctx, k) for k in binding.KERNEL_KINDS}
    binding.hs_timing_enable(ctx, False)
    dec_kernel_ms = {k: v[0] / v[1] for k, v in dk.items() if v[1]}
    # Dominant decode kernel: single-row attention, which reads every cached key/value row once.
    kv_bytes = 2 * ts_shape.n_kv_heads * ts_shape.head_dim * 2 * int(np.sum(kv_lens + 1))
    da_ms = dec_kernel_ms["decode_attn"]
    da_gbs = kv_bytes / (da_ms / 1e3) / 1e9
    w_bytes = {"qkv": ts_shape.qkv_rows * ts_shape.hidden * 2, "o_proj": ts_shape.hidden * ts_shape.n_q_heads * ts_shape.head_dim * 2,
               "gate_up": 2 * ts_shape.ffn * ts_shape.hidden * 2, "down": ts_shape.hidden * ts_shape.ffn * 2}
    decode_roofline = {
        "bound": "hbm", "kernel": "decode_attn", "cus": 128,
        "achieved": round(da_gbs, 1), "peak": PEAK_HBM / 1e9, "unit": "GB/s",
        "frac": round(da_gbs / (PEAK_HBM / 1e9), 4),
        "frac_cu_scaled": round(da_gbs / (PEAK_HBM / 1e9 * 128 / N_CUS), 4),
        "bytes_per_launch": kv_bytes, "avg_launch_ms": round(da_ms, 4),
        "gemm_weight_gbs": {k: round(w_bytes[k] / (dec_kernel_ms[k] / 1e3) / 1e9, 1) for k in w_bytes
                            if k in dec_kernel_ms},
    }
    log("[bench] decode kernels: " + ", ".join(f"{k} {v * 1e3:.1f} us" for k, v in dec_kernel_ms.items()))

    # Solo prefill on its 128 CUs.
    p0, p1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    p0.record(s_sh)
    binding.hs_shared_stage_forward(ctx, shape, wdev, x, y, batch.seq_offsets, None, None, 128, None, ws)
    p1.record(s_sh)
    torch.cuda.synchronize()
    prefill_solo = p0.elapsed_time(p1)

    # Co-run: both streams start after a common point.
    def corun(graph):
        torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        start.record(s_sh)
        s_dn.wait_event(start)
        binding.hs_shared_stage_forward(ctx, shape, wdev, x, y, batch.seq_offsets, None, None, 128, None, ws)
        p_end = torch.cuda.Event(enable_timing=True)
        p_end.record(s_sh)
        dec_ev = []
        while True:
            dec_ev += decode(1, graph=graph)
            if p_end.query():
                break
            if len(dec_ev) > 4:
                dec_ev[-4].synchronize()
            if len(dec_ev) > 2000:
                break
        torch.cuda.synchronize()
        window = start.elapsed_time(p_end)
        done = [start.elapsed_time(e) for e in dec_ev]
        n_in = sum(1 for t in done if t <= window)
        t_last = max([t for t in done if t <= window], default=0.0)
        return window, (t_last / n_in if n_in else float("nan")), n_in

    window, dec_ms, n_in = corun(False)
    window_g, dec_graph_ms, n_in_g = corun(True)
    tgraph.close()
    T = batch.n_tokens
    res = {
        "shared_cus": 128, "down_cus": 128,
        "prefill_ms": round(window, 3), "prefill_tok_s": round(T / (window / 1e3)),
        "prefill_solo_ms": round(prefill_solo, 3),
        "prefill_mfma_frac_cu_scaled": round(flops_step / (window / 1e3) / (PEAK_BF16 * 128 / N_CUS), 4),
        "decode_steps_in_window": n_in,
        "decode_ms_per_step": round(dec_ms, 4),
        "decode_tok_s": round(32 / (dec_ms / 1e3)) if n_in else None,
        "decode_hbm_frac_cu_scaled": round(step_bytes / (dec_ms / 1e3) / (PEAK_HBM * 128 / N_CUS), 4) if n_in else None,
        "decode_path": "eager decode steps (decode_graph_*: the captured step replayed, hs_decode_graph_launch)",
        "decode_graph_ms_per_step": round(dec_graph_ms, 4), "prefill_ms_with_graph_decode": round(window_g, 3),
        "decode_graph_solo_ms_per_step": round(solo_graph_ms, 4),
        "decode_host_ms_per_step": {"graph": round(host_graph_ms, 4), "eager": round(host_eager_ms, 4)},
        "decode_solo_ms_per_step": round(solo_ms, 4),
        "decode_solo_tok_s": round(32 / (solo_ms / 1e3)),
        "decode_solo_hbm_frac_cu_scaled": round(step_bytes / (solo_ms / 1e3) / (PEAK_HBM * 128 / N_CUS), 4),
        "decode_bytes_per_step": int(step_bytes),
        "decode_kernel_ms": {k: round(v, 4) for k, v in dec_kernel_ms.items()},
        "decode_roofline": decode_roofline,
        "talker": "16 layers, hidden 1024, 16/16 heads, dh 64, ffn 4096, batch 32, kv_len U[128,1024] (sum 17437)",
    }
    log(f"[bench] co-run: prefill {window:.2f} ms (solo {prefill_solo:.2f}), decode {dec_ms:.3f} ms/step "
        f"(solo {solo_ms:.3f}), {n_in} steps in window; captured decode step: {dec_graph_ms:.3f} ms/step "
        f"(solo {solo_graph_ms:.3f}); host time per step: graph {host_graph_ms:.3f} ms, eager {host_eager_ms:.3f} ms")

    # Talker step time against its CU count (the complement of each ladder level).
    sweep = {}
    for c in DOWN_SWEEP:
        sc = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, N_CUS - c, binding.HS_ROLE_DOWN))
        decode(3, c, None, sc)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e0.record(sc)
        ev = decode(10, c, None, sc)
        torch.cuda.synchronize()
        sweep[c] = round(e0.elapsed_time(ev[-1]) / 10, 4)
    res["decode_ms_vs_cus"] = sweep
    log("[bench] talker step vs CUs: " + ", ".join(f"{c}: {v:.3f} ms" for c, v in sweep.items()))

    # No spatial control: both stages on the whole chip (no CU masks), time-sharing it.
    full = torch.cuda.Stream()
    s_full = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, 256, binding.HS_ROLE_SHARED))
    decode(3, 256, full.cuda_stream, full)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e0.record(full)
    ev = decode(20, 256, full.cuda_stream, full)
    torch.cuda.synchronize()
    full_solo = e0.elapsed_time(ev[-1]) / 20
    p0, p1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    p0.record(s_full)
    binding.hs_shared_stage_forward(ctx, shape, wdev, x, y, batch.seq_offsets, None, None, 256, None, ws)
    p1.record(s_full)
    torch.cuda.synchronize()
    prefill_full_solo = p0.elapsed_time(p1)
    w_un, d_un, n_un = corun_window(s_full, 256, 256, full.cuda_stream, full)
    res["unmasked"] = {"prefill_ms": round(w_un, 3), "prefill_solo_ms": round(prefill_full_solo, 3),
                       "decode_ms_per_step": round(d_un, 4) if n_un else None,
                       "decode_solo_ms_per_step": round(full_solo, 4),
                       "decode_steps_in_window": n_un}
    log(f"[bench] unmasked co-run: prefill {w_un:.2f} ms (solo {prefill_full_solo:.2f}), decode {d_un:.3f} ms/step "
        f"(solo {full_solo:.3f}), {n_un} steps in window")

    # Pressure calibration: talker-only loops held for ~1.3 s (past one refresh of the
    # memory-controller activity) at 64 / 128 / 256 CUs, with the AMD SMI reading polled
    # meanwhile, against the loop's event-timed traffic share of the 8 TB/s peak.
    calib = {}
    for c in (64, 128, 256):
        if c == N_CUS:
            st, rec_s = full.cuda_stream, full
        else:
            rec_s = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, N_CUS - c, binding.HS_ROLE_DOWN))
            st = None
        decode(2, c, st, rec_s)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e0.record(rec_s)
        t_end, polls, evs = time.perf_counter() + 1.3, [], []
        while time.perf_counter() < t_end:
            evs += decode(8, c, st, rec_s)
            try:
                polls.append(binding.hs_pressure_sample(0))
            except binding.HorizonError:
                pass
            while len(evs) > 16 and not evs[-16].query():
                time.sleep(0.0005)
        torch.cuda.synchronize()
        ms_ = e0.elapsed_time(evs[-1])
        share = len(evs) * step_bytes / (ms_ / 1e3) / PEAK_HBM
        calib[c] = {"steps": len(evs), "ms_per_step": round(ms_ / len(evs), 4), "traffic_share": round(share, 4),
                    "umc_readings": sorted(set(round(v, 3) for v in polls)),
                    "umc_max": round(max(polls), 3) if polls else None}
        log(f"[bench] pressure calibration @{c} CUs: traffic share {share:.3f} of 8 TB/s, AMD SMI memory activity "
            f"{calib[c]['umc_readings']}")
    res["pressure_calibration"] = calib
    return res


def corun_mixed(torch, binding, W, ctx, dev, steps=4):
    """Downstream-heavy mix: one 4096-wide thinker layer over four 2048-row chunks
    behind 0/2048/4096/6144 cached rows plus 64 decode rows behind 4096, throttled
    to 96 CUs, while the 16-layer talker decodes a batch of 128 on the other 160."""
    from paper_2608_01785_amd.device_data import DeviceCache, prepare_f16, to_device, upload_weights
    shape = W.THINKER_MIXED
    seeds = W.SEEDS["thinker_mixed"]
    lengths, ctx_lens = W.thinker_mixed_layout()
    B = len(lengths)
    wth = prepare_f16(ctx, upload_weights(W.make_weights(shape, 1, seeds["weights"]), dev))
    batch = W.random_batch(shape.hidden, lengths, seeds["tokens"], ctx_lens)
    cache = DeviceCache(1, B, 8192, shape.n_kv_heads, shape.head_dim, dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(seeds["cache"])
    for b in range(B):
        cache.fill_random(0, b, int(ctx_lens[b]), gen)
    x = to_device(batch.x, dev)
    y = torch.empty(x.shape, dtype=torch.float32, device=dev)
    ws = torch.empty(binding.hs_workspace_size(shape, batch.n_tokens, B, 8192), dtype=torch.uint8, device=dev)
    lin, att = thinker_flops(shape, lengths, ctx_lens)
    th_flops = lin + att

    ts_shape, ts_layers, bt = W.TALKER, 16, 128
    tseeds = W.SEEDS["talker"]
    kv_lens = W.talker_kv_lens(bt, 4004)
    tl = prepare_f16(ctx, upload_weights(W.make_weights(ts_shape, ts_layers, tseeds["weights"]), dev))
    max_ctx = int(np.ceil((kv_lens.max() + 1) / 64) * 64)
    tcache = DeviceCache(ts_layers, bt, max_ctx, ts_shape.n_kv_heads, ts_shape.head_dim, dev)
    for l in range(ts_layers):
        for b in range(bt):
            tcache.fill_random(l, b, int(kv_lens[b]), gen)
    xt = to_device(W.token_rows(tseeds["tokens"] + 17, bt, ts_shape.hidden), dev)
    yt = torch.empty(xt.shape, dtype=torch.float32, device=dev)
    wst = torch.empty(binding.hs_workspace_size(ts_shape, bt, bt, int(kv_lens.max()) + 1), dtype=torch.uint8,
                      device=dev)
    t_bytes = talker_bytes(ts_shape, ts_layers, kv_lens)
    s_sh = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, 96, binding.HS_ROLE_SHARED))
    s_dn = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, 96, binding.HS_ROLE_DOWN))

    def thinker(k):
        for _ in range(k):
            binding.hs_shared_stage_forward(ctx, shape, wth, x, y, batch.seq_offsets, ctx_lens, cache.as_arg(), 96,
                                            None, ws)

    wsg = torch.empty(binding.hs_workspace_size(ts_shape, bt, bt, max_ctx), dtype=torch.uint8, device=dev)
    tgraph = binding.DecodeGraph(ctx, ts_shape, tl, xt, yt, tcache.as_arg(), bt, 160, None, wsg)

    def talker(n, graph=True):
        ev = []
        for _ in range(n):
            if graph:
                tgraph.launch(kv_lens)
            else:
                binding.hs_downstream_decode_step(ctx, ts_shape, tl, xt, yt, tcache.as_arg(), kv_lens, 160, None,
                                                  wst)
            e = torch.cuda.Event(enable_timing=True)
            e.record(s_dn)
            ev.append(e)
        return ev

    # Solo figures on the same masks.
    thinker(1)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(s_sh)
    thinker(steps)
    e1.record(s_sh)
    torch.cuda.synchronize()
    th_solo = e0.elapsed_time(e1) / steps
    talker(2, graph=False)
    torch.cuda.synchronize()
    e0.record(s_dn)
    ev = talker(10, graph=False)
    torch.cuda.synchronize()
    tk_solo_eager = e0.elapsed_time(ev[-1]) / 10
    talker(2)
    torch.cuda.synchronize()
    e0.record(s_dn)
    ev = talker(10)
    torch.cuda.synchronize()
    tk_solo = e0.elapsed_time(ev[-1]) / 10

    # Co-run: talker steps loop on the 160 CUs while the thinker runs `steps` steps on 96;
    # eager talker launches, then the captured step.
    def corun(graph):
        torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        start.record(s_sh)
        s_dn.wait_event(start)
        thinker(steps)
        end = torch.cuda.Event(enable_timing=True)
        end.record(s_sh)
        dec = []
        while True:
            dec += talker(1, graph)
            if end.query() or len(dec) > 500:
                break
            if len(dec) > 3:
                dec[-3].synchronize()
        torch.cuda.synchronize()
        window = start.elapsed_time(end)
        done = [start.elapsed_time(e) for e in dec]
        n_in = sum(1 for t in done if t <= window)
        t_last = max([t for t in done if t <= window], default=0.0)
        return window, (t_last / n_in if n_in else float("nan")), n_in

    window, tk_ms, n_in = corun(False)
    window_g, tk_ms_g, n_in_g = corun(True)
    th_ms = window / steps
    res = {
        "workload": "thinker layer hidden 4096, 32/8 heads, ffn 14336: 4 x 2048-row chunks behind 0/2048/4096/6144 "
                    "cached rows + 64 decode rows behind 4096, 96 CUs; talker 16 layers, batch 128, "
                    f"kv_len U[128,1024] (sum {int(kv_lens.sum())}), 160 CUs",
        "thinker_ms": round(th_ms, 3), "thinker_solo_ms": round(th_solo, 3),
        "thinker_tflops": round(th_flops / (th_ms / 1e3) / 1e12, 1),
        "thinker_mfma_frac_cu_scaled": round(th_flops / (th_ms / 1e3) / (PEAK_BF16 * 96 / N_CUS), 4),
        "thinker_solo_mfma_frac_cu_scaled": round(th_flops / (th_solo / 1e3) / (PEAK_BF16 * 96 / N_CUS), 4),
        "talker_ms_per_step": round(tk_ms, 4), "talker_solo_ms_per_step": round(tk_solo_eager, 4),
        "talker_graph_solo_ms_per_step": round(tk_solo, 4),
        "talker_tok_s": round(bt / (tk_ms / 1e3)) if n_in else None,
        "talker_hbm_frac_cu_scaled": round(t_bytes / (tk_ms / 1e3) / (PEAK_HBM * 160 / N_CUS), 4) if n_in else None,
        "talker_solo_hbm_frac_cu_scaled": round(t_bytes / (tk_solo_eager / 1e3) / (PEAK_HBM * 160 / N_CUS), 4),
        "talker_steps_in_window": n_in, "thinker_flops": th_flops, "talker_bytes_per_step": int(t_bytes),
        "talker_path": "eager decode steps (talker_graph_*: the captured step replayed)",
        "talker_graph_ms_per_step": round(tk_ms_g, 4) if n_in_g else None,
        "talker_graph_steps_in_window": n_in_g, "thinker_ms_beside_graph": round(window_g / steps, 3),
    }
    log(f"[bench] mixed co-run: thinker {th_ms:.3f} ms/step (solo {th_solo:.3f}), talker {tk_ms:.3f} ms/step "
        f"(solo {tk_solo_eager:.3f}), {n_in} talker steps in window; captured talker step: {tk_ms_g:.3f} ms/step "
        f"(solo {tk_solo:.3f}), {n_in_g} steps beside a {window_g / steps:.3f} ms thinker step")
    tgraph.close()
    del wth, tl, cache, tcache
    return res


def dit_corun(torch, binding, W, ctx, th_shape, wdev, x, y, batch, ws, dev, flops_th, steps=6):
    """Second downstream workload: a DiT denoising step (16 adaLN-Zero blocks, hidden 1024,
    16 heads, MLP 4096) over 4 latents of 1024 tokens, solo on 128 CUs and co-running with the
    thinker prefill on the other 128."""
    from paper_2608_01785_amd.device_data import prepare_dit_f16, to_device, upload_weights
    shape, n_blocks = W.DIT, 16
    seeds = W.SEEDS["dit"]
    lengths = [1024] * 4
    off = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    T = int(off[-1])
    wd = prepare_dit_f16(ctx, upload_weights(W.make_dit_weights(shape, n_blocks, seeds["weights"]), dev))
    xd = to_device(W.token_rows(seeds["tokens"], T, shape.hidden), dev)
    yd = torch.empty((T, shape.hidden), dtype=torch.float32, device=dev)
    cond = torch.from_numpy(W.dit_cond(seeds["cond"], len(lengths), shape.hidden)).to(dev)
    wsd = torch.empty(binding.hs_dit_workspace_size(shape, T, len(lengths)), dtype=torch.uint8, device=dev)
    d, m = shape.hidden, shape.mlp
    flops = n_blocks * (2.0 * T * (4 * d * d + 2 * d * m) + 4.0 * d * float(np.sum(np.square(lengths))))
    s_sh = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, 128, binding.HS_ROLE_SHARED))
    s_dn = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, 128, binding.HS_ROLE_DOWN))

    def dit(n):
        ev = []
        for _ in range(n):
            binding.hs_dit_forward(ctx, shape, wd, xd, yd, cond, off, 128, None, wsd)
            e = torch.cuda.Event(enable_timing=True)
            e.record(s_dn)
            ev.append(e)
        return ev

    dit(1)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e0.record(s_dn)
    ev = dit(steps)
    torch.cuda.synchronize()
    solo = e0.elapsed_time(ev[-1]) / steps
    binding.hs_timing_enable(ctx, True)
    dit(1)
    kms = {k: binding.hs_timing_read(ctx, k) for k in binding.KERNEL_KINDS}
    clk = {k: binding.hs_timing_read_clock(ctx, k)[0] for k in binding.KERNEL_KINDS}
    binding.hs_timing_enable(ctx, False)
    kms = {k: round(v[0] / v[1], 4) for k, v in kms.items() if v[1]}
    # Co-run: DiT steps loop on the 128 DOWN CUs while the thinker stack prefills on the other 128.
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    start.record(s_sh)
    s_dn.wait_event(start)
    binding.hs_shared_stage_forward(ctx, th_shape, wdev, x, y, batch.seq_offsets, None, None, 128, None, ws)
    p_end = torch.cuda.Event(enable_timing=True)
    p_end.record(s_sh)
    dec = []
    while True:
        dec += dit(1)
        if p_end.query() or len(dec) > 200:
            break
        if len(dec) > 2:
            dec[-2].synchronize()
    torch.cuda.synchronize()
    window = start.elapsed_time(p_end)
    done = [start.elapsed_time(e) for e in dec]
    n_in = sum(1 for t in done if t <= window)
    t_last = max([t for t in done if t <= window], default=0.0)
    co = t_last / n_in if n_in else float("nan")
    peak128 = PEAK_BF16 * 128 / N_CUS
    res = {"workload": f"DiT {n_blocks} blocks, hidden 1024, 16 heads, MLP 4096, 4 latents x 1024 tokens, "
                       "on 128 CUs beside the thinker prefill on 128",
           "flops_per_step": flops, "solo_ms_per_step": round(solo, 3),
           "solo_mfma_frac_cu_scaled": round(flops / (solo / 1e3) / peak128, 4),
           "corun_ms_per_step": round(co, 3) if n_in else None, "steps_in_window": n_in,
           "corun_mfma_frac_cu_scaled": round(flops / (co / 1e3) / peak128, 4) if n_in else None,
           "prefill_ms": round(window, 3), "prefill_tok_s": round(batch.n_tokens / (window / 1e3)),
           "prefill_mfma_frac_cu_scaled": round(flops_th / (window / 1e3) / peak128, 4),
           "kernel_ms": kms, "kernel_clock_mhz": {k: round(v, 1) for k, v in clk.items() if v > 0}}
    log(f"[bench] DiT step: solo {solo:.3f} ms ({res['solo_mfma_frac_cu_scaled']:.3f} of CU-scaled MFMA) on 128 "
        f"CUs; co-run {co:.3f} ms/step, {n_in} steps beside a {window:.2f} ms thinker prefill")
    del wd
    return res


TPOT_CAPS = [16, 32, 48, 64, 96, 128, 192, 256]
LOOP_SEEDS = (11, 12, 13, 14, 15, 16)
DOWN_SWEEP = (64, 128, 160, 192, 224, 240)   # talker CU counts of the co-run sweep


def thinker_decode_sweep(torch, binding, W, ctx, shape, wdev, n_layers, dev, batch=16):
    """Decode step of the thinker stack (one new row for each of `batch` sequences
    behind 1024-2048 cached rows) at each CU cap: the shared stage's TPOT curve."""
    from paper_2608_01785_amd.device_data import DeviceCache, to_device
    caps = TPOT_CAPS
    try:
        rng = np.random.default_rng(5001)
        ctx_lens = rng.integers(1024, 2048, size=batch, endpoint=True).astype(np.int32)
        max_ctx = int(np.ceil((ctx_lens.max() + 1) / 64) * 64)
        cache = DeviceCache(n_layers, batch, max_ctx, shape.n_kv_heads, shape.head_dim, dev)
        gen = torch.Generator(device=dev)
        gen.manual_seed(5002)
        for l in range(n_layers):
            for b in range(batch):
                cache.fill_random(l, b, int(ctx_lens[b]), gen)
        x = to_device(W.token_rows(5003, batch, shape.hidden), dev)
        y = torch.empty(x.shape, dtype=torch.float32, device=dev)
        offsets = list(range(batch + 1))
        ws = torch.empty(binding.hs_workspace_size(shape, batch, batch, int(ctx_lens.max()) + 1), dtype=torch.uint8,
                         device=dev)
        step_bytes = talker_bytes(shape, n_layers, ctx_lens)
        out = {"workload": f"thinker {n_layers}-layer stack, {batch} single-row sequences behind "
                           f"{int(ctx_lens.min())}-{int(ctx_lens.max())} cached rows (sum {int(ctx_lens.sum())})",
               "bytes_per_step": int(step_bytes), "cus": [], "tpot_ms": [], "hbm_frac_cu_scaled": [],
               "host_ms_per_call": []}
        for c in caps:
            s = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, c, binding.HS_ROLE_SHARED))

            def step(k):
                for _ in range(k):
                    binding.hs_shared_stage_forward(ctx, shape, wdev, x, y, offsets, ctx_lens, cache.as_arg(), c, None,
                                                    ws)
            step(3)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            h0 = time.perf_counter()
            step(20)
            host_ms = (time.perf_counter() - h0) * 1e3 / 20
            e1.record(s)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / 20
            out["host_ms_per_call"].append(round(host_ms, 4))
            out["cus"].append(c)
            out["tpot_ms"].append(round(ms, 4))
            out["hbm_frac_cu_scaled"].append(round(step_bytes / (ms / 1e3) / (PEAK_HBM * c / N_CUS), 4))
        best = min(out["tpot_ms"])
        out["saturation_cus"] = next(c for c, t in zip(out["cus"], out["tpot_ms"]) if t <= 1.05 * best)
        log("[bench] thinker decode TPOT vs CUs: " + ", ".join(
            f"{c}: {t:.3f} ms (host {h:.3f})" for c, t, h in zip(out["cus"], out["tpot_ms"], out["host_ms_per_call"]))
            + f"; within 5 % of the best from {out['saturation_cus']} CUs")
        return out
    finally:
        torch.cuda.synchronize()


def policy_model(W, shape, batch, per_budget, corun):
    """Algorithm 1's loop in the discrete-event model, with the times measured above (model output)."""
    from paper_2608_01785_amd import sim
    T = batch.n_tokens
    ts = W.TALKER
    weights = 16 * ts.params_per_layer * 2
    un = corun["unmasked"]
    t = sim.Timing(
        prefill_ms_per_token={int(b): v["ms_per_step"] / T for b, v in per_budget.items()},
        decode_ms_per_step={int(c): v for c, v in corun["decode_ms_vs_cus"].items()},
        decode_batch=32, weight_share=weights / corun["decode_bytes_per_step"],
        masked_prefill_factor=corun["prefill_ms"] / corun["prefill_solo_ms"],
        masked_decode_factor=corun["decode_ms_per_step"] / corun["decode_solo_ms_per_step"],
        unmasked_prefill_factor=un["prefill_ms"] / un["prefill_solo_ms"],
        # No step finished beside an unmasked prefill: the downstream stalls (a factor of 1e9).
        unmasked_decode_factor=(un["decode_ms_per_step"] / un["decode_solo_ms_per_step"]
                                if un["decode_steps_in_window"] else 1e9),
        decode_full_ms=un["decode_solo_ms_per_step"],
        hbm_share=corun["decode_hbm_frac_cu_scaled"] * corun["down_cus"] / N_CUS)
    per_req_ms = 1152 * t.prefill_ms_per_token[N_CUS]  # mean prompt of U[256, 2048]
    capacity = 1000.0 / per_req_ms
    out = {"note": "model output on measured kernel times, not a measurement", "timing": dataclasses.asdict(t),
           "capacity_req_s": round(capacity, 1), "loads": []}
    # Calibration (§4.2): the shared stage's decode TPOT keeps improving up to the whole chip, so
    # S_cap is the top ladder level below S_aggr; B_sat is the downstream's measured HBM share,
    # so its usual pressure maps to S_cap and a lighter downstream batch cedes CUs to it.
    ccfg = dict(total_cus=N_CUS, aggressive_cus=N_CUS, ladder=[128, 160, 192, 224], ewma_weight=0.4,
                saturation=t.hbm_share, hysteresis_steps=1)
    out["controller_cfg"] = ccfg
    out["temporal_cfg"] = dict(n_min=2, n_max=8, m=2, u_guard=1.0, long_cap=4)
    for load in (0.5, 0.8, 0.95):
        w = sim.Workload(n_requests=400, rate_per_s=load * capacity)
        res = [sim.simulate(p, t, w, out["temporal_cfg"], ccfg) for p in ("baseline", "temporal", "spatial", "joint")]
        out["loads"].append({"load": load, "rate_req_s": round(w.rate_per_s, 1), "policies": res})
        log(f"[bench] policy model at {load:.0%} of shared-stage capacity: " + "; ".join(
            f"{r['policy']} short {r['short']['slo_attainment']:.3f} long {r['long']['slo_attainment']:.3f}"
            for r in res))
    return out


def serving_loop(torch, binding, W, ctx, wdev, dev, policy, n_req=48, first_chunk=20, seed=11, load=0.6,
                 saturation=0.25, short_budget=0):
    """Algorithm 1 on the GPU (measured, unlike the model; the loop is
    paper_2608_01785_amd.serving.Algorithm1): a seeded Poisson stream of requests at `load`
    times the shared stage's capacity, half long-path, prompts of 256-1024 rows through the
    4-layer thinker stack, long-path requests decoding talker steps (16 layers, 128-512 cached
    rows, paged cache) on the complementary stream.  Baseline: every request visible, both
    stages unmasked on the whole chip.  The pressure signal is the talker's event-timed
    traffic share; B_sat = `saturation`."""
    from paper_2608_01785_amd import serving
    from paper_2608_01785_amd.device_data import prepare_f16, to_device, upload_weights
    th, ts = W.THINKER, W.TALKER
    per_tok, talker_ms = 0.00185, 0.9       # solo ms per prompt token at 256 CUs, talker step at 128
    cfg = serving.LoopConfig(policy=policy, token_budget=4096, short_budget=short_budget, first_chunk=first_chunk,
                             saturation=saturation)
    reqs = serving.make_requests(n_req, seed, load, per_tok, talker_ms, first_chunk)
    tl = prepare_f16(ctx, upload_weights(W.make_weights(ts, 16, W.SEEDS["talker"]["weights"]), dev))
    x_pool = to_device(W.token_rows(seed, 4096, th.hidden), dev)
    xt = to_device(W.token_rows(seed + 1, n_req, ts.hidden), dev)
    loop = serving.Algorithm1(ctx, (th, wdev, 4), (ts, tl, 16), reqs, x_pool, cfg, max_ctx=576, x_talker=xt,
                              device=dev)
    try:
        out = loop.run()
    finally:
        loop.close()
    out["load"] = load
    out["rate_req_s"] = round(1e3 * n_req / reqs[-1].arrival, 1)
    out["saturation"] = saturation
    out["short_budget"] = short_budget or cfg.token_budget
    log(f"[bench] serving loop ({policy}, short budget {out['short_budget']}, B_sat {saturation:.3f}): short p50/p95 "
        f"{out['short']['p50_ms']}/{out['short']['p95_ms']} ms (SLO {out['short']['slo_attainment']}), long p50/p95 "
        f"{out['long']['p50_ms']}/{out['long']['p95_ms']} ms (SLO {out['long']['slo_attainment']}), makespan "
        f"{out['makespan_ms']} ms, mean shared CUs {out['mean_shared_cus']}")
    return out


def controller_measure(torch, binding, ctx, ladder, dev):
    """Costs of the spatial controller's control path on the GPU.

    * switch_us: extra GPU-side delay when consecutive dependent launches move
      from the SHARED stream of one ladder level to that of another (an event
      on the old stream, a wait on the new one), against staying on one stream.
      Each launch is one probe work-group that spins ~20 us and stamps its
      start on the constant-rate clock, so the host stays ahead of the GPU.
    * switch_synced_us: the same when the host waits for each launch before
      issuing the next (a serving loop reads every step's output), so the new
      level's stream is idle when it receives work.
    * decide_us: host time of one controller step plus the stream lookup.
    * pressure_sample_us / pressure: one AMD SMI memory-activity reading.
    """
    n = 64
    s_a = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, 128, binding.HS_ROLE_SHARED))
    s_b = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, 256, binding.HS_ROLE_SHARED))
    out = torch.zeros((n, 4), dtype=torch.int32, device=dev)

    def chain(alternate, synced=False):
        torch.cuda.synchronize()
        prev = s_a
        for i in range(n):
            cur = (s_a if i % 2 == 0 else s_b) if alternate else s_a
            if cur is not prev and not synced:
                ev = torch.cuda.Event()
                ev.record(prev)
                cur.wait_event(ev)
            binding.hs_probe_hw_ids(ctx, cur.cuda_stream, 1, out[i])
            if synced:
                cur.synchronize()
            prev = cur
        torch.cuda.synchronize()
        t = out[:, 3].cpu().numpy().astype(np.int64)
        d = np.diff(t) % (1 << 32)
        return float(np.median(d[1:])) / 100.0  # 100 MHz clock -> us

    chain(False)
    same = chain(False)
    alt = chain(True)
    same_synced = chain(False, synced=True)
    alt_synced = chain(True, synced=True)

    ctrl = binding.Controller(N_CUS, N_CUS, ladder, 0.4, 0.8, 1)
    k = 20000
    t0 = time.perf_counter()
    for i in range(k):
        sp = binding.hs_controller_step(ctrl, i % 3 != 0, (i % 10) / 10.0)
        binding.hs_context_stream(ctx, sp.shared_cus, binding.HS_ROLE_SHARED)
    decide_us = (time.perf_counter() - t0) / k * 1e6
    ctrl.close()

    pressure, sample_us = None, None
    try:
        binding.hs_pressure_sample(0)
        t0 = time.perf_counter()
        for _ in range(200):
            pressure = binding.hs_pressure_sample(0)
        sample_us = (time.perf_counter() - t0) / 200 * 1e6
    except binding.HorizonError as e:
        log(f"[bench] AMD SMI pressure sample unavailable: {e}")
    res = {"same_stream_gap_us": round(same, 2), "switch_gap_us": round(alt, 2),
           "switch_us": round(alt - same, 2), "switch_synced_us": round(alt_synced - same_synced, 2),
           "synced_gap_us": round(same_synced, 2), "decide_us": round(decide_us, 2),
           "pressure_sample_us": None if sample_us is None else round(sample_us, 1), "pressure": pressure,
           "note": "switch = event on the old level's stream + wait on the new one; decide = controller step "
                   "+ stream lookup through the Python binding"}
    log(f"[bench] controller: switch {alt - same:.2f} us (gap {alt:.2f} vs {same:.2f} us), host-synced switch "
        f"{alt_synced - same_synced:.2f} us (gap {alt_synced:.2f} vs {same_synced:.2f}), decide {decide_us:.2f} us, "
        f"pressure sample {sample_us} us = {pressure}")
    return res


def cpu_baseline(W, layers, batch, shape, rows_per_seq, target_s=15.0):
    """The float64 reference on the host: first rows of every request through all layers.

    By causality the first r rows of a request depend only on themselves, so the
    sample is a faithful slice of the same workload.  With rows_per_seq = 0 the
    sample size is chosen from a short calibration run to take about target_s.
    """
    from oracle import layer as ref
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [os.cpu_count()])
    except Exception:
        cores = os.cpu_count()
    w64 = [{k: W.bf16_to_f32(v).astype(np.float64) for k, v in lw.items()} for lw in layers]

    def sample(r, n_layers):
        xs = np.concatenate([batch.x[o:o + r] for o in batch.seq_offsets[:-1]])
        off = np.arange(batch.n_seqs + 1) * r
        x64 = W.bf16_to_f32(xs).astype(np.float64)
        t0 = time.time()
        ref.stack_forward(x64, w64[:n_layers], shape, off)
        return time.time() - t0, int(off[-1])

    r = rows_per_seq
    if r <= 0:
        t_cal, rows_cal = sample(32, 1)
        per_row_layer = t_cal / rows_cal
        r = int(target_s / (per_row_layer * batch.n_seqs * len(layers)))
        r = max(32, min(r, int(batch.lengths.min())))
    dt, rows = sample(r, len(layers))
    log(f"[bench] CPU reference: {rows} rows x {len(layers)} layers in {dt:.1f}s ({cores} threads)")
    out = {"value": round(rows / dt, 2), "unit": "tok/s", "cores": int(cores), "kind": "oracle",
           "sample": f"first {r} rows of each of the {batch.n_seqs} requests through all {len(layers)} layers "
                     f"({rows} rows), float64 NumPy", "seconds": round(dt, 2)}
    out.update(host_info())
    out["talker_step"] = cpu_talker_step(W, ref)
    return out


def host_info():
    """CPU model and the BLAS library NumPy runs on (as threadpoolctl reports it)."""
    info = {"cpu_model": None, "blas": None}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    info["cpu_model"] = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        libs = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if libs:
            i = libs[0]
            info["blas"] = f"{i.get('internal_api')} {i.get('version')} ({i.get('threading_layer')}, " \
                           f"{i.get('num_threads')} threads)"
    except Exception:
        pass
    return info


def cpu_talker_step(W, ref, n_layers=4):
    """The float64 reference of one talker decode step (batch 32, kv_len U[128, 1024]): the first
    n_layers of the 16 (the seeded weights and cache of those layers), scaled to the whole step."""
    ts, seeds = W.TALKER, W.SEEDS["talker"]
    db = W.talker_batch(ts, n_layers, 32, seeds)
    layers = W.make_weights(ts, n_layers, seeds["weights"])
    w64 = [{k: W.bf16_to_f32(v).astype(np.float64) for k, v in lw.items()} for lw in layers]
    ck = [[W.f16_to_f32(a).astype(np.float64) for a in per] for per in db.cache.k]
    cv = [[W.f16_to_f32(a).astype(np.float64) for a in per] for per in db.cache.v]
    x = W.bf16_to_f32(db.x).astype(np.float64)
    t0 = time.time()
    ref.decode_step(x, w64, ts, db.kv_lens, ck, cv)
    dt = (time.time() - t0) * 16 / n_layers
    log(f"[bench] CPU reference talker step: {dt * 1e3:.0f} ms per 16-layer step ({n_layers} layers timed)")
    return {"ms_per_step": round(dt * 1e3, 1), "tok_s": round(32 / dt, 2),
            "sample": f"layers 0-{n_layers - 1} of the 16-layer batch-32 step, scaled by 16/{n_layers}"}


if __name__ == "__main__":
    main()
