"""Benchmark of the selective affix-KV recompute hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config NAME] [--no-cpu]

The default workload is the serving-scale LLaDA-8B-shaped stack (32 layers,
32 requests sharing an 8192-token affix, 256 unique and 256 masked tokens
each, anchor ratio 0.2), the largest configuration on one GPU.

A step is one pass of the whole hot path over one batch: the one-shot probe
(gather the non-affix rows, every layer with masked-to-affix scoring),
top-K anchor selection, the device-side write/read slot maps, the row
gather and the selective refresh of anchors plus request rows through every
layer.  Inputs, weights and the shared affix cache are resident in HBM
before the timed region.  `value` is recomputed tokens per second: the
refresh's recomputed rows (B * R) per step divided by the step time.

The JSON line also carries the full-recompute baseline timed the same way,
the per-kernel breakdown, the dominant kernel's roofline (algorithmic
FLOPs per launch / its mean launch duration from HIP events recorded around
each of its launches during the timed region) and the fp64 CPU oracle timed
on this host's cores on a bounded sample.  Workloads with a decode schedule
add the end-to-end serving schedule (one probe, then per 32-token block a
refresh, LM head and greedy commit) against the same schedule with full
recomputation, the peak KV memory of each, and the time of one decode step.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"bf16": (2500.0, "mfma"), "f32": (157.3, "alu")}  # TFLOP/s, dense
HBM_GBS = 8000.0  # MI355X HBM3E peak, GB/s
KERNELS = ["gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down", "attention", "score_lse", "score_colsum",
           "score_reduce", "rmsnorm", "residual", "topk", "gather", "maps"]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="llada-serve-b32")
    ap.add_argument("--ratio", type=float, default=None)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--only-step", action="store_true",
                    help="run only the warmup and timed steps (for profilers): no breakdown, phases or CPU leg")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="instead of the workload, run the row-gather kernel as a plain copy of MIB MiB "
                         "--steps times (the known-size reference for the HBM byte counters)")
    ap.add_argument("--block-size", type=int, default=256,
                    help="KV block size of the serving schedule's paged slot plan (0: flat plan)")
    ap.add_argument("--tau", type=float, default=-1.0,
                    help="run the threshold-decoding schedule with this confidence threshold (negative: skip it)")
    ap.add_argument("--no-schedule", action="store_true", help="skip the serving-schedule extras")
    ap.add_argument("--phase-budget-ms", type=float, default=6000.0,
                    help="time budget of each extra phase measurement (repetitions are cut to fit)")
    return ap.parse_args()


def flops_model(w, K):
    """Algorithmic FLOPs of one step, by kernel (see the design notes):
    linear 2 * params / layer / row, attention 4 * S * H * d_h / row / layer,
    probe scoring 2 * G * L * H * d_h / request / layer per sweep over the
    affix keys: the column sums, and the log-sum-exp where the layer's
    attention does not hand it over (timed as score_colsum on the bf16 path,
    where both sweeps are one kernel)."""
    d = w.dims
    lay = w.layout
    B, S, L, G, N = w.batch, lay.seq_len, lay.affix_len, lay.mask_len, d.n_layers
    P = lay.n_nonaffix
    R = K + P
    hq, hkv = d.n_heads * d.head_dim, d.n_kv_heads * d.head_dim
    per_row = {
        "gemm_qkv": 2 * d.d_model * (hq + 2 * hkv),
        "gemm_o": 2 * hq * d.d_model,
        "gemm_gate_up": 2 * d.d_model * 2 * d.d_ff,
        "gemm_down": 2 * d.d_ff * d.d_model,
        "attention": 4 * S * hq,
    }
    rows = {"probe": B * P, "refresh": B * R, "full": B * S}
    out = {}
    for phase, m in rows.items():
        out[phase] = {k: v * m * N for k, v in per_row.items()}
    # the probe's last layer computes only what its score reads: the masked
    # rows' queries (acache_layer_score under the affix-only normalisation)
    out["probe"] = {k: v * B * P * (N - 1) for k, v in per_row.items()}
    out["probe"]["gemm_qkv"] += 2 * d.d_model * hq * B * G
    sweep = 2 * G * L * hq * B
    if d.dtype == "bf16":
        # one kernel: the column-sum sweep, and the log-sum-exp sweep except
        # where the attention takes it (the probe reads the affix keys first;
        # whole 64-key tiles: every probe layer but the last, which runs no
        # attention)
        lse_sweeps = 1 if L % 64 == 0 else N
        out["probe"]["score_colsum"] = sweep * (N + lse_sweeps)
    else:
        out["probe"]["score_lse"] = sweep * N
        out["probe"]["score_colsum"] = sweep * N
    return out, rows


def bytes_model(w, K, A, dims):
    """Algorithmic HBM bytes of one step for the data-movement kernels: each
    operand read once and each result written once (split-K partials are an
    implementation choice and not counted).  Which norm and residual kernels
    run depends on the K splits the layer call picks for its row count
    (acache_layer_schedule): with one split the second RMSNorm is a kernel of
    its own, with more the reduction kernel adds the residual (and normalises)."""
    d = w.dims
    lay = w.layout
    B, S, L, N = w.batch, lay.seq_len, lay.affix_len, d.n_layers
    es = 2 if d.dtype == "bf16" else 4
    P, R, G = B * lay.n_nonaffix, B * (K + lay.n_nonaffix), B * lay.mask_len
    hq = d.n_heads * d.head_dim
    row = d.d_model * es
    norm = res = 0
    for m, layers in ((P, N - 1), (R, N)):
        o_sp, dn_sp = A.acache_layer_schedule(dims, m)
        norm += layers * 2 * m * row * (1 if o_sp > 1 else 2)
        res += layers * ((3 * m * row if o_sp > 1 else 0) + (2 * m * row if dn_sp > 1 else 0))
    # the probe's last layer: its masked rows gathered and normalised, and
    # their queries written by the split-K reduction (timed as "residual")
    norm += 2 * G * row
    res += G * hq * es
    rows = P + R
    return {
        "gather": 2 * rows * row,
        "rmsnorm": norm,
        "residual": res,
        "topk": B * L * 4 + B * K * 4,
        "maps": 4 * (3 * rows + 2 * B * S),
        "score_reduce": 4 * (d.n_heads + 1) * B * L * N,
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (--gpus {args.gpus} requested). "
              "Requests are independent, so N GPUs would each run this workload on their own share.",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import workloads as W
    from paper_2608_26140_amd import acache as A
    from paper_2608_26140_amd import driver as D
    from paper_2608_26140_amd import workload as WL

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_calibration:
        copy_calibration(args, A)
        return
    w = W.get_config(args.config)
    if args.ratio is not None:
        w = w.with_ratio(args.ratio)
    d, lay = w.dims, w.layout
    B, S, L = w.batch, lay.seq_len, lay.affix_len
    K = A.acache_anchor_count(w.ratio, L)
    R = K + lay.n_nonaffix
    print(f"[bench] building {w.name}: layers {d.n_layers} batch {B} S {S} L {L} K {K} R {R}", file=sys.stderr,
          flush=True)
    t0 = time.time()
    setup = WL.build(w, keep_host=not args.no_cpu,
                     block_size=(args.block_size or None) if w.decode_block else None)
    batch = setup.batch
    torch.cuda.synchronize()
    print(f"[bench] setup {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    every = torch.arange(L, dtype=torch.int32, device="cuda").repeat(B, 1).contiguous()

    def step():
        anchors, _ = batch.select_anchors(K)
        batch.refresh(anchors, K)

    def timed(fn, n):
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    def timed_budget(fn):
        """Mean time of fn over as many repetitions (1 .. --steps) as fit the
        phase budget, after one untimed call."""
        first = timed(fn, 1)
        n = int(max(1, min(args.steps, args.phase_budget_ms // max(first, 1e-3))))
        return timed(fn, n)

    for i in range(args.warmup):
        step()
        if i == 0:
            torch.cuda.synchronize()
            print("[bench] first step done", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    print("[bench] warmed up", file=sys.stderr, flush=True)

    # per-kernel breakdown: one armed step per kernel, outside the timed region
    launches_per_step = 4 * d.n_layers + 4
    breakdown = {}
    armed_ms = []
    # the bf16 path scores in one kernel (timed as score_colsum); score_lse is the fp32 path's first sweep
    timed_kernels = [k for k in KERNELS if not (k == "score_lse" and d.dtype == "bf16")]
    for kname in ([] if args.only_step else timed_kernels):
        kt = A.KernelTimer(kname, 4 * launches_per_step)
        torch.cuda.synchronize()
        a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with kt:
            a0.record()
            step()
            a1.record()
        torch.cuda.synchronize()
        armed_ms.append(a0.elapsed_time(a1))
        ds = kt.durations()
        kt.close()
        breakdown[kname] = {"launches": len(ds), "us_per_step": 1e3 * sum(ds)}
    if breakdown:
        print("[bench] kernel breakdown done", file=sys.stderr, flush=True)
    dominant = max(breakdown, key=lambda k: breakdown[k]["us_per_step"]) if breakdown else "gemm_gate_up"

    # timed region: K steps, the dominant kernel's launches bracketed by events
    fl, rows = flops_model(w, K)
    kt = A.KernelTimer(dominant, args.steps * launches_per_step + 8)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with kt:
        e0.record()
        for _ in range(args.steps):
            step()
        e1.record()
        torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    durs = kt.durations()
    kt.close()
    print(f"[bench] timed {args.steps} steps: {ms_step:.3f} ms/step", file=sys.stderr, flush=True)
    dom_flops_step = fl["probe"].get(dominant, 0) + fl["refresh"].get(dominant, 0)
    dom_launches_step = len(durs) / args.steps
    dom_ms_step = sum(durs) / args.steps

    # phases, each timed on its own within the phase budget
    anchors_fixed, _ = batch.select_anchors(K)
    shift_dir = [1]

    def shift():
        # reuse of the shared cache one position away and back (re-rotation of its K, all layers)
        batch.shift_affix(shift_dir[0])
        shift_dir[0] = -shift_dir[0]

    phases = None
    if not args.only_step:
        phases = {
            "select_anchors": timed_budget(lambda: batch.select_anchors(K)),
            "select_anchors_full_last_layer": timed_budget(lambda: batch.select_anchors(K, full_probe=True)),
            "selective_refresh": timed_budget(lambda: batch.refresh(anchors_fixed, K)),
            "full_refresh": timed_budget(lambda: batch.refresh(every, L)),
            "selective_refresh_dropna": timed_budget(lambda: batch.refresh(anchors_fixed, K, drop_non_anchor=True)),
            "select_anchors_hkvd": timed_budget(lambda: batch.select_anchors_hkvd(K)),
        }
        first = timed(shift, 2)
        phases["shift_affix"] = timed(shift, 2 * int(max(1, min(args.steps // 2, args.phase_budget_ms // (2 * first)))))
        phases = {k: round(v, 4) for k, v in phases.items()}
        print("[bench] phases done", file=sys.stderr, flush=True)

    # for launch-bound workloads: the step recorded once into a HIP graph and
    # replayed, and the step with cold caches (a 512 MiB write before each
    # step evicts the 256 MB MALL and the L2s)
    graph_replay = cold = None
    if not args.only_step and ms_step < 50:
        graph, _ = D.capture(step)
        torch.cuda.synchronize()
        ms_graph = timed(graph.replay, args.steps)
        del graph
        graph_replay = {"ms_per_step": round(ms_graph, 4), "value": round(B * R / (ms_graph * 1e-3), 1)}
        flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
        n_cold = max(1, min(args.steps, 20))
        tot = 0.0
        for _ in range(n_cold):
            flush.fill_(1)
            c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            c0.record()
            step()
            c1.record()
            torch.cuda.synchronize()
            tot += c0.elapsed_time(c1)
        del flush
        ms_cold = tot / n_cold
        cold = {"ms_per_step": round(ms_cold, 4), "value": round(B * R / (ms_cold * 1e-3), 1), "steps": n_cold,
                "flush_MiB": 512}

    peak, bound = PEAK[d.dtype]
    step_flops = sum(fl["probe"].values()) + sum(fl["refresh"].values())
    by = bytes_model(w, K, A, batch.model.dims)
    kernel_roofline = {}
    for k, v in breakdown.items():
        sec = v["us_per_step"] * 1e-6
        if sec <= 0:
            continue
        f = fl["probe"].get(k, 0) + fl["refresh"].get(k, 0)
        if f:
            a = f / sec / 1e12
            kernel_roofline[k] = {"us": round(v["us_per_step"], 2), "achieved": round(a, 1), "unit": "TFLOP/s",
                                  "frac": round(a / peak, 4)}
        elif k in by:
            a = by[k] / sec / 1e9
            kernel_roofline[k] = {"us": round(v["us_per_step"], 2), "achieved": round(a, 1), "unit": "GB/s",
                                  "frac": round(a / HBM_GBS, 4)}
    achieved = dom_flops_step / (dom_ms_step * 1e-3) / 1e12 if dom_ms_step > 0 else 0.0
    traffic = None
    tfile = os.path.join(ROOT, "profiles", "traffic.json")
    if os.path.exists(tfile):
        try:
            rec = json.load(open(tfile)).get(f"{w.name}:{dominant}")
            from paper_2608_26140_amd.build import source_digest
            if rec and rec.get("source_digest") == source_digest():
                traffic = rec["bytes_per_launch"]
        except Exception:
            traffic = None
    ksum = sum(v["us_per_step"] for v in breakdown.values())
    ms_refresh = phases["selective_refresh"] if phases else None
    ms_full = phases["full_refresh"] if phases else None

    result = {
        "metric": "selective-recompute latency/request + recomputed tokens/s, MFMA util vs full recompute",
        "value": round(B * R / (ms_step * 1e-3), 1),
        "unit": "recomputed tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": d.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "layers": d.n_layers, "batch": B, "seq_len": S, "affix_len": L,
                   "masked": lay.mask_len, "ratio": w.ratio, "anchors": K, "recomputed_rows": R,
                   "probe_rows": lay.n_nonaffix, "d_model": d.d_model, "heads": d.n_heads,
                   "kv_heads": d.n_kv_heads, "d_ff": d.d_ff},
        "latency_ms_per_request": round(ms_step / B, 4),
        "refresh_latency_ms_per_request": None if ms_refresh is None else round(ms_refresh / B, 4),
        "phases_ms": phases,
        "cold_caches": cold,
        "graph_replay": graph_replay,
        "shift_affix_GB_per_s": None if not phases else round(
            2 * L * d.n_kv_heads * d.head_dim * (2 if d.dtype == "bf16" else 4) * d.n_layers
            / (phases["shift_affix"] * 1e-3) / 1e9, 1),
        "refresh_speedup_vs_full": None if ms_refresh is None else round(ms_full / ms_refresh, 3),
        "speedup_target_S_over_R": round(S / R, 3),
        "refresh_recomputed_tokens_per_s": None if ms_refresh is None else round(B * R / (ms_refresh * 1e-3), 1),
        "full_recomputed_tokens_per_s": None if ms_full is None else round(B * S / (ms_full * 1e-3), 1),
        "step_tflops": round(step_flops / (ms_step * 1e-3) / 1e12, 1),
        "step_mfma_util": round(step_flops / (ms_step * 1e-3) / 1e12 / peak, 4),
        "refresh_mfma_util": None if ms_refresh is None else round(
            sum(fl["refresh"].values()) / (ms_refresh * 1e-3) / 1e12 / peak, 4),
        "full_mfma_util": None if ms_full is None else round(
            sum(fl["full"].values()) / (ms_full * 1e-3) / 1e12 / peak, 4),
        "kernel_us_per_step": {k: round(v["us_per_step"], 2) for k, v in breakdown.items()},
        # each kernel's events come from its own armed step; their sum against
        # the mean of those steps shows how much of a step the kernels cover
        "kernel_sum_us": round(ksum, 1) if breakdown else None,
        "armed_step_us": round(1e3 * sum(armed_ms) / len(armed_ms), 1) if armed_ms else None,
        "kernel_roofline": kernel_roofline,
        "roofline": {"kernel": dominant, "bound": bound, "achieved": round(achieved, 1), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(achieved / peak, 4), "traffic": traffic,
                     "launches_per_step": dom_launches_step,
                     "flops_per_launch": round(dom_flops_step / max(dom_launches_step, 1)),
                     "mean_launch_us": round(1e3 * dom_ms_step / max(dom_launches_step, 1), 2)},
    }

    if w.decode_block and not args.only_step and not args.no_schedule:
        result.update(schedule_extras(args, w, setup, K, fl))

    if not args.no_cpu and not args.only_step:
        cb = cpu_baseline(w, setup.host, args.cpu_seconds)
        cb.pop("_probe_s"), cb.pop("_refresh_s")
        result["cpu_baseline"] = cb
    print(json.dumps(result), flush=True)


def schedule_extras(args, w, setup, K, fl):
    """The serving schedule: one probe per request, then per block of the
    masked span a selective refresh, LM head and greedy commit; against the
    same schedule with full recomputation.  One run of each, plus the peak KV
    memory each holds (paged plan) and the time of a decode step (a block's
    rows through every layer against the refresh's view)."""
    import torch

    import workloads as W
    from paper_2608_26140_amd import driver as D
    from paper_2608_26140_amd.workload import upload

    d, lay = w.dims, w.layout
    batch = setup.batch
    B, G, blk = w.batch, lay.mask_len, w.decode_block
    n_blocks = G // blk
    R = K + lay.n_nonaffix
    g_bits, head_bits = W.draw_lm_head(w)
    head = D.Head(upload(g_bits, d.dtype), upload(head_bits, d.dtype))
    ids0 = batch.remap.clone()
    plans = {"selective": D.DecodePlan(batch, K, blk, n_blocks, full=False),
             "full": D.DecodePlan(batch, K, blk, n_blocks, full=True)}
    logits = torch.empty((B * blk, d.vocab), dtype=head.w.dtype, device="cuda")
    committed = torch.empty((n_blocks, B * blk), dtype=torch.int32, device="cuda")
    paged = batch.pages is not None
    kv, ms = {}, {}
    for mode in ("selective", "full"):
        if paged:
            batch.release_private()
            batch.pages.reset_peak()
        batch.remap.copy_(ids0)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        D.decode_schedule(batch, head, plans[mode], K, logits, committed)
        e1.record()
        torch.cuda.synchronize()
        ms[mode] = e0.elapsed_time(e1)
        if mode == "selective":
            ids_sel = committed.cpu()
        if paged:
            st = batch.pages.stats()
            shared = len(batch.shared_host)
            kv[mode] = dict(peak_blocks=st["peak"], shared_blocks=shared, private_blocks=st["peak"] - shared)
        print(f"[bench] schedule {mode}: {ms[mode]:.0f} ms", file=sys.stderr, flush=True)
    batch.remap.copy_(ids0)

    # one decode step of block 0 after its refresh (selective mode), timed over 3 steps
    anchors, _ = batch.select_anchors(K)
    _, m = batch.refresh(anchors, K)
    D.decode_step(batch, plans["selective"], 0, m, anchors)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(3):
        D.decode_step(batch, plans["selective"], 0, m, anchors)
    e1.record()
    torch.cuda.synchronize()
    ms_decode = e0.elapsed_time(e1) / 3
    batch.remap.copy_(ids0)

    peak, _ = PEAK[d.dtype]
    tokens = B * G
    sched_flops = sum(fl["probe"].values()) + n_blocks * sum(fl["refresh"].values())
    out = {"schedule": {"blocks": n_blocks, "block": blk,
                        "selective_ms": round(ms["selective"], 2), "full_ms": round(ms["full"], 2),
                        "committed_tokens_per_s": round(tokens / (ms["selective"] * 1e-3), 1),
                        "full_committed_tokens_per_s": round(tokens / (ms["full"] * 1e-3), 1),
                        "speedup_vs_full": round(ms["full"] / ms["selective"], 3),
                        "recomputed_tokens_per_s": round(B * R * n_blocks / (ms["selective"] * 1e-3), 1),
                        "mfma_util": round(sched_flops / (ms["selective"] * 1e-3) / 1e12 / peak, 4),
                        "committed_ids_checksum": int(ids_sel.to(torch.int64).sum()),
                        "decode_step_ms": round(ms_decode, 3)}}
    if paged:
        GiB = float(1 << 30)
        sel, full = kv["selective"], kv["full"]
        out["kv_memory"] = {
            "block_size": batch.bs,
            "selective_peak_GiB": round(batch.kv_bytes(sel["peak_blocks"]) / GiB, 3),
            "selective_blocks": sel,
            # a system without ACache holds no shared affix region: its
            # requests' private blocks are its whole KV
            "full_recompute_peak_GiB": round(batch.kv_bytes(full["private_blocks"]) / GiB, 3),
            "full_blocks": full,
            "reduction": round(1 - sel["peak_blocks"] / full["private_blocks"], 4),
        }
    if args.tau >= 0:
        # block decoding with confidence-threshold commits: one run per mode
        decode = {"tau": args.tau}
        for mode in ("selective", "full"):
            batch.remap.copy_(ids0)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            steps = D.decode_threshold_schedule(batch, head, plans[mode], K, args.tau)
            torch.cuda.synchronize()
            t = (time.perf_counter() - t0) * 1e3
            decode[mode] = {"ms": round(t, 1), "steps_per_block": steps,
                            "committed_tokens_per_s": round(tokens / (t * 1e-3), 1)}
            print(f"[bench] threshold decode {mode}: {t:.0f} ms, steps {steps}", file=sys.stderr, flush=True)
        decode["speedup_vs_full"] = round(decode["full"]["ms"] / decode["selective"]["ms"], 3)
        batch.remap.copy_(ids0)
        out["threshold_decode"] = decode
    return out


def copy_calibration(args, A):
    """Identity row gather of MIB MiB: each launch reads every source row once
    (plus one int32 index per row) and writes it once."""
    import torch
    row = 8192
    n = args.copy_calibration * (1 << 20) // row
    src = torch.randint(0, 256, (n, row), dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    idx = torch.arange(n, dtype=torch.int32, device="cuda")
    for _ in range(args.warmup):
        A.acache_gather_rows(src, idx, out=dst)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        A.acache_gather_rows(src, idx, out=dst)
    e1.record()
    torch.cuda.synchronize()
    assert torch.equal(src, dst)
    ms = e0.elapsed_time(e1) / args.steps
    print(json.dumps({"copy_calibration": {"kernel": "gather_rows_kernel", "bytes_read": n * row + 4 * n,
                                           "bytes_written": n * row, "launches": args.warmup + args.steps,
                                           "ms_per_launch": round(ms, 4),
                                           "GB_per_s": round(2 * n * row / (ms * 1e-3) / 1e9, 1)}}), flush=True)


def cpu_baseline(w, host, budget_s):
    """The fp64 oracle on this host's cores: probe + top-K + selective refresh
    of request 0 (one request of the batch), repeated until about budget_s;
    reported as recomputed tokens/s of that sample.  For a stack the sample
    is layer 0 only (its shared affix cache is the layer-0 K/V of the affix
    rows, which are row-local), and the rate is extrapolated to all layers.
    cores: the BLAS threads the oracle ran on; host_cpus: the CPUs this
    process may run on."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import acache_oracle as O
    from tests.oracle_side import oracle_dims, oracle_layers, oracle_request, oracle_stale

    dims = oracle_dims(w)
    req = oracle_request(w, host, 0)
    n_layers = w.dims.n_layers
    K = O.anchor_count(w.ratio, w.layout.affix_len)
    R = K + w.layout.n_nonaffix
    if n_layers == 1:
        layers = oracle_layers(w, host)
        sk, sv = oracle_stale(w, host, layers)
    else:
        lay = w.layout
        layers = [O.layer_from_bits(host["layers"][0], dims, w.dims.dtype)]
        affix = np.arange(lay.affix_begin, lay.affix_end)
        k0, v0 = O.layer_kv(layers[0], dims, O.from_bits(host["embedding"][host["donor_ids"][affix]],
                                                          w.dims.dtype), affix)
        sk, sv = [k0], [v0]
    n, t, t_probe = 0, 0.0, 0.0
    while t < budget_s and n < 100:
        t0 = time.perf_counter()
        a, _ = O.select_anchors(layers, dims, req, sk, sv, K)
        t1 = time.perf_counter()
        O.selective_refresh(layers, dims, req, a, sk, sv)
        t += time.perf_counter() - t0
        t_probe += t1 - t0
        n += 1
    threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    sample = (f"request 0 of {w.batch}: probe + top-K + selective refresh ({R} rows), "
              f"{n} repetitions in {t:.1f}s, fp64 NumPy")
    if n_layers > 1:
        sample += f"; layer 0 only, rate extrapolated to {n_layers} layers (time x {n_layers})"
    return {"value": round(n * R / (t * n_layers), 2), "unit": "recomputed tokens/s",
            "cores": threads, "host_cpus": len(os.sched_getaffinity(0)), "kind": "oracle", "sample": sample,
            "_probe_s": t_probe / n * n_layers, "_refresh_s": (t - t_probe) / n * n_layers}


if __name__ == "__main__":
    main()
