"""Summaries of rocprofv3 runs of bench.py for profiles/ (runs on the host, no GPU).

    python profile_summary.py stats   RUN_DIR NAME BENCH_JSON OUT_TXT "COMMAND" [--steps N]
    python profile_summary.py traffic FETCH_CSV WRITE_CSV COPY_FETCH_CSV COPY_WRITE_CSV WORKLOAD OUT_TXT \
                                      "STEP_COMMAND" "COPY_COMMAND" [--steps N] [--copy-mib M]
    python profile_summary.py mfma    PMC_CSV WORKLOAD OUT_TXT "COMMAND" [--steps N]

stats: the kernel statistics of a `rocprofv3 --kernel-trace --stats` run
(RUN_DIR/NAME_kernel_stats.csv), and, from its kernel trace, the mean
duration of the dominant kernel's launches over the run's last N steps
beside bench.py's HIP-event figure for the same launches.

traffic: HBM bytes per launch of each operation of the step from two
`--pmc FETCH_SIZE` / `--pmc WRITE_SIZE` passes, scaled by what the same
counters read for the row-gather kernel copying M MiB (bench.py
--copy-calibration M); written to profiles/traffic.json (keyed by workload
and operation, with the digest of the kernel sources they were taken on)
and OUT_TXT.

mfma: the matrix units' activity per kernel over the last N steps from one
`--pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE SQ_INSTS_VALU_MFMA_MOPS_BF16`
pass: the share of cycles in which a SIMD's matrix unit is busy, the clock
the dispatch ran at, and the hardware-counted MFMA work.

A step holds one top-K launch, between its probe and its refresh.  The
run's last N steps are taken as the span from the launch after the
(N+1)-th last top-K to the last top-K: N refreshes and N probes of
identical steps.
"""

from __future__ import annotations

import csv
import json
import os
import re
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))

# operation -> (kernel-name patterns summed per launch unit, pattern that starts a unit); launches of
# one operation that follow each other directly are one unit (attention's whole-tile and remainder
# kernels, a GEMM and its stream-K fixup)
OPERATIONS = {
    # 256 x 256 tiles run gemm_bf16_w4_kernel (+ gemm_bf16_fixup16), 256 x 128 tiles gemm_bf16_kernel
    "gemm_gate_up": ([r"gemm_bf16_(w4_)?kernel<4,", r"gemm_bf16_fixup(16)?<4,"], r"gemm_bf16_(w4_)?kernel<4,"),
    "gemm_qkv": ([r"gemm_bf16_(w4_)?kernel<3,", r"gemm_bf16_fixup(16)?<3,"], r"gemm_bf16_(w4_)?kernel<3,"),
    "gemm_accum": ([r"gemm_bf16_(w4_)?kernel<1,", r"gemm_bf16_fixup(16)?<1,"], r"gemm_bf16_(w4_)?kernel<1,"),
    "gemm_partial": ([r"gemm_bf16_(w4_)?kernel<2,"], r"gemm_bf16_(w4_)?kernel<2,"),
    "attention": ([r"attention_(pv|wide)_kernel", r"attention_merge_kernel"], r"attention_(pv|wide)_kernel"),
    "score": ([r"score_fused_kernel"], r"score_fused_kernel"),
    "score_reduce": ([r"head_reduce_kernel"], r"head_reduce_kernel"),
    "rmsnorm": ([r"rmsnorm_vec_kernel", r"rmsnorm_rows_kernel"], r"rmsnorm_(vec|rows)_kernel"),
    "residual": ([r"reduce_residual_kernel", r"q_rotary_reduce_kernel"], r"(reduce_residual|q_rotary_reduce)_kernel"),
    "gather": ([r"gather_rows_kernel"], r"gather_rows_kernel"),
}
# bench.py's kernel names -> the operation whose launches it times
BENCH_KERNEL = {"gemm_gate_up": "gemm_gate_up", "gemm_qkv": "gemm_qkv", "attention": "attention"}


def _unmangled(name: str) -> str:
    """The last component of a mangled nested name (_ZN <len><id>... E), for
    the few rows the profiler leaves mangled."""
    if not name.startswith("_ZN"):
        return name
    i, last = 3, name
    while i < len(name) and name[i].isdigit():
        j = i
        while name[j].isdigit():
            j += 1
        n = int(name[i:j])
        last, i = name[j:j + n], j + n
    return last


def short(name: str) -> str:
    n = _unmangled(name)
    n = n.replace("acache::(anonymous namespace)::", "").replace("acache::", "").replace("void ", "")
    return re.sub(r"\(.*\)$", "", n)[:90]


def _rows(path):
    """CSV rows in launch order (the trace lists kernels as they complete)."""
    rows = list(csv.DictReader(open(path)))
    if rows and "Dispatch_Id" in rows[0]:
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    return rows


def _col(row, *names):
    for n in names:
        if n in row:
            return row[n]
    raise KeyError(names)


def _segment(rows, steps):
    """Rows of the last `steps` steps (see the module docstring)."""
    topk = [i for i, r in enumerate(rows) if "topk_kernel" in _col(r, "Kernel_Name", "Name")]
    if len(topk) < steps + 1:
        raise SystemExit(f"only {len(topk)} top-K launches; need {steps + 1}")
    return rows[topk[-steps - 1] + 1:topk[-1] + 1]


def stats(argv):
    run_dir, name, bench_json, out, cmd = argv[:5]
    steps = int(argv[argv.index("--steps") + 1]) if "--steps" in argv else 3
    st = _rows(os.path.join(run_dir, f"{name}_kernel_stats.csv"))
    bench = json.loads(open(bench_json).read().strip().splitlines()[-1])
    lines = [f"# rocprofv3 kernel statistics: {bench['config']['workload']} step", "",
             "command (from the repository root on the GPU box):", f"  {cmd}", "",
             f"{'kernel':92s} {'calls':>6s} {'avg_us':>10s} {'min_us':>9s} {'max_us':>9s} {'total_ms':>9s} {'pct':>6s}"]
    for r in st:
        lines.append(f"{short(r['Name']):92s} {r['Calls']:>6s} {float(r['AverageNs']) / 1e3:10.2f} "
                     f"{float(r['MinNs']) / 1e3:9.2f} {float(r['MaxNs']) / 1e3:9.2f} "
                     f"{float(r['TotalDurationNs']) / 1e6:9.3f} {float(r['Percentage']):6.2f}")
    lines += ["", "The calls include the setup (the shared cache's materialisation), the warmup steps and the",
              "timed steps."]
    trace = os.path.join(run_dir, f"{name}_kernel_trace.csv")
    roof = bench["roofline"]
    op = BENCH_KERNEL.get(roof["kernel"])
    if os.path.exists(trace) and op:
        seg = _segment(_rows(trace), steps)
        pats, unit = OPERATIONS[op]
        durs, n_units, prev = [], 0, False
        for r in seg:
            k = _col(r, "Kernel_Name", "Name")
            hit = any(re.search(p, k) for p in pats)
            if hit:
                d = int(_col(r, "End_Timestamp")) - int(_col(r, "Start_Timestamp"))
                if re.search(unit, k) and not prev:
                    durs.append(d)
                    n_units += 1
                else:
                    durs[-1] += d
            prev = hit
        mean = sum(durs) / max(n_units, 1) / 1e3
        lines += ["", f"Dominant kernel ({roof['kernel']}): {n_units} launches in the last {steps} steps of the trace "
                  f"({n_units / steps:g} per step), mean {mean:.2f} us per launch (a stream-K launch counts its fixup);",
                  f"bench.py's HIP events over its own timed region: {roof['mean_launch_us']:.2f} us "
                  f"({100 * (roof['mean_launch_us'] / mean - 1):+.1f}%)."]
    lines += ["", "bench.py line of the same run (timed region, HIP events):", json.dumps(bench)]
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines[:40]))


SIMDS = 1024  # 256 CUs x 4 SIMDs
XCDS = 8


def mfma(argv):
    csv_path, workload, out, cmd = argv[:4]
    steps = int(argv[argv.index("--steps") + 1]) if "--steps" in argv else 1
    per = {}  # dispatch -> (kernel, duration ns, {counter: value})
    for r in _rows(csv_path):
        d = int(r["Dispatch_Id"])
        if d not in per:
            per[d] = (r["Kernel_Name"], int(r["End_Timestamp"]) - int(r["Start_Timestamp"]), {})
        per[d][2][r["Counter_Name"]] = per[d][2].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    order = [{"Kernel_Name": per[d][0], "d": d} for d in sorted(per)]
    seg = _segment(order, steps)
    agg, names = {}, []
    for r in seg:
        k = short(r["Kernel_Name"])
        _, dur, c = per[r["d"]]
        if k not in agg:
            agg[k] = [0, 0.0, 0.0, 0.0, 0.0]
            names.append(k)
        a = agg[k]
        a[0] += 1
        a[1] += dur
        a[2] += c.get("GRBM_GUI_ACTIVE", 0.0)
        a[3] += c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        a[4] += c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0)
    lines = [f"# MFMA activity per kernel: {workload} step (rocprofv3 SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE,",
             "# SQ_INSTS_VALU_MFMA_MOPS_BF16)", "", "command (from the repository root on the GPU box):", f"  {cmd}", "",
             f"Dispatches of the last {steps} step(s).  GRBM_GUI_ACTIVE per dispatch is summed over the {XCDS} XCDs:",
             f"divided by {XCDS} and by the dispatch's duration it gives the clock.  MFMA busy =",
             f"SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / {XCDS} x {SIMDS} SIMDs): the share of cycles in which a",
             "SIMD's matrix unit is busy.  MFMA GFLOP = MOPS x 512 (hardware-counted, padded rows included).", "",
             f"{'kernel':60s} {'calls':>6s} {'avg_us':>9s} {'clock GHz':>9s} {'MFMA busy':>9s} {'MFMA GFLOP':>10s} "
             f"{'TFLOP/s':>8s}"]
    for k in sorted(names, key=lambda n: -agg[n][1]):
        n, dur, grbm, busy, mops = agg[k]
        cyc = grbm / XCDS
        lines.append(f"{k[:60]:60s} {n:6d} {dur / n / 1e3:9.1f} {cyc / dur if dur else 0:9.2f} "
                     f"{100 * busy / (cyc * SIMDS) if cyc else 0:8.1f}% {mops * 512 / 1e9 / n:10.1f} "
                     f"{mops * 512 / dur / 1e3 if dur else 0:8.0f}")
    lines += ["", "Short launches read a higher clock: the counting window is longer than the kernel."]
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def traffic(argv):
    fetch, write, cfetch, cwrite, workload, out, step_cmd, copy_cmd = argv[:8]
    steps = int(argv[argv.index("--steps") + 1]) if "--steps" in argv else 1
    mib = int(argv[argv.index("--copy-mib") + 1]) if "--copy-mib" in argv else 256
    sys.path.insert(0, ROOT)
    from paper_2608_26140_amd.build import source_digest

    def copy_mean(path):
        v = [float(_col(r, "Counter_Value")) for r in _rows(path) if "gather_rows_kernel" in _col(r, "Kernel_Name")]
        return sum(v) / len(v)

    n = mib * (1 << 20) // 8192
    read_b, write_b = n * 8192 + 4 * n, n * 8192
    rs = read_b / (copy_mean(cfetch) * 1024)
    ws = write_b / (copy_mean(cwrite) * 1024)

    def per_unit(path, pats, unit):
        seg = _segment(_rows(path), steps)
        tot, units, prev = 0.0, 0, False
        for r in seg:
            k = _col(r, "Kernel_Name")
            hit = any(re.search(p, k) for p in pats)
            if hit:
                tot += float(_col(r, "Counter_Value"))
                units += bool(re.search(unit, k)) and not prev
            prev = hit
        return tot / max(units, 1), units / steps

    lines = [f"# HBM traffic per launch: {workload} step (rocprofv3 FETCH_SIZE / WRITE_SIZE)", "",
             "commands (from the repository root on the GPU box), one pass per counter (C = FETCH_SIZE, WRITE_SIZE):",
             f"  {step_cmd}", f"  {copy_cmd}", "",
             f"calibration: gather_rows_kernel identity copy of {mib} MiB reads {read_b} B, writes {write_b} B per launch;",
             f"  FETCH_SIZE reads {copy_mean(cfetch):.0f} KiB -> read scale {rs:.4f}; "
             f"WRITE_SIZE {copy_mean(cwrite):.0f} KiB -> write scale {ws:.4f}", "",
             f"Launches of the last {steps} step(s); a stream-K GEMM launch counts its fixup kernel, attention its",
             "remainder-tile and key-split merge kernels.", "",
             f"{'operation':14s} {'per step':>8s} {'fetch_KiB':>11s} {'write_KiB':>11s} {'MB/launch':>10s}"]
    tfile = os.path.join(ROOT, "profiles", "traffic.json")
    rec = json.load(open(tfile)) if os.path.exists(tfile) else {}
    rec = {k: v for k, v in rec.items() if not k.startswith(workload + ":")}
    for op, (pats, unit) in OPERATIONS.items():
        fk, per = per_unit(fetch, pats, unit)
        wk, _ = per_unit(write, pats, unit)
        if per == 0:
            continue
        b = fk * 1024 * rs + wk * 1024 * ws
        lines.append(f"{op:14s} {per:8g} {fk:11.0f} {wk:11.0f} {b / 1e6:10.1f}")
        rec[f"{workload}:{op}"] = {"source_digest": source_digest(), "bytes_per_launch": round(b),
                                   "fetch_kib_per_launch": round(fk, 1), "write_kib_per_launch": round(wk, 1),
                                   "read_scale": round(rs, 4), "write_scale": round(ws, 4)}
    lines.append(f"\nsource digest of the measured kernels: {source_digest()}")
    json.dump(rec, open(tfile, "w"), indent=1)
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


if __name__ == "__main__":
    {"stats": stats, "traffic": traffic, "mfma": mfma}[sys.argv[1]](sys.argv[2:])
