#!/usr/bin/env python3
"""Benchmark of the LibraSpec verification step on one MI355X.

One step = the whole hot path on one batch:
  lsv_select_length (MARGINAL rule on the measured per-gamma cost table)
  -> lsv_verify_block (target forward over [root, x_1..x_gamma] against the KV cache)
  -> lsv_accept (greedy or speculative rejection sampling; commits the cached length),
captured once as a HIP graph and replayed.  Inputs are resident in HBM before the
timed region.  Default workload: Llama-3-70B-shaped random-init bf16 decoder (80
layers, d 8192, 64/8 x 128 heads, SwiGLU 28672, vocab 128256), batch 4, context 8192
per sequence prefilled from seeded random prompt ids, 32 drafted tokens per sequence
with confidences Beta(5, 3) * 0.9^i, greedy acceptance.  The drafts are planted: draft
v is the target's own greedy token with probability equal to its confidence, so the
realized acceptance follows the confidence model.

Prints one JSON line.  `value` = expected emitted tokens per second of the timed step
(sum over sequences of 1 + N_b(gamma_b), divided by the step latency); the line also
carries the realized tokens, the verified rows per second, and per gamma the latency,
tokens/s and the HBM / MFMA fractions (`per_gamma`).  `other_workloads` holds the same
figures for the --secondary workloads (default: Llama-3-8B shape, batch 1, context 2048).
With --rounds R (default 0: off, so profiles of the step see only its kernels) the line also
carries `decode_loop`: R rounds of multi-round decoding per length policy (static lengths,
the marginal rule, Algorithm 1, the G4-style rule) fed by a planted calibrated drafter, as
tokens per second against plain greedy decoding.
"""
import argparse
import ctypes
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "verify-step latency (us) & tokens/s vs gamma; % of HBM BW / MFMA bf16 peak"
HBM_PEAK_GBPS = 8000.0
HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000
MFMA_PEAK_FLOPS = 2.5e15  # dense bf16


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="llama3-70b-b4")
    p.add_argument("--secondary", default="llama3-8b-b1-c2048",
                   help="comma-separated workloads also measured after the primary one (their step, sweep and "
                        "dominant kernel only), or 'none'")
    p.add_argument("--secondary-steps", type=int, default=50)
    p.add_argument("--drafts", choices=("planted", "uniform"), default="planted",
                   help="greedy workloads: drafts planted from the target's own greedy continuation with "
                        "probability equal to their confidence, or the configs' uniform random ids")
    p.add_argument("--sweep-reps", type=int, default=10)
    p.add_argument("--roofline-steps", type=int, default=3)
    p.add_argument("--accept", choices=("greedy", "sample"), default=None,
                   help="acceptance rule of the timed steps (default: greedy where the workload has it, else "
                        "speculative rejection sampling at the workload's temperature)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--rounds", type=int, default=12,
                   help="multi-round decoding of the primary workload: rounds per length policy (planted drafter; "
                        "0 skips it)")
    p.add_argument("--calib-copy", action="store_true",
                   help="also run one plain 256 MiB copy kernel (counter calibration for --pmc runs)")
    p.add_argument("--counters-only", default="", metavar="GAMMA[,GAMMA...]",
                   help="counter runs of the profile: no prefill, sweep or CPU baseline; the eager roofline steps "
                        "at each uniform GAMMA in turn (every sequence), then the calibration copy")
    p.add_argument("--summarize", nargs=3, metavar=("TRACE_DIR", "FETCH_DIR", "WRITE_DIR"),
                   help="no GPU work: turn the csv output of three rocprofv3 runs of this script (kernel trace, "
                        "--pmc FETCH_SIZE, --pmc WRITE_SIZE; each dir also holds that run's bench.json) into the "
                        "gate/up profile summary of the run's workload")
    p.add_argument("--summarize-counters", nargs="+", metavar="DIR",
                   help="no GPU work: per-kernel counter summary (markdown) of --counters-only runs: the first "
                        "DIR holds a kernel-trace run of the same workload (durations), the others one --pmc "
                        "run each (bench.json + counter csv)")
    p.add_argument("--summarize-mfma", nargs=2, metavar=("TRACE_DIR", "PMC_DIR"),
                   help="no GPU work: matrix-core summary of the batched workload's uniform-gamma-max sweep "
                        "step from a kernel-trace run and a --pmc SQ_INSTS_MFMA SQ_VALU_MFMA_BUSY_CYCLES run "
                        "of the same bench command")
    return p.parse_args()


def log(msg):
    print(msg, file=sys.stderr, flush=True)


class HipEvents:
    """Raw hipEvent_t handles from the process's HIP runtime (for the timing hook)."""

    def __init__(self, n):
        from paper_2608_08721_amd import lsv
        self.hip = lsv.hip_runtime()
        self.ev = []
        for _ in range(n):
            e = ctypes.c_void_p()
            # timing-only events: no system-scope fence (cache write-back) when they are recorded
            assert self.hip.hipEventCreateWithFlags(ctypes.byref(e), ctypes.c_uint(HIP_EVENT_DISABLE_SYSTEM_FENCE)) == 0
            self.ev.append(e.value)

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(self.ev[a]), ctypes.c_void_p(self.ev[b]))
        assert rc == 0, rc
        return ms.value


def gateup_bytes(m, rows):
    """Algorithmic HBM bytes of one gate/up launch: the packed gate and up weights once, the
    normalised activation rows in, the SwiGLU output out."""
    es = 2 if m.dtype == "bf16" else 4
    return 2 * m.d_ff * m.d_model * es + rows * m.d_model * es + rows * m.d_ff * es


KERNEL_SOURCES = ("gemm.hip", "lsv_gemm.h", "lsv_device.h", "forward.hip")


def gateup_profile(workload):
    return os.path.join(ROOT, "profiles", f"gemm_gateup_{workload}.md")


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_08721_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, rows):
    """HBM bytes (read + written) per gate/up launch of `workload` at `rows` block rows, from the
    committed counter profile; None when there is none or the kernel sources changed since."""
    try:
        lines = open(gateup_profile(workload)).read().splitlines()
    except OSError:
        return None
    vals = dict(l.split(":", 1) for l in lines if l.startswith(("source_hash:", "traffic_rows_")))
    if vals.get("source_hash", "").strip() != kernel_source_hash():
        return None
    v = vals.get(f"traffic_rows_{rows}")
    return None if v is None else float(v)


def is_gateup(name):
    """The gate/up + SwiGLU launches: the 64-row kernel (kind 2, or 5 = the wide-model
    configuration) and the fused 64-row / batched kernel of batched bounds (kind 2)."""
    return ("gemm_kernel<unsigned short, 2," in name or "gemm_kernel<unsigned short, 5," in name
            or "gemm_fused_kernel<2," in name)


SELECT_KERNEL = "select_length_kernel"
CALIB_BYTES = 256 << 20


def _short(name):
    name = name.replace("void lsv::", "").replace("lsv::", "")
    return name.split("(")[0] if not name.startswith("__") else name


def _launch_groups(rows):
    """Dispatches of one logical gate/up launch: under a batched row bound the 64-row and the
    batched kernel run back to back (one of them returns at once), so runs of consecutive
    dispatch ids form one launch."""
    groups = []
    for r in rows:
        if groups and int(r["Dispatch_Id"]) == int(groups[-1][-1]["Dispatch_Id"]) + 1:
            groups[-1].append(r)
        else:
            groups.append([r])
    return groups


def summarize(trace_dir, fetch_dir, write_dir):
    """Profile summary (markdown) of the dominant kernel from three rocprofv3 runs of this
    script (--secondary none): the gate/up launches of the eager roofline steps (the last
    gate/up launches of the run), their kernel-trace durations and HBM counters, and the
    per-kernel split of the timed graph replays.  The timed region runs from the selector
    launch of the first timed replay to that of the first roofline step."""
    import csv
    import glob
    from synth import configs

    def one(d, pat):
        f = glob.glob(os.path.join(d, pat))
        assert len(f) == 1, (d, pat, f)
        return f[0]

    def bench_json(d):
        return json.loads(open(os.path.join(d, "bench.json")).read().strip().splitlines()[-1])

    bt = bench_json(trace_dir)
    wl = configs.WORKLOADS[bt["config"]["workload"]]
    m = wl.model
    rows = bt["roofline"]["rows"]
    trace = sorted(csv.DictReader(open(one(trace_dir, "*kernel_trace.csv"))), key=lambda r: int(r["Dispatch_Id"]))
    dur = lambda r: (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    n_roof = bt["roofline"]["launches_timed"]
    gu = _launch_groups([r for r in trace if is_gateup(r["Kernel_Name"])])[-n_roof:]
    roof_sum = [sum(dur(r) for r in g) for g in gu]
    roof_span = [(int(g[-1]["End_Timestamp"]) - int(g[0]["Start_Timestamp"])) / 1e3 for g in gu]
    names = sorted({_short(r["Kernel_Name"]) for g in gu for r in g})
    # one selector launch per step: a batch's timed step selects with the joint rule, whose kernel
    # first ran 1 + 2 x 20 times (the selection and its timing graph); a single sequence's with
    # MARGINAL, after the three rules' own selections; then the step before capture and the warmups
    if bt["config"]["batch"] > 1:
        sel = [r for r in trace if "select_joint_kernel" in r["Kernel_Name"]]
        i0 = 1 + 2 * 20 + 1 + bt["warmup"]
    else:
        sel = [r for r in trace if SELECT_KERNEL in r["Kernel_Name"]]
        i0 = 3 + 1 + bt["warmup"]
    t_lo, t_hi = int(sel[i0]["Start_Timestamp"]), int(sel[i0 + bt["steps"]]["Start_Timestamp"])
    per = {}
    for r in trace:
        if t_lo <= int(r["Start_Timestamp"]) < t_hi and "spin_kernel" not in r["Kernel_Name"]:
            per.setdefault(_short(r["Kernel_Name"]), []).append(dur(r))
    steps = bt["steps"]
    busy = sum(sum(v) for v in per.values()) / steps

    out = []
    w = out.append
    base = f"python3 bench.py --workload {wl.name} --secondary none --no-cpu-baseline --rounds 0"
    dirs = [os.path.normpath(d) for d in (trace_dir, fetch_dir, write_dir)]
    cmd_t = (f"rocprofv3 --kernel-trace --stats --output-format csv -d {dirs[0]} -o t -- {base} "
             f"--steps {bt['steps']} --warmup {bt['warmup']}")
    bf, bw = bench_json(fetch_dir), bench_json(write_dir)
    assert bf["config"]["counters_gammas"] == bw["config"]["counters_gammas"], "the two counter runs differ"
    cmd_c = ("rocprofv3 --pmc {c} --output-format csv -d {d} -o {o} -- " +
             f"python3 bench.py --workload {wl.name} --counters-only {bf['config']['counters_gammas']} "
             "--roofline-steps 2")
    w(f"# gate/up GEMM + SwiGLU: {wl.name} ({m.name} shape, batch {wl.batch}, context {bt['config']['context']}, "
      f"{rows} rows)")
    w("")
    w("Commands (repository root, after `cd /tmp && export TMPDIR=/tmp` for the profiler's own files; each")
    w("run's stdout saved as bench.json in its output directory):")
    w("")
    w("```")
    w(cmd_t)
    w(cmd_c.format(c="FETCH_SIZE", d=dirs[1], o="f"))
    w(cmd_c.format(c="WRITE_SIZE", d=dirs[2], o="w"))
    w(f"python3 bench.py --summarize {' '.join(dirs)}")
    w("```")
    w("")
    w(f"source_hash: {kernel_source_hash()}")
    w("")
    w("## Timing run")
    w("")
    w(f"- bench line: {bt['ms_per_step'] * 1e3:.1f} us per step at gamma {bt['config']['gamma']} "
      f"({bt['value']:.1f} tokens/s), step HBM fraction {bt['step']['hbm_frac']:.3f}")
    w(f"- gate/up launches of the eager roofline steps: {len(gu)} ({', '.join(names)}); kernel time "
      f"{statistics.mean(roof_sum):.2f} us per launch on average (first dispatch start to last dispatch end: "
      f"{statistics.mean(roof_span):.2f} us) vs {bt['roofline']['avg_launch_us']:.2f} us from the script's HIP "
      f"events (frac {bt['roofline']['frac']:.3f} of 8 TB/s)")
    w(f"- timed graph replays: kernels busy {busy:.1f} us of {bt['ms_per_step'] * 1e3:.1f} us per step")
    w("")
    w("| kernel (timed replays) | launches/step | avg us | us/step | share |")
    w("|---|---:|---:|---:|---:|")
    for k, v in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        w(f"| `{k}` | {len(v) / steps:g} | {statistics.mean(v):.2f} | {sum(v) / steps:.1f} | "
          f"{sum(v) / steps / busy * 100:.1f}% |")
    w("")

    def counters(d, name):
        """Calibration copy and, per row count of the run (in launch order), the counter summed
        over the dispatches of each gate/up launch."""
        rs = sorted(csv.DictReader(open(one(d, "*counter_collection.csv"))), key=lambda r: int(r["Dispatch_Id"]))
        rs = [r for r in rs if r["Counter_Name"] == name]
        copy = [float(r["Counter_Value"]) for r in rs if "copyBuffer" in r["Kernel_Name"]
                and int(r["Grid_Size"]) >= 131072]
        groups = _launch_groups([r for r in rs if is_gateup(r["Kernel_Name"])])
        rf = bench_json(d)["roofline"]
        last = groups[-rf["launches_timed"]:]
        n = rf["launches_per_rows"]
        return copy[-1], {r: [sum(float(x["Counter_Value"]) for x in g) for g in last[i * n:(i + 1) * n]]
                          for i, r in enumerate(rf["rows_list"])}
    f_copy, f_gu = counters(fetch_dir, "FETCH_SIZE")
    w_copy, w_gu = counters(write_dir, "WRITE_SIZE")
    assert rows in f_gu, f"the counter runs cover rows {sorted(f_gu)}, not the timed step's {rows}"
    f_scale = (CALIB_BYTES / 1024) / f_copy
    w_scale = (CALIB_BYTES / 1024) / w_copy
    w("## HBM traffic (two counter runs)")
    w("")
    w(f"Calibration: a plain {CALIB_BYTES >> 20} MiB device copy reads FETCH_SIZE {f_copy:.0f} KiB and "
      f"WRITE_SIZE {w_copy:.0f} KiB, so FETCH_SIZE is scaled by {f_scale:.3f} and WRITE_SIZE by {w_scale:.3f}.")
    w(f"Per gate/up launch ({len(f_gu[rows])} launches at each row count, uniform gamma per sequence, counters of "
      f"both dispatches of a launch summed), against the algorithmic bytes; the timed step ran {rows} rows:")
    w("")
    w("| rows | read MB | written MB | traffic MB | algorithmic MB | ratio |")
    w("|---:|---:|---:|---:|---:|---:|")
    traffic = {}
    for r in sorted(f_gu):
        rd = statistics.mean(f_gu[r]) * 1024 * f_scale
        wr = statistics.mean(w_gu[r]) * 1024 * w_scale
        alg = gateup_bytes(m, r)
        traffic[r] = rd + wr
        mark = "**" if r == rows else ""
        w(f"| {mark}{r}{mark} | {rd / 1e6:.2f} | {wr / 1e6:.2f} | {(rd + wr) / 1e6:.2f} | {alg / 1e6:.2f} | "
          f"{(rd + wr) / alg:.3f} |")
    w("")
    w("Bytes per launch (read + written) by block rows, read by bench.py while source_hash matches:")
    w("")
    w("```")
    for r in sorted(traffic):
        w(f"traffic_rows_{r}: {traffic[r]:.0f}")
    w("```")
    return "\n".join(out) + "\n"


MFMA_FLOPS_PER_INST = 16 * 16 * 32 * 2  # v_mfma_f32_16x16x32_bf16, the only MFMA of these kernels


def summarize_counters(trace_dir, pmc_dirs):
    """Per-kernel counter means of --counters-only runs (one --pmc run per directory), next to
    the kernel durations of a kernel-trace run, as markdown.  FETCH_SIZE and WRITE_SIZE are in
    KiB per dispatch as rocprofv3 reports them; the calibration copy at the end of each run
    gives the factor that turns them into bytes (a plain copy of CALIB_BYTES reads and writes
    that many bytes)."""
    import csv
    import glob
    import re

    def short(name):
        return re.sub(r"\(.*$", "", re.sub(r"^void ", "", name)).replace("lsv::", "").replace("unsigned short", "bf16")

    f = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)
    dur = {}
    for r in (csv.DictReader(open(f[0])) if f else []):
        dur.setdefault(short(r["Kernel_Name"]), []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    per = {}  # kernel -> counter -> [per-dispatch values]
    scale = {}
    runs = []
    bt = json.loads(open(os.path.join(trace_dir, "bench.json")).read().strip().splitlines()[-1])
    for d in pmc_dirs:
        f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        assert len(f) == 1, (d, f)
        disp = {}
        for r in csv.DictReader(open(f[0])):
            e = disp.setdefault(int(r["Dispatch_Id"]), {"name": short(r["Kernel_Name"]), "grid": int(r["Grid_Size"])})
            e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        cmds = json.loads(open(os.path.join(d, "bench.json")).read().strip().splitlines()[-1])
        names = sorted({k for e in disp.values() for k in e if k not in ("name", "grid")})
        runs.append((d, names, cmds["config"]["workload"]))
        # a run over several gammas: only the verify calls (each starts at its embedding kernel)
        # at the trace run's row count
        rows_list = cmds["roofline"].get("rows_list", [cmds["roofline"]["rows"]])
        n_calls = sum("embed_kernel" in e["name"] for e in disp.values())
        per_rows = n_calls // len(rows_list)
        gi = rows_list.index(bt["roofline"]["rows"]) if len(rows_list) > 1 else 0
        call = -1
        for i in sorted(disp):
            e = disp[i]
            if "embed_kernel" in e["name"]:
                call += 1
            if len(rows_list) > 1 and call >= 0 and not gi * per_rows <= call < (gi + 1) * per_rows \
                    and "copyBuffer" not in e["name"]:
                continue
            if "copyBuffer" in e["name"]:
                if e["grid"] >= 131072:  # the calibration copy (the last one): bytes per counter unit
                    for c in ("FETCH_SIZE", "WRITE_SIZE"):
                        if e.get(c, 0.0) > 0:
                            scale[c] = CALIB_BYTES / e[c]
                continue
            for c in names:
                if c in e:
                    per.setdefault(e["name"], {}).setdefault(c, []).append(e[c])
    wl = runs[0][2] if runs else "?"
    from synth import configs
    B = configs.WORKLOADS[wl].batch if wl in configs.WORKLOADS else 1
    cmds = [f"rocprofv3 --kernel-trace --stats --output-format csv -d {os.path.normpath(trace_dir)} -o t -- python3 "
            f"bench.py --workload {wl} --secondary none --no-cpu-baseline --rounds 0 --steps {bt['steps']} "
            f"--warmup {bt['warmup']}"]
    for d, names, _ in runs:
        bj = json.loads(open(os.path.join(d, "bench.json")).read().strip().splitlines()[-1])
        g = bj["config"].get("counters_gammas", bj["roofline"]["rows"] // B - 1)
        dn = os.path.normpath(d)
        cmds.append(f"rocprofv3 --pmc {' '.join(names)} --output-format csv -d {dn} -o {os.path.basename(dn)[0]} -- "
                    f"python3 bench.py --workload {wl} --counters-only {g} --roofline-steps 2")
    cmds.append("python3 bench.py --summarize-counters " + " ".join(os.path.normpath(x) for x in [trace_dir] + list(pmc_dirs)))
    out = [f"# Per-kernel counters: {wl}\n",
           "Commands (repository root, after `cd /tmp && export TMPDIR=/tmp` for the profiler's own files; each run's "
           "stdout saved as bench.json in its output directory):\n", "```", *cmds, "```\n",
           "Counter runs (`--counters-only`: eager verify steps at uniform gammas, the cache holding zeros, which "
           "changes no kernel's traffic or instruction mix), one `--pmc` set per run; values are means per "
           f"dispatch over the calls at the kernel-trace run's {bt['roofline']['rows']} rows. Kernels are listed by "
           "their total time in the kernel-trace run; the timed step's per-kernel durations are in the gate/up "
           "summary of the same workload.\n"]
    for d, names, _ in runs:
        out.append(f"- `{os.path.basename(os.path.normpath(d))}`: {' '.join(names)}")
    out.append("")
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        if c in scale:
            out.append(f"- {c} scale from the calibration copy: {scale[c]:.3f} bytes per counter unit")
    out.append("")
    # the verify step's kernels only (not the packing, the workspace fills or the calibration copy)
    per = {k: v for k, v in per.items() if re.match(r"(gemm_|attn_|rmsnorm_|embed_|tree_|commit_)", k)}
    cols = sorted({c for k in per.values() for c in k})
    hdr = "| kernel | dispatches | " + " | ".join(cols) + " |"
    out.append(hdr)
    out.append("|---|---:|" + "---:|" * len(cols))
    order = sorted(per, key=lambda k: -sum(dur.get(k, [0.0])))
    for k in order:
        n = max(len(v) for v in per[k].values())
        row = [f"`{k[:60]}`", str(n)]
        for c in cols:
            v = per[k].get(c)
            if not v:
                row.append("-")
                continue
            mean = sum(v) / len(v)
            if c in scale:
                row.append(f"{mean * scale[c] / 1e6:.2f} MB")
            else:
                row.append(f"{mean:.4g}")
        out.append("| " + " | ".join(row) + " |")
    out.append("")
    # derived ratios where the counters are there
    for k in order:
        c = {n: sum(v) / len(v) for n, v in per[k].items()}
        notes = []
        if c.get("SQ_INSTS_LDS"):
            if "SQ_LDS_BANK_CONFLICT" in c:
                notes.append(f"SQ_LDS_BANK_CONFLICT / SQ_INSTS_LDS {c['SQ_LDS_BANK_CONFLICT'] / c['SQ_INSTS_LDS']:.3f}")
        if c.get("SQ_WAVE_CYCLES") and "SQ_WAIT_INST_ANY" in c:
            notes.append(f"SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES {c['SQ_WAIT_INST_ANY'] / c['SQ_WAVE_CYCLES']:.2f}")
        if c.get("SQ_BUSY_CYCLES") and "SQ_WAVE_CYCLES" in c:
            notes.append(f"SQ_WAVE_CYCLES / SQ_BUSY_CYCLES {c['SQ_WAVE_CYCLES'] / c['SQ_BUSY_CYCLES']:.1f}")
        if notes:
            out.append(f"- `{k[:60]}`: " + "; ".join(notes))
    return "\n".join(out) + "\n"


def summarize_mfma(trace_dir, pmc_dir):
    """Matrix-core summary (markdown) of the batched workload at its largest uniform gamma:
    per kernel kind, duration from a kernel-trace run and SQ_INSTS_MFMA / SQ_VALU_MFMA_BUSY_CYCLES
    from a counter run of the same command.  Both runs issue the same calls in the same order;
    a call starts at its embedding kernel, and the calls at the largest gamma are the ones whose
    gate/up launches issue the most MFMAs (the row count picks the kernel body on the device)."""
    import csv
    import glob
    from synth import configs, gen

    def one(d, pat):
        f = glob.glob(os.path.join(d, "**", pat), recursive=True)
        assert len(f) == 1, (d, pat, f)
        return f[0]

    bt = json.loads(open(os.path.join(trace_dir, "bench.json")).read().strip().splitlines()[-1])
    wl = configs.WORKLOADS[bt["config"]["workload"]]
    m, G, B = wl.model, wl.G, wl.batch
    ctx = [int(c) for c in gen.contexts(wl)]
    rows = B * (G + 1)

    def calls_of(rows_in):
        calls, cur = [], None
        for r in rows_in:
            if r["Kernel_Name"].startswith("void lsv::embed_kernel") or "embed_kernel" in r["Kernel_Name"]:
                cur = []
                calls.append(cur)
            if cur is not None:
                cur.append(r)
        return calls

    trace = sorted(csv.DictReader(open(one(trace_dir, "*kernel_trace.csv"))), key=lambda r: int(r["Dispatch_Id"]))
    tcalls = calls_of(trace)
    pm = {}
    for r in csv.DictReader(open(one(pmc_dir, "*counter_collection.csv"))):
        d = pm.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"], "grid": int(r["Grid_Size"])})
        d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    prow = [dict(Dispatch_Id=k, Kernel_Name=v["name"], **v) for k, v in sorted(pm.items())]
    pcalls = calls_of(prow)
    assert len(pcalls) == len(tcalls), (len(pcalls), len(tcalls))

    def gateup_mfma(call):
        v = [r["SQ_INSTS_MFMA"] for r in call if "gemm_fused_kernel<2," in r["Kernel_Name"]]
        return max(v) if v else 0
    top = max(gateup_mfma(c) for c in pcalls)
    hits = [i for i, c in enumerate(pcalls) if top > 0 and gateup_mfma(c) == top]
    assert hits, "no batched gate/up launches in the counter run"
    # prefill chunks of full blocks issue as many; the sweep's last gamma is the last run of
    # consecutive calls that do
    picked = [hits[-1]]
    while picked[0] - 1 in hits:
        picked.insert(0, picked[0] - 1)

    d, F, V = m.d_model, m.d_ff, m.vocab
    n_qkv = (m.n_q_heads + 2 * m.n_kv_heads) * m.head_dim
    att_flops = sum(sum(4 * m.n_q_heads * m.head_dim * (C + v + 1) for v in range(G + 1)) for C in ctx)
    useful = {"QKV": 2.0 * rows * n_qkv * d, "O": 2.0 * rows * d * m.n_q_heads * m.head_dim,
              "gate/up": 2.0 * rows * 2 * F * d, "down": 2.0 * rows * d * F, "LM head": 2.0 * rows * V * d,
              "attention split": float(att_flops)}

    def kind(name, seen):
        for k, label in (("gemm_fused_kernel<2,", "gate/up"), ("gemm_fused_kernel<1,", "O"),
                         ("gemm_fused_kernel<3,", "down"), ("gemm_fused_kernel<0,", "QKV"),
                         ("gemm_fused_kernel<4,", "LM head")):
            if k in name:
                return label
        if "attn_split" in name:
            return "attention split"
        return None

    stats = {}
    for i in picked:
        seen = {"resid": 0, "logits": 0}
        for tr, pr in zip(tcalls[i], pcalls[i]):
            assert _short(tr["Kernel_Name"]) == _short(pr["Kernel_Name"]), (tr["Kernel_Name"], pr["Kernel_Name"])
            k = kind(tr["Kernel_Name"], seen)
            if k is None:
                continue
            s = stats.setdefault(k, {"dur": [], "mfma": [], "busy": []})
            s["dur"].append((int(tr["End_Timestamp"]) - int(tr["Start_Timestamp"])) / 1e3)
            s["mfma"].append(pr.get("SQ_INSTS_MFMA", 0.0))
            s["busy"].append(pr.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0))

    out = []
    w = out.append
    cmd = ("python3 bench.py --workload {w} --secondary none --rounds 0 --steps 2 --warmup 1 --sweep-reps 1 "
           "--roofline-steps 1 --no-cpu-baseline").format(w=wl.name)
    td, pd = os.path.normpath(trace_dir), os.path.normpath(pmc_dir)
    w(f"# Batched GEMMs and attention on the matrix cores: {wl.name}, uniform gamma {G} ({rows} rows)")
    w("")
    w("Commands (repository root, after `cd /tmp && export TMPDIR=/tmp`; each run's stdout saved as bench.json in")
    w("its output directory):")
    w("")
    w("```")
    w(f"rocprofv3 --kernel-trace --output-format csv -d {td} -o t -- {cmd}")
    w(f"rocprofv3 --pmc SQ_INSTS_MFMA SQ_VALU_MFMA_BUSY_CYCLES --output-format csv -d {pd} -o c -- {cmd}")
    w(f"python3 bench.py --summarize-mfma {td} {pd}")
    w("```")
    w("")
    w(f"Calls at gamma {G}: {len(picked)} (the sweep's graph body, run 1 + 3 + 1 times). Durations are kernel-trace")
    w("times of the plain run. Issued rate: SQ_INSTS_MFMA x 16384 flops (v_mfma_f32_16x16x32_bf16) per second;")
    w("useful rate: the product's own 2·M·N·K (attention: QKᵀ and PV over each row's causal context) per second;")
    w("both as a share of the 2.5 PFLOP/s dense bf16 peak. The busy column is SQ_VALU_MFMA_BUSY_CYCLES over")
    w("duration x 2.4 GHz x 1024 SIMDs.")
    w("")
    w("| kernel | launches per call | avg us | MFMA instructions per launch | issued % of peak | useful % of peak | MFMA busy |")
    w("|---|---:|---:|---:|---:|---:|---:|")
    order = ["gate/up", "attention split", "down", "O", "QKV", "LM head"]
    for k in order:
        if k not in stats:
            continue
        s = stats[k]
        dur = statistics.mean(s["dur"])
        inst = statistics.mean(s["mfma"])
        busy = statistics.mean(s["busy"])
        issued = inst * MFMA_FLOPS_PER_INST / (dur * 1e-6) / MFMA_PEAK_FLOPS
        use = useful[k] / (dur * 1e-6) / MFMA_PEAK_FLOPS  # per launch (attention: one layer)
        w(f"| {k} | {len(s['dur']) / len(picked):g} | {dur:.2f} | {inst:.0f} | {issued * 100:.1f}% | {use * 100:.1f}% | "
          f"{busy / (dur * 1e-6 * 2.4e9 * 1024) * 100:.1f}% |")
    w("")
    sw = bt.get("uniform_gamma_max", {})
    if sw:
        w(f"Whole step at gamma {G} (HIP events, graph replays, no profiler): {sw['latency_us']:.0f} us, "
          f"{sw['mfma_frac'] * 100:.1f}% of the MFMA peak, {sw['hbm_frac'] * 100:.1f}% of 8 TB/s.")
    return "\n".join(out) + "\n"


def step_bytes(m, contexts, rows):
    es = 2 if m.dtype == "bf16" else 4
    kv_row = 2 * m.n_kv_heads * m.head_dim * es
    return m.matmul_params() * es + m.n_layers * (sum(contexts) + rows) * kv_row


def step_flops(m, contexts, rows_per_seq):
    M = sum(rows_per_seq)
    att = 0
    for C, r in zip(contexts, rows_per_seq):
        att += sum(4 * m.n_q_heads * m.head_dim * (C + v + 1) for v in range(r))
    return 2 * M * m.matmul_params() + m.n_layers * att


def expected_tokens(conf_np, gammas):
    """Expected emitted tokens of one step under the drafter-confidence model (Assumption 3.7):
    sum_b 1 + N_b(gamma_b), N_b(g) = sum_{j<=g} prod_{k<=j} q_{b,k} (Eq. 2's numerator)."""
    e = 0.0
    for b, g in enumerate(gammas):
        e += 1.0 + float(np.cumprod(conf_np[b].astype(np.float64))[:g].sum())
    return e


def cpu_baseline(m, seed, ctx, rows_per_seq, tokens, exp_tok):
    """The oracle (fp64 numpy) on a bounded sample of the same step: the verify forward of the
    same block (every sequence, every row) at full width with 1 and then 2 of the model's layers
    (+ embedding and LM head), followed by greedy acceptance, context from the seeded KV generator;
    the per-layer time is extrapolated to all layers.  Value: the step's expected emitted tokens
    per second of oracle time."""
    from threadpoolctl import threadpool_info

    from oracle import accept as OA
    from oracle import forward as OF
    from synth import gen
    B = len(ctx)
    off = np.concatenate([[0], np.cumsum(rows_per_seq)]).astype(np.int64)
    ws = {"embed": gen.embed_weights(m, seed), "final_norm": gen.final_norm_weights(m),
          "lm_head": gen.lm_head_weights(m, seed), "layers": [gen.layer_weights(m, seed, l) for l in range(2)]}
    times = []
    for L in (1, 2):
        shape = m.with_layers(L)
        cache = OF.KVCache(shape, B, max(ctx) + max(rows_per_seq))
        for l in range(L):
            for b in range(B):
                k, v = gen.synthetic_kv(shape, seed + 31 * b, l, 1, ctx[b])
                cache.k[l][b, :, :ctx[b]] = OF.stored_to_f64(k[0], m.dtype)
                cache.v[l][b, :, :ctx[b]] = OF.stored_to_f64(v[0], m.dtype)
        model = OF.Model(shape, {**ws, "layers": ws["layers"][:L]})
        t0 = time.perf_counter()
        lg, _ = OF.verify_block(model, cache, ctx, tokens, off)
        OA.accept_greedy(lg, off, tokens)
        times.append(time.perf_counter() - t0)
        log(f"cpu baseline: {L} layer(s) {times[-1]:.1f} s")
    per_layer = max(times[1] - times[0], 1e-9)
    fixed = max(times[0] - per_layer, 0.0)
    t_step = fixed + m.n_layers * per_layer
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    return {"value": exp_tok / t_step, "unit": "tokens/s (expected emitted, confidence model)", "cores": int(threads),
            "kind": "oracle",
            "sample": f"fp64 numpy oracle: the step's verify forward ({sum(rows_per_seq)} rows over {B} sequences, "
                      f"contexts {sorted(set(ctx))}) at {m.name} width with 1 and 2 of {m.n_layers} layers + embedding "
                      f"+ LM head, then greedy acceptance; {times[0]:.1f} s + {times[1]:.1f} s measured, per-layer "
                      f"time extrapolated to {m.n_layers} layers; host cpu_count {os.cpu_count()}",
            "seconds_per_step": t_step}


def length_rules(wl, cost, dev, n_rows=4096):
    """The length rules on the measured cost table over many draws of the workload's
    confidence model -- the synthetic analogue of the trade-off sensitivity of Table 4 and of
    the deviation from the oracle length of Sec. 4.7.  Per rule: mean length, mean
    |gamma - gamma_exhaustive|, and the mean of f(gamma) / f(gamma_exhaustive) with
    f = (sum_{j<=gamma} prod_{k<=j} q_k) / cost[gamma], Eq. 2's objective as the selectors run it
    (no LSV_SEL_BONUS), so EXHAUSTIVE's own ratio is 1 and no rule's exceeds it; Algorithm 1 also
    the drafter blocks of n its budget requests.  All selections run in the library's selector on
    the GPU."""
    import torch

    from paper_2608_08721_amd import lsv
    from synth import gen
    G = wl.G
    conf_np = gen.confidences(wl, seed=wl.seed + 7, batch=n_rows)
    conf = torch.tensor(conf_np, device=dev)
    cost_t = torch.tensor(cost, dtype=torch.float64, device=dev)
    gamma = torch.zeros(n_rows, dtype=torch.int32, device=dev)
    aux = torch.zeros(n_rows, dtype=torch.int32, device=dev)
    p = np.cumprod(conf_np.astype(np.float64), axis=1)
    n_tok = np.cumsum(p, axis=1)                            # N(gamma), gamma = 1..G
    f = n_tok / np.asarray(cost[1:G + 1], dtype=np.float64)[None, :]
    rows = np.arange(n_rows)

    def run(mode, alpha=2.2, n=8, d_init=1):
        lsv.lsv_select_length(mode, n_rows, G, conf, cost_t, d_init, G, alpha, n, 0, gamma, aux, None, None)
        torch.cuda.synchronize()
        return gamma.cpu().numpy().astype(np.int64), aux.cpu().numpy().astype(np.int64)

    g_ex, _ = run(lsv.LSV_SEL_EXHAUSTIVE)
    f_ex = f[rows, g_ex - 1]

    def summary(g, extra=None):
        r = {"mean_gamma": round(float(g.mean()), 3), "mad_vs_exhaustive": round(float(np.abs(g - g_ex).mean()), 3),
             "objective_vs_exhaustive": round(float((f[rows, g - 1] / f_ex).mean()), 4)}
        if extra:
            r.update(extra)
        return r
    out = {"rows": n_rows, "confidence_model": list(wl.conf), "cost": "the measured per-gamma step latency",
           "exhaustive": summary(g_ex)}
    out["marginal_from_1"] = summary(run(lsv.LSV_SEL_MARGINAL, d_init=1)[0])
    out["marginal_from_G"] = summary(run(lsv.LSV_SEL_MARGINAL, d_init=G)[0])
    for n in (8, 16):
        if n > G:
            continue
        for a in (1.8, 2.0, 2.2, 2.6):
            g, blk = run(lsv.LSV_SEL_ALG1, alpha=a, n=n)
            out[f"alg1_n{n}_alpha{a}"] = summary(g, {"mean_blocks": round(float(blk.mean()), 3),
                                                     "blocks_all_up_front": -(-G // n)})
    mean_f = f.mean(axis=0)
    g_st = int(np.argmax(mean_f)) + 1                       # the best single static length on these draws
    out[f"static_best_{g_st}"] = summary(np.full(n_rows, g_st))
    return out


def decode_loop_measure(m, cfg, dm, B, G, ctx, prompts, pre, rows_buf, roots, cost, cost_total, seed, n_rounds, dev):
    """Multi-round decoding (select or a baseline policy -> pack -> verify -> accept -> next
    roots, one graph per round) on its own cache with room for the rounds, fed by the planted
    calibrated drafter: realized tokens per second for each length policy, against plain greedy
    decoding (gamma = 0) on the same GPU.  The drafter plants the target's own greedy stream,
    taken from the plain run."""
    import torch

    from paper_2608_08721_amd import decode, lsv, runtime
    from synth import drafter
    i32 = lambda x: torch.tensor(np.asarray(x, dtype=np.int32), device=dev)
    n_tok = n_rounds * (G + 1) + G + 2  # the longest stream any policy can consume
    cap2 = runtime.kv_capacity(max(ctx) + n_tok + G + 2)
    kv2 = runtime.KVCache(cfg, B, cap2, dev)
    ws2 = runtime.Workspace(lsv.lsv_verify_workspace_bytes(cfg, B, rows_buf, cap2), dev)
    lg2 = torch.zeros((rows_buf, m.vocab), dtype=torch.float32, device=dev)
    st2 = torch.zeros(B, dtype=torch.int32, device=dev)
    filled = [0] * B
    while filled != ctx:
        take = [min(pre, ctx[b] - filled[b]) for b in range(B)]
        off = runtime.row_offsets_of(take)
        toks = np.concatenate([prompts[b][filled[b]:filled[b] + take[b]] for b in range(B)])
        lsv.lsv_verify_block(cfg, dm.buf, kv2.buf, cap2, B, i32(filled), i32(toks), i32(off), rows_buf, cap2, lg2,
                             st2, ws2.buf, ws2.nbytes)
        filled = [filled[b] + take[b] for b in range(B)]
    del ws2, lg2
    ev = lambda: torch.cuda.Event(enable_timing=True)

    def timed(loop):
        loop.reset(ctx, roots)
        torch.cuda.synchronize()
        e0, e1 = ev(), ev()
        e0.record()
        for _ in range(n_rounds):
            loop.replay()
        e1.record()
        torch.cuda.synchronize()
        toks = int((loop.seq_len.cpu() - torch.tensor(ctx, dtype=torch.int32)).sum())
        return e0.elapsed_time(e1), toks

    cost_d = torch.tensor(cost, dtype=torch.float64, device=dev)
    g_ex = torch.zeros(B, dtype=torch.int32, device=dev)

    def streams(loop, n, mad=None, blocks=None):
        """Replay round by round until every sequence emitted n tokens; with mad (a list), also
        append |gamma - gamma_exhaustive| per sequence and round, the exhaustive length taken on
        the round's own confidences and the measured cost table."""
        loop.reset(ctx, roots)
        got = [[] for _ in range(B)]
        while min(len(g) for g in got) < n:
            loop.replay()
            if mad is not None:
                lsv.lsv_select_length(lsv.LSV_SEL_EXHAUSTIVE, B, G, loop.conf, cost_d, 1, G, 0.0, 1, 0, g_ex, None,
                                      None, None)
                mad += [abs(a - e) for a, e in zip(loop.gamma.cpu().tolist(), g_ex.cpu().tolist())]
            if blocks is not None:  # blocks the drafter produced this round (on demand for alg1)
                blocks += loop.blocks.cpu().tolist()
            for b, e in enumerate(loop.emitted()):
                got[b] += e
        return got

    plain = decode.DecodeLoop(cfg, dm, kv2, cap2, B, G, "static", None, gamma0=0)
    plain.reset(ctx, roots)
    plain.round()
    plain.capture()
    greedy = streams(plain, n_tok)
    ms_plain, tok_plain = timed(plain)
    del plain
    stream = np.zeros((B, cap2), np.int64)
    for b in range(B):
        stream[b, ctx[b]] = roots[b]
        stream[b, ctx[b] + 1:ctx[b] + 1 + n_tok] = greedy[b][:n_tok]
    q = drafter.confidences(seed, B, cap2)
    dr = drafter.PlantedDrafter(stream, q, seed, m.vocab, G, device=dev)
    base_tps = tok_plain / (ms_plain * 1e-3)
    out = {"rounds": n_rounds, "drafter": "planted greedy stream, confidences Beta(6, 1.5), calibrated",
           "stream_note": "blocks of more than 64 rows take the batched GEMM path, whose split-K sum rounds "
                          "differently in bf16 from the 64-row path that plain decoding takes: such a policy's "
                          "greedy stream can part from plain decoding at a near-tie (the blocks of at most 64 rows "
                          "give bit-identical rows whatever their size)",
           "plain_decoding": {"tokens_per_s": base_tps, "ms_per_token": ms_plain / max(tok_plain, 1)},
           "policies": {}}
    policies = [("static", g, None) for g in (2, 4, 8, G)] + [("marginal", None, None), ("g4", 8, None)]
    if B > 1:
        policies.append(("joint", None, None))
    policies += [("alg1", None, a) for a in (1.8, 2.0, 2.2, 2.6)]  # the trade-off sweep
    for pol, g0, alpha in policies:
        loop = decode.DecodeLoop(cfg, dm, kv2, cap2, B, G, pol, dr, cost=cost_total if pol == "joint" else cost,
                                 block_n=8, gamma0=g0, alpha=alpha or 2.2)
        loop.reset(ctx, roots)
        loop.round()
        loop.capture()
        ms, toks = timed(loop)
        mad, blocks = [], ([] if pol == "alg1" else None)
        got = streams(loop, n_rounds, mad, blocks)  # the emitted stream of n_rounds tokens or more per sequence
        n_cmp = min(min(len(g) for g in got), n_tok)
        same = all(got[b][:n_cmp] == greedy[b][:n_cmp] for b in range(B))
        name = {"static": f"static{g0}", "alg1": f"alg1_alpha{alpha}"}.get(pol, pol)
        out["policies"][name] = {"tokens_per_round": toks / (n_rounds * B), "ms_per_round": ms / n_rounds,
                                 "tokens_per_s": toks / (ms * 1e-3), "speedup_vs_plain": toks / (ms * 1e-3) / base_tps,
                                 "mad_vs_exhaustive": statistics.mean(mad), "stream_equals_plain": same}
        if blocks:  # drafter blocks of n = 8 that Algorithm 1's budget requested per sequence and round
            out["policies"][name]["blocks_per_round"] = statistics.mean(blocks)
            out["policies"][name]["blocks_all_up_front"] = -(-G // 8)
        del loop
    return out


class Workload:
    """One workload's device state: packed model, KV cache prefilled from seeded prompts,
    workspaces and the pending root token of every sequence (all untimed set-up)."""

    def __init__(self, wl, dev):
        import torch

        from paper_2608_08721_amd import lsv, runtime
        from synth import gen
        self.wl, self.m, self.dev = wl, wl.model, dev
        m = self.m
        self.i32 = lambda x: torch.tensor(np.asarray(x, dtype=np.int32), device=dev)
        self.seed, self.B, self.G = wl.seed, wl.batch, wl.G
        B, G = self.B, self.G
        self.ctx = [int(c) for c in gen.contexts(wl)]
        self.rows_seq = G + 1                # root + drafts per sequence
        # prefill rows per sequence and call: for batches, keep the whole block within the
        # batched GEMM path's row bound
        self.pre = 64 if B == 1 else max(1, min(64, lsv.LSV_WIDE_ROWS // B))
        self.rows_step = B * self.rows_seq   # host row bound of the verify steps
        self.rows_buf = max(self.rows_step, B * self.pre)
        self.cap = runtime.kv_capacity(max(self.ctx) + self.rows_seq)
        self.cfg = runtime.model_config(m)
        t0 = time.time()
        self.dm = runtime.DeviceModel(self.cfg, dev)
        self.dm.pack_globals(gen.embed_weights(m, self.seed), gen.final_norm_weights(m),
                             gen.lm_head_weights(m, self.seed))
        for l in range(m.n_layers):
            self.dm.pack_layer(l, gen.layer_weights(m, self.seed, l))
            if l % 8 == 7:
                log(f"{wl.name}: packed layer {l + 1}/{m.n_layers} ({time.time() - t0:.1f} s)")
        self.kv = runtime.KVCache(self.cfg, B, self.cap, dev)
        self.ws = runtime.Workspace(lsv.lsv_verify_workspace_bytes(self.cfg, B, self.rows_buf, self.cap), dev)
        self.aws = runtime.Workspace(lsv.lsv_accept_workspace_bytes(B, self.rows_buf, m.vocab), dev)
        self.logits = torch.zeros((self.rows_buf, m.vocab), dtype=torch.float32, device=dev)
        self.status = torch.zeros(B, dtype=torch.int32, device=dev)
        self.acc = torch.zeros(B, dtype=torch.int32, device=dev)
        self.out = torch.zeros((B, self.rows_seq), dtype=torch.int32, device=dev)
        # prefill every context from seeded prompt ids, in chunks of `pre` rows per sequence; a
        # sequence starts late enough that all of them end in the last call
        self.prompts = gen.prefix_ids(self.seed, B, self.ctx, m.vocab)
        chunks = [(c + self.pre - 1) // self.pre for c in self.ctx]
        n_calls = max(chunks)
        filled = [0] * B
        for i in range(n_calls):
            take = []
            for b in range(B):
                first = n_calls - chunks[b]
                take.append(0 if i < first else (self.ctx[b] - (chunks[b] - 1) * self.pre if i == first else self.pre))
            off = runtime.row_offsets_of(take)
            toks = np.concatenate([self.prompts[b][filled[b]:filled[b] + take[b]] for b in range(B)])
            self.verify(filled, toks, off, self.rows_buf)
            filled = [filled[b] + take[b] for b in range(B)]
        assert filled == self.ctx
        # roots = greedy tokens after each prompt, by the library's own acceptance on one row each
        last_rows = torch.tensor(off[1:] - 1, dtype=torch.long, device=dev)
        self.status.zero_()
        lsv.lsv_accept(lsv.LSV_ACC_GREEDY, B, m.vocab, self.logits[last_rows].contiguous(),
                       self.i32(np.arange(B + 1)), B, self.rows_seq, self.i32([p[-1] for p in self.prompts]), None,
                       0.0, 0, 0, self.acc, self.out, None, self.status, self.aws.buf, self.aws.nbytes)
        torch.cuda.synchronize()
        assert bool((self.status == 0).all())
        self.roots = [int(x) for x in self.out[:, 0].cpu()]
        log(f"{wl.name}: model + prefill of {self.ctx} tokens ready ({time.time() - t0:.1f} s); roots {self.roots}")

    def verify(self, seq_len, toks, off, bound):
        from paper_2608_08721_amd import lsv
        lsv.lsv_verify_block(self.cfg, self.dm.buf, self.kv.buf, self.cap, self.B, self.i32(seq_len), self.i32(toks),
                             self.i32(off), bound, self.cap, self.logits, self.status, self.ws.buf, self.ws.nbytes)

    def greedy_continuation(self, n):
        """The target's own greedy tokens after each root, [B, n], by n plain decoding steps of
        one row per sequence (their K/V go to the positions every verify block rewrites)."""
        import torch

        from paper_2608_08721_amd import lsv, runtime
        B = self.B
        cur, pos, cont = list(self.roots), list(self.ctx), []
        off = runtime.row_offsets_of([1] * B)
        for _ in range(n):
            self.verify(pos, cur, off, self.rows_buf)
            self.status.zero_()
            lsv.lsv_accept(lsv.LSV_ACC_GREEDY, B, self.m.vocab, self.logits, self.i32(off), B, 1, self.i32(cur),
                           None, 0.0, 0, 0, self.acc, self.out, None, self.status, self.aws.buf, self.aws.nbytes)
            torch.cuda.synchronize()
            assert bool((self.status == 0).all())
            cur = [int(x) for x in self.out[:, 0].cpu()]
            cont.append(cur)
            pos = [p + 1 for p in pos]
        return np.array(cont, dtype=np.int64).T

    def free(self):
        import torch
        for k in ("dm", "kv", "ws", "aws", "logits"):
            setattr(self, k, None)
        torch.cuda.empty_cache()


def counters_only(wl, args, dev):
    """Counter passes: the gate/up launches of eager verify steps at uniform gamma (no prefill: the
    cache holds zeros, which changes no projection's traffic), then a plain copy for calibration.
    Prints the roofline fields summarize() reads."""
    import torch

    from paper_2608_08721_amd import lsv, runtime
    from synth import gen
    m, B, G = wl.model, wl.batch, wl.G
    gammas = [int(x) for x in args.counters_only.split(",")]
    if not all(1 <= g <= G for g in gammas):
        raise SystemExit(f"--counters-only: every gamma must lie in [1, {G}]")
    cfg = runtime.model_config(m)
    ctx = [int(c) for c in gen.contexts(wl)]
    cap = runtime.kv_capacity(max(ctx) + G + 1)
    rows_step = B * (G + 1)
    dm = runtime.DeviceModel(cfg, dev)
    dm.pack_globals(gen.embed_weights(m, wl.seed), gen.final_norm_weights(m), gen.lm_head_weights(m, wl.seed))
    for l in range(m.n_layers):
        dm.pack_layer(l, gen.layer_weights(m, wl.seed, l))
    kv = runtime.KVCache(cfg, B, cap, dev)
    ws = runtime.Workspace(lsv.lsv_verify_workspace_bytes(cfg, B, rows_step, cap), dev)
    logits = torch.zeros((rows_step, m.vocab), dtype=torch.float32, device=dev)
    status = torch.zeros(B, dtype=torch.int32, device=dev)
    i32 = lambda x: torch.tensor(np.asarray(x, dtype=np.int32), device=dev)
    seq = i32(ctx)
    steps = args.roofline_steps
    for g in gammas:
        off = i32(runtime.row_offsets_of([g + 1] * B))
        toks = i32(gen.randint(wl.seed, 900, B * (g + 1), m.vocab))
        for _ in range(steps):
            lsv.lsv_verify_block(cfg, dm.buf, kv.buf, cap, B, seq, toks, off, rows_step, cap, logits, status, ws.buf,
                                 ws.nbytes)
    torch.cuda.synchronize()
    x = torch.empty(CALIB_BYTES, dtype=torch.uint8, device=dev)
    torch.empty_like(x).copy_(x)
    torch.cuda.synchronize()
    rows = [B * (g + 1) for g in gammas]
    print(json.dumps({"config": {"workload": wl.name, "counters_gammas": args.counters_only},
                      "roofline": {"rows": rows[0], "rows_list": rows, "launches_per_rows": steps * m.n_layers,
                                   "launches_timed": steps * m.n_layers * len(rows)}}), flush=True)


def measure(w, args, primary=True):
    """The measurement of one workload: per-gamma sweep (the measured cost table), selection,
    the timed select -> verify -> accept graph, the dominant kernel's events, and (primary
    workload only) the decode loop and the CPU baseline."""
    import torch

    from paper_2608_08721_amd import lsv, runtime
    from synth import drafter, gen
    wl, m, dev, i32 = w.wl, w.m, w.dev, w.i32
    seed, B, G, ctx, roots = w.seed, w.B, w.G, w.ctx, w.roots
    rows_step, rows_seq, cap = w.rows_step, w.rows_seq, w.cap
    cfg, dm, kv, ws, aws, logits, status, acc, out = (w.cfg, w.dm, w.kv, w.ws, w.aws, w.logits, w.status, w.acc,
                                                      w.out)
    mode_name = args.accept or ("greedy" if "greedy" in wl.accept else "sample")
    if mode_name not in wl.accept:
        raise SystemExit(f"workload {wl.name} has no {mode_name} acceptance")
    sampling = mode_name == "sample"
    conf_np = gen.confidences(wl)

    # drafts: planted (the target's own greedy token with probability equal to its confidence,
    # so realized acceptance follows the confidence model) or the configs' uniform random ids
    if sampling:
        # draft distributions q_v (a seeded softmax of N(0,1) logits per drafted position) and
        # drafts drawn from them; accept rows index q at (row offset - b + v - 1) < B * G
        q_np = gen.draft_probs(seed, B * G, m.vocab)
        qrng = np.random.default_rng(seed)
        drafts = np.array([[int(qrng.choice(m.vocab, p=q_np[b * G + v] / q_np[b * G + v].sum()))
                            for v in range(G)] for b in range(B)], dtype=np.int64)
        q_dev = torch.tensor(q_np, dtype=torch.float32, device=dev)
        acc_mode, acc_q, acc_T = lsv.LSV_ACC_SAMPLE, q_dev, float(wl.temperature)
        draft_kind = "drawn from the seeded draft distributions"
    elif args.drafts == "planted":
        t0 = time.time()
        cont = w.greedy_continuation(G)
        drafts = drafter.plant_block(cont, conf_np, seed, m.vocab)
        acc_mode, acc_q, acc_T = lsv.LSV_ACC_GREEDY, None, 0.0
        draft_kind = "planted: the target's greedy token with probability = its confidence"
        log(f"{wl.name}: greedy continuation of {G} tokens per sequence ({time.time() - t0:.1f} s)")
    else:
        drafts = gen.draft_ids(seed, B, G, m.vocab)
        acc_mode, acc_q, acc_T = lsv.LSV_ACC_GREEDY, None, 0.0
        draft_kind = "uniform random ids"

    def layout(gammas):
        """Verify rows [root_b, x_1..x_gamma_b] per sequence, concatenated."""
        return i32(np.concatenate([[roots[b]] + list(drafts[b][:gammas[b]]) for b in range(B)]))

    conf = torch.tensor(conf_np, device=dev)
    seq_base = i32(ctx)
    seq_work = i32(ctx)

    # ---- per-gamma latency sweep (graph of verify + accept per uniform gamma): the measured cost table
    sweep = {}
    for g in range(1, G + 1):
        ro = i32(runtime.row_offsets_of([g + 1] * B))
        tok_g = layout([g] * B)

        def body():
            seq_work.copy_(seq_base)
            lsv.lsv_verify_block(cfg, dm.buf, kv.buf, cap, B, seq_base, tok_g, ro, rows_step, cap, logits, status,
                                 ws.buf, ws.nbytes)
            lsv.lsv_accept(acc_mode, B, m.vocab, logits, ro, rows_step, rows_seq, tok_g, acc_q, acc_T, seed, 0,
                           acc, out, seq_work, status, aws.buf, aws.nbytes)
        body()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            body()
        for _ in range(3):
            graph.replay()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.sweep_reps + 1)]
        ev[0].record()
        for r in range(args.sweep_reps):
            graph.replay()
            ev[r + 1].record()
        torch.cuda.synchronize()
        lat = [ev[r].elapsed_time(ev[r + 1]) for r in range(args.sweep_reps)]
        sweep[g] = statistics.median(lat)
        del graph
    cost = np.array([0.0] + [sweep[g] for g in range(1, G + 1)], dtype=np.float64)
    log(f"{wl.name}: sweep (us): " + " ".join(f"{g}:{sweep[g] * 1e3:.0f}" for g in range(1, G + 1)))

    # ---- LibraSpec selection on the measured table (reported for all three rules); each
    # sequence selects on the uniform-gamma table of the batch
    cost_t = torch.tensor(cost, device=dev)
    gamma = torch.zeros(B, dtype=torch.int32, device=dev)
    aux = torch.zeros(B, dtype=torch.int32, device=dev)
    row_off = torch.zeros(B + 1, dtype=torch.int32, device=dev)
    n_alg1 = 8 if G <= 16 else 16
    chosen = {}
    for name, mode in (("exhaustive", lsv.LSV_SEL_EXHAUSTIVE), ("alg1", lsv.LSV_SEL_ALG1),
                       ("marginal", lsv.LSV_SEL_MARGINAL)):
        lsv.lsv_select_length(mode, B, G, conf, cost_t, 1, G, 2.2, n_alg1, 0, gamma, aux, row_off, status)
        torch.cuda.synchronize()
        chosen[name] = [int(x) for x in gamma.cpu()]
    g_marginal = chosen["marginal"]

    # ---- joint batched selection on a cost table over total drafts R (linear between the
    # uniform-gamma points R = B * gamma of the sweep), with its launch time
    cost_j = np.empty(B * G + 1)
    for R in range(B * G + 1):
        lo = max(1, min(R // B, G))
        hi = min(lo + 1, G)
        fr = 0.0 if lo == hi else max(0.0, (R - B * lo) / B)
        cost_j[R] = sweep[lo] * (1.0 - fr) + sweep[hi] * fr
    cost_jt = torch.tensor(cost_j, device=dev)
    g_joint = torch.zeros(B, dtype=torch.int32, device=dev)
    tot_joint = torch.zeros(1, dtype=torch.int32, device=dev)

    def joint():
        lsv.lsv_select_joint(B, G, conf, cost_jt, G, 0, g_joint, tot_joint, None, None)
    joint()
    torch.cuda.synchronize()
    chosen["joint"] = [int(x) for x in g_joint.cpu()]
    jg = torch.cuda.CUDAGraph()
    with torch.cuda.graph(jg):
        for _ in range(20):
            joint()
    jg.replay()
    torch.cuda.synchronize()
    ej0, ej1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ej0.record()
    jg.replay()
    ej1.record()
    torch.cuda.synchronize()
    joint_us = ej0.elapsed_time(ej1) * 1e3 / 20
    del jg
    joint_info = {"gamma": chosen["joint"], "total_drafts": int(tot_joint.cpu()[0]), "launch_us": round(joint_us, 2),
                  "predicted_tokens_per_ms": expected_tokens(conf_np, chosen["joint"]) / cost_j[sum(chosen["joint"])],
                  "predicted_tokens_per_ms_marginal": expected_tokens(conf_np, g_marginal) / cost_j[sum(g_marginal)]}
    # the timed step's rule: a single sequence takes MARGINAL on the per-gamma table; a batch takes the
    # joint rule, Eq. 2 over the batch's total drafts, because one step verifies all of the batch's rows
    # and its cost follows their total (the per-sequence rule prices each sequence as if the whole batch
    # had its length, and can pick a length that lengthens everyone's step)
    rule = "joint" if B > 1 else "marginal"
    g_star = chosen[rule]
    tokens = layout(g_star)
    log(f"{wl.name}: chosen gamma: {chosen}; timed step: {rule}")

    # ---- the timed step: select -> verify -> accept, one graph, dominant kernel bracketed by events
    n_slots = m.n_layers
    hev = HipEvents(2 * n_slots)

    def step():
        seq_work.copy_(seq_base)
        if B > 1:
            lsv.lsv_select_joint(B, G, conf, cost_jt, G, 0, gamma, tot_joint, row_off, status)
        else:
            lsv.lsv_select_length(lsv.LSV_SEL_MARGINAL, B, G, conf, cost_t, 1, G, 2.2, n_alg1, 0, gamma, aux,
                                  row_off, status)
        lsv.lsv_verify_block(cfg, dm.buf, kv.buf, cap, B, seq_base, tokens, row_off, rows_step, cap, logits, status,
                             ws.buf, ws.nbytes)
        lsv.lsv_accept(acc_mode, B, m.vocab, logits, row_off, rows_step, rows_seq, tokens, acc_q, acc_T, seed, 0,
                       acc, out, seq_work, status, aws.buf, aws.nbytes)
    step()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    steps, warmup = (args.steps, args.warmup) if primary else (args.secondary_steps, 3)
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record()
    for _ in range(steps):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms_step = e0.elapsed_time(e1) / steps
    del graph
    # dominant kernel: the same steps launched eagerly with HIP events recorded around every
    # gate/up launch on the step's stream (one launch per layer, several steps)
    lsv.lsv_set_timing_events(lsv.LSV_KERNEL_GATEUP, hev.ev, n_slots, 0)
    gateup_ms = []
    for _ in range(args.roofline_steps):
        # a bounded spin kernel first, so that the host has queued the whole step before the GPU
        # reaches it and each event pair brackets back-to-back execution, not launch latency
        torch.cuda._sleep(20_000_000)
        step()
        torch.cuda.synchronize()
        gateup_ms += [hev.elapsed_ms(2 * i, 2 * i + 1) for i in range(n_slots)]
    lsv.lsv_set_timing_events(lsv.LSV_KERNEL_GATEUP, [], 0, 0)
    assert bool((status == 0).all()) and [int(x) for x in gamma.cpu()] == g_star
    a_len = [int(x) for x in acc.cpu()]
    rows = sum(g + 1 for g in g_star)

    # dominant kernel: bytes and flops of one gate/up launch at this step's rows
    avg_gu = statistics.mean(gateup_ms)
    gu_bytes = gateup_bytes(m, rows)
    gu_flops = 2.0 * rows * 2 * m.d_ff * m.d_model
    t_gu = avg_gu * 1e-3
    hbm_gu, mfma_gu = gu_bytes / t_gu / 1e9 / HBM_PEAK_GBPS, gu_flops / t_gu / MFMA_PEAK_FLOPS
    bound = "mfma" if gu_flops / MFMA_PEAK_FLOPS > gu_bytes / (HBM_PEAK_GBPS * 1e9) else "hbm"
    if bound == "hbm":
        roof = {"bound": "hbm", "achieved": gu_bytes / t_gu / 1e9, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": hbm_gu, "traffic": measured_traffic(wl.name, rows)}
    else:
        roof = {"bound": "mfma", "achieved": gu_flops / t_gu / 1e12, "peak": MFMA_PEAK_FLOPS / 1e12, "unit": "TFLOP/s",
                "frac": mfma_gu, "traffic": None}
    roof.update({"kernel": "gemm gate/up + SwiGLU (one launch per layer)", "rows": rows, "bytes_per_launch": gu_bytes,
                 "flops_per_launch": gu_flops, "hbm_frac": hbm_gu, "mfma_frac": mfma_gu,
                 "avg_launch_us": avg_gu * 1e3, "launches_timed": len(gateup_ms),
                 "how": "HIP events around each gate/up launch in eagerly launched steps"})
    rows_per_seq = [g + 1 for g in g_star]
    sb = step_bytes(m, ctx, rows)
    sf = step_flops(m, ctx, rows_per_seq)
    if args.calib_copy and primary:
        x = torch.empty(CALIB_BYTES, dtype=torch.uint8, device=dev)
        y = torch.empty_like(x)
        y.copy_(x)
        torch.cuda.synchronize()
        del x, y

    # baseline length policy (the G4-style rule of the comparison experiments): the next
    # lengths from this step's outcome, and the rule's launch time (a graph of 100 launches)
    g_in = torch.tensor(g_star, dtype=torch.int32, device=dev)
    g_next = torch.zeros(B, dtype=torch.int32, device=dev)
    ro_next = torch.zeros(B + 1, dtype=torch.int32, device=dev) if B <= lsv.LSV_MAX_BATCH else None

    def g4():
        lsv.lsv_next_length_g4(B, g_in, acc, status, 1, G, g_next, ro_next, None)
    g4()
    torch.cuda.synchronize()
    g4_next = [int(x) for x in g_next.cpu()]
    g4_graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g4_graph):
        for _ in range(100):
            g4()
    g4_graph.replay()
    torch.cuda.synchronize()
    e2, e3 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e2.record()
    g4_graph.replay()
    e3.record()
    torch.cuda.synchronize()
    g4_us = e2.elapsed_time(e3) * 1e3 / 100
    del g4_graph

    exp_tok = expected_tokens(conf_np, g_star)
    realized = sum(a + 1 for a in a_len)
    one = (lambda v: v[0]) if B == 1 else (lambda v: v)
    per_gamma = {}
    for g in range(1, G + 1):
        t = sweep[g] * 1e-3
        per_gamma[str(g)] = {"latency_us": round(sweep[g] * 1e3, 2),
                             "tokens_per_s": round(expected_tokens(conf_np, [g] * B) / t, 2),
                             "hbm_frac": round(step_bytes(m, ctx, B * (g + 1)) / t / 1e9 / HBM_PEAK_GBPS, 4),
                             "mfma_frac": round(step_flops(m, ctx, [g + 1] * B) / t / MFMA_PEAK_FLOPS, 4)}
    result = {
        "metric": METRIC,
        "value": exp_tok / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if m.dtype == "bf16" else "f32",
        "data": f"synthetic (seeded random-init weights, random prompt ids; drafts {draft_kind})",
        "config": {"workload": wl.name, "model_shape": m.name, "batch": B, "context": one(ctx), "drafted": G,
                   "gamma": one(g_star), "rows": rows,
                   "selector": ("joint (Eq. 2 over the batch's total drafts)" if B > 1 else "marginal") + " on measured cost",
                   "accept": "greedy" if not sampling else f"sample T={wl.temperature}"},
        "value_is": "expected emitted tokens per second of the step: sum_b (1 + N_b(gamma_b)) / step latency, "
                    "N_b from the drafter confidences (Eq. 2's numerator, Assumption 3.7)",
        "roofline": roof,
        "step": {"latency_us": ms_step * 1e3, "wall_ms_per_step": t_wall / steps * 1e3,
                 "algorithmic_bytes": sb, "hbm_frac": sb / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                 "flops": sf, "mfma_frac": sf / (ms_step * 1e-3) / MFMA_PEAK_FLOPS,
                 "expected_tokens": exp_tok, "expected_tokens_per_s": exp_tok / (ms_step * 1e-3),
                 "realized_tokens": realized, "realized_tokens_per_s": realized / (ms_step * 1e-3),
                 "accept_len": one(a_len), "verified_rows_per_s": rows / (ms_step * 1e-3)},
        "selection": {k: one(v) for k, v in chosen.items()},
        "per_gamma": per_gamma,
        "joint_selection": joint_info,
        "baseline_policies": {"static": "the sweep: one gamma for every sequence and round",
                              "g4_next_gamma": one(g4_next), "g4_launch_us": round(g4_us, 2)},
    }
    if B > 1:
        # every sequence at the largest gamma: the batched regime the matrix cores serve
        rows_g = B * (G + 1)
        t_g = sweep[G] * 1e-3
        result["uniform_gamma_max"] = {"gamma": G, "rows": rows_g, "latency_us": sweep[G] * 1e3,
                                       "mfma_frac": step_flops(m, ctx, [G + 1] * B) / t_g / MFMA_PEAK_FLOPS,
                                       "hbm_frac": step_bytes(m, ctx, rows_g) / t_g / 1e9 / HBM_PEAK_GBPS}
    if primary:
        result["length_rules"] = length_rules(wl, cost, dev)
    if primary and args.rounds > 0:
        log(f"decode loop: {args.rounds} rounds per length policy")
        try:
            result["decode_loop"] = decode_loop_measure(m, cfg, dm, B, G, ctx, w.prompts, w.pre, w.rows_buf, roots,
                                                        cost, cost_j, seed, args.rounds, dev)
        except Exception as e:  # reported in the line; the verify-step measurement above stands
            log(f"decode loop failed: {e!r}")
            result["decode_loop"] = {"error": repr(e)}
    if primary and not args.no_cpu_baseline:
        log("cpu baseline: timing the oracle on a bounded sample")
        toks_np = np.concatenate([[roots[b]] + list(drafts[b][:g_star[b]]) for b in range(B)])
        result["cpu_baseline"] = cpu_baseline(m, seed, ctx, rows_per_seq, toks_np, exp_tok)
    return result


def main():
    args = parse()
    if args.summarize:
        sys.stdout.write(summarize(*args.summarize))
        return
    if args.summarize_counters:
        sys.stdout.write(summarize_counters(args.summarize_counters[0], args.summarize_counters[1:]))
        return
    if args.summarize_mfma:
        sys.stdout.write(summarize_mfma(*args.summarize_mfma))
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: this build has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)
    import torch

    from synth import configs
    torch.cuda.set_device(0)
    if args.counters_only:
        counters_only(configs.WORKLOADS[args.workload], args, "cuda")
        return
    w = Workload(configs.WORKLOADS[args.workload], "cuda")
    result = measure(w, args, primary=True)
    w.free()
    del w
    others = {}
    for name in ([] if args.secondary == "none" else args.secondary.split(",")):
        log(f"secondary workload {name}")
        w2 = Workload(configs.WORKLOADS[name], "cuda")
        r2 = measure(w2, args, primary=False)
        w2.free()
        del w2
        others[name] = {k: r2[k] for k in ("value", "unit", "ms_per_step", "config", "roofline", "step", "selection",
                                           "per_gamma")}
    if others:
        result["other_workloads"] = others
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
