#!/usr/bin/env python3
"""Benchmark of the CDSL lookahead step on one MI355X.

A step = draft rollout + target verification + reward + beam selection +
commit over the whole batch, on the seeded synthetic workload (random-init
Llama-style decoders, uniform-random prompts).  Prints ONE JSON line:
lookahead tokens verified per second (B * k * d per step), CDSL steps per
second, the roofline of the dominant kernel class and the CPU oracle timed
on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_MFMA_BF16_TFS = 2500.0    # dense bf16 MFMA
PEAK_FP32_TFS = 157.3          # fp32 vector


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="7b1b")
    ap.add_argument("--batch", type=int, default=None)
    ap.add_argument("--k", type=int, default=None)
    ap.add_argument("--d", type=int, default=None)
    ap.add_argument("--profile-steps", type=int, default=3)
    ap.add_argument("--phase-steps", type=int, default=3)
    ap.add_argument("--methods-steps", type=int, default=3,
                    help="iterations timed per decoding method in the 'methods' comparison (0: skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 256 MiB device copy (reference for HBM byte counters)")
    ap.add_argument("--summarize-profile", nargs="+",
                    metavar="BENCH_JSON TRACE_DIR FETCH_DIR WRITE_DIR [UTIL_DIR]",
                    help="write a markdown summary of rocprofv3 runs of this script (kernel trace, FETCH_SIZE and "
                         "WRITE_SIZE passes with --calibrate-copy, optionally a MfmaUtil/LdsUtil pass) and exit; "
                         "no GPU needed")
    ap.add_argument("--grid", default=None, metavar="K1,K2,..:D1,D2,..",
                    help="measure every (k, d) point of the grid on one engine (a fresh prefill per point) and "
                         "print one JSON line with a row per point instead of the bench line")
    ap.add_argument("--summarize-ranges", default=None, metavar="TRACE_DIR",
                    help="markdown summary of a rocprofv3 --kernel-trace --marker-trace --hip-runtime-trace run "
                         "of this script: per library call (roctx range), its calls, host time, kernels launched "
                         "and their GPU time; no GPU needed")
    ap.add_argument("--summarize-trace", nargs=2, default=None, metavar=("BENCH_JSON", "TRACE_DIR"),
                    help="markdown summary of a rocprofv3 --kernel-trace --stats run of this script on any "
                         "workload: top kernels, and one step's launches by kernel and grid; no GPU needed")
    ap.add_argument("--summary-out", default=None)
    ap.add_argument("--commands", default=None, help="text file with the exact profiling commands (for the summary)")
    return ap.parse_args()


# Kernel (rocprofv3 name pattern) and source files behind each timed class.
CLASS_KERNEL = {
    "gemm_dense": (r"gemm_bf16_dense<[^>]*, 0>\(", ["gemm.hip", "gemm.h", "common.h"]),
    "gemm_skinny": (r"gemm_bf16_skinny<", ["gemm.hip", "gemm.h", "common.h"]),
    "attention": (r"attn_split<", ["attention.hip", "attention.h", "common.h"]),
    "attn_combine": (r"attn_combine<", ["attention.hip", "attention.h", "common.h"]),
    "splitk_reduce": (r"splitk_reduce_kernel", ["gemm.hip", "gemm.h", "common.h"]),
}
TRAFFIC_TAG = "<!-- traffic "
# Kernels whose HBM rate the profile summary reports against the peak: the
# decode (rollout) and verification attention, and the rollout projections
# by shape family.
HBM_RATE_KERNELS = [
    ("rollout attention (draft, hd 64, key groups)", r"attn_split<64, "),
    ("verification attention (target, hd 128)", r"attn_split<128, "),
    ("rollout projections, 16 columns per wave, ring 8 (gate/up)", r"gemm_bf16_skinny<\d+, 1, 8, "),
    ("rollout projections, 16 columns per wave, ring 4 (q/k/v, o, down)", r"gemm_bf16_skinny<\d+, 1, 4, "),
    ("rollout LM head, 32 columns per wave", r"gemm_bf16_skinny<\d+, 2, 4, "),
]


def source_digest(files):
    """Digest of a kernel's source files with comments, blank lines and
    indentation left out, so that an edit of the comments alone keeps the
    counters taken for the code."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2412_10418_amd", "csrc", f)) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        code = "\n".join(ln.strip() for ln in text.splitlines() if ln.strip())
        h.update(code.encode())
    return h.hexdigest()[:16]


def stored_traffic(cls, workload):
    """HBM bytes per launch of the class's kernel from a committed rocprofv3
    counter summary, or None when there is none for this workload or the
    kernel's sources changed since the counters were taken."""
    if cls not in CLASS_KERNEL:
        return None
    d = os.path.join(ROOT, "profiles")
    if not os.path.isdir(d):
        return None
    digest = source_digest(CLASS_KERNEL[cls][1])
    for fn in sorted(os.listdir(d)):
        if not fn.endswith(".md"):
            continue
        with open(os.path.join(d, fn)) as fh:
            for line in fh:
                if line.startswith(TRAFFIC_TAG):
                    rec = json.loads(line[len(TRAFFIC_TAG):].rstrip().rstrip("->").strip())
                    if rec.get("class") == cls and rec.get("workload") == workload and rec.get("source") == digest:
                        return rec
    return None


def roofline(stats, workload):
    """Dominant kernel class of the instrumented steps and its roofline."""
    best = max(stats, key=lambda nm: stats[nm]["ms"])
    st = stats[best]
    sec = st["ms"] / 1e3
    n = max(1, st["launches"])
    per_launch_ms = st["ms"] / n
    tr = stored_traffic(best, workload)
    extra = {"kernel": best, "avg_launch_us": round(per_launch_ms * 1e3, 2), "launches": st["launches"],
             "alg_bytes_per_launch": round(st["bytes"] / n), "traffic_unit": "HBM bytes per launch",
             "traffic_source": tr["file"] if tr else None}
    traffic = tr["bytes_per_launch"] if tr else None
    if best in ("gemm_dense",):
        ach = st["flops"] / sec / 1e12
        # the executed MFMA work is twice the algorithmic flops (the hi and
        # lo products of the fp32 activations)
        return best, {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_MFMA_BF16_TFS, "unit": "TFLOP/s",
                      "frac": round(ach / PEAK_MFMA_BF16_TFS, 4), "traffic": traffic,
                      "alg_flops_per_launch": round(st["flops"] / n),
                      "executed_frac": round(2.0 * ach / PEAK_MFMA_BF16_TFS, 4), **extra}
    ach = st["bytes"] / sec / 1e9
    return best, {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                  "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": traffic, **extra}


def mangled_short(nm):
    """The function name of an Itanium-mangled kernel name the tracer left
    mangled ("_ZN4cdsl12_GLOBAL__N_110embed_rowsI..." -> "embed_rows<...>")."""
    i, last = (3 if nm.startswith("_ZN") else 2), nm
    while i < len(nm) and nm[i].isdigit():
        j = i
        while j < len(nm) and nm[j].isdigit():
            j += 1
        n = int(nm[i:j])
        last, i = nm[j:j + n], j + n
    return last + ("<...>" if i < len(nm) and nm[i] == "I" else "")


def summarize_profile(args):
    """Markdown summary of the three rocprofv3 runs of this script."""
    import csv
    import re
    if len(args.summarize_profile) not in (4, 5):
        raise SystemExit("--summarize-profile takes BENCH_JSON TRACE_DIR FETCH_DIR WRITE_DIR [UTIL_DIR]")
    bench_json, trace_dir, fetch_dir, write_dir = args.summarize_profile[:4]
    util_dir = args.summarize_profile[4] if len(args.summarize_profile) == 5 else None
    with open(bench_json) as fh:
        line = [ln for ln in fh.read().splitlines() if ln.startswith("{")][-1]
    b = json.loads(line)
    wl = b["config"]["workload"]
    stats = list(csv.DictReader(open(os.path.join(trace_dir, "bench_kernel_stats.csv"))))
    total = sum(float(r["TotalDurationNs"]) for r in stats)

    def counters(dn):
        rows = list(csv.DictReader(open(os.path.join(dn, "bench_counter_collection.csv"))))
        return rows

    fetch, write = counters(fetch_dir), counters(write_dir)
    copy_bytes_kib = 262144.0

    def copy_scale(rows):
        # the last three dispatches are the 256 MiB calibration copies
        cal = [float(r["Counter_Value"]) for r in rows[-3:] if "copyBuffer" in r["Kernel_Name"]]
        if len(cal) != 3:
            raise SystemExit("calibration copies not found at the end of the counter run")
        return copy_bytes_kib / (sum(cal) / 3), sum(cal) / 3

    fs, fcal = copy_scale(fetch)
    ws, wcal = copy_scale(write)
    out = [f"# rocprofv3 summary: CDSL step, workload {wl}", ""]
    if args.commands:
        out += ["Commands (run from the repository root on one MI355X):", "", "```"]
        out += [ln.rstrip() for ln in open(args.commands) if ln.strip()]
        out += ["```", ""]
    out += [f"Bench line of the traced run: {b['ms_per_step']} ms/step, {b['value']} {b['unit']} "
            f"(B={b['config']['batch']}, k={b['config']['k']}, d={b['config']['d']}).", "",
            "## Kernel trace (--kernel-trace --stats), top kernels by total time", "",
            "| kernel | calls | total ms | avg us | share |", "|---|---:|---:|---:|---:|"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"]))[:16]:
        nm = r["Name"]
        nm = nm.replace("cdsl::(anonymous namespace)::", "").replace("cdsl::", "")
        nm = nm.split("(")[0] if not nm.startswith("_Z") else mangled_short(nm)
        out.append(f"| `{nm[:80]}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.2f} | "
                   f"{float(r['AverageNs']) / 1e3:.2f} | {100 * float(r['TotalDurationNs']) / total:.1f}% |")
    out += ["", "Calls include the prompt prefill (separately named `gemm_bf16_dense<..., 1>`) and the warmup, "
            "timed and instrumented steps.", ""]
    trace_csv = os.path.join(trace_dir, "bench_kernel_trace.csv")
    if os.path.exists(trace_csv):
        # one timed step: the launches between two commits in the middle of
        # the run (the instrumented steps at the end carry timing events)
        tr = sorted(csv.DictReader(open(trace_csv)), key=lambda r: int(r["Start_Timestamp"]))
        cut = [i for i, r in enumerate(tr) if "commit_kernel" in r["Kernel_Name"]]
        if len(cut) >= 4:
            u = len(cut) // 2
            seg = tr[cut[u - 1] + 1:cut[u] + 1]
            ksum = sum(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in seg) / 1e6
            wall = (int(seg[-1]["End_Timestamp"]) - int(seg[0]["Start_Timestamp"])) / 1e6
            gaps = sorted(int(seg[i + 1]["Start_Timestamp"]) - int(seg[i]["End_Timestamp"])
                          for i in range(len(seg) - 1))
            fam = {}
            for r in seg:
                nm = r["Kernel_Name"].replace("cdsl::(anonymous namespace)::", "").replace("cdsl::", "")
                nm = "embed_rows" if "embed_rows" in nm else re.sub(r"[<(].*$", "", nm.replace("void ", ""))
                fam[nm] = fam.get(nm, 0) + 1
            top = ", ".join(f"{k} {v}" for k, v in sorted(fam.items(), key=lambda kv: -kv[1])[:8])
            out += ["## Launches per step", "",
                    f"One timed step of the traced run (between two commits): {len(seg)} launches, "
                    f"{ksum:.2f} ms of kernel time in {wall:.2f} ms; median gap between kernels "
                    f"{gaps[len(gaps) // 2] / 1e3:.2f} us. By kernel: {top}.", ""]
    out += [
            "## HBM traffic (FETCH_SIZE and WRITE_SIZE passes)", "",
            f"Calibration: a plain 256 MiB device copy (262144 KiB read, 262144 KiB written) reads "
            f"FETCH_SIZE = {fcal:.1f} KiB and WRITE_SIZE = {wcal:.1f} KiB per dispatch, so the counters are "
            f"scaled by {fs:.4f} (fetch) and {ws:.4f} (write).", "",
            "| class | kernel | dispatches | FETCH KiB | WRITE KiB | HBM MB per launch (scaled) | "
            "bench alg. MB per launch | rocprof avg us | bench avg us |",
            "|---|---|---:|---:|---:|---:|---:|---:|---:|"]
    recs = []
    for cls, (pat, files) in CLASS_KERNEL.items():
        rx = re.compile(pat)
        fv = [float(r["Counter_Value"]) for r in fetch if rx.search(r["Kernel_Name"])]
        wv = [float(r["Counter_Value"]) for r in write if rx.search(r["Kernel_Name"])]
        tv = [r for r in stats if rx.search(r["Name"])]
        if not fv or not wv or not tv:
            continue
        calls = sum(int(r["Calls"]) for r in tv)
        avg_us = sum(float(r["TotalDurationNs"]) for r in tv) / calls / 1e3
        f_kib, w_kib = sum(fv) / len(fv), sum(wv) / len(wv)
        bpl = (f_kib * fs + w_kib * ws) * 1024.0
        kb = b.get("kernels", {}).get(cls, {})
        alg = b["roofline"].get("alg_bytes_per_launch") if b["roofline"].get("kernel") == cls else None
        out.append(f"| {cls} | `{pat}` | {len(fv)} | {f_kib:.0f} | {w_kib:.0f} | {bpl / 1e6:.1f} | "
                   f"{alg / 1e6 if alg else float('nan'):.1f} | {avg_us:.2f} | {kb.get('avg_launch_us', float('nan'))} |")
        recs.append({"class": cls, "workload": wl, "source": source_digest(files),
                     "file": os.path.basename(args.summary_out or "summary.md"),
                     "fetch_kib_per_dispatch": round(f_kib, 1), "write_kib_per_dispatch": round(w_kib, 1),
                     "fetch_scale": round(fs, 4), "write_scale": round(ws, 4),
                     "bytes_per_launch": round(bpl), "rocprof_avg_us": round(avg_us, 2)})
    out += ["", "The bench times each class with HIP events around its launches on the library stream; "
            "its average per launch is expected to agree with the rocprofv3 average of the same kernel.", ""]
    out += ["## HBM rate of the memory-bound kernels", "",
            "Measured bytes per dispatch (FETCH_SIZE + WRITE_SIZE, scaled as above) over the rocprofv3 average "
            f"duration, against the {PEAK_HBM_GBS:.0f} GB/s peak.", "",
            "| kernel | pattern | dispatches | HBM MB per launch | rocprof avg us | GB/s | % of peak |",
            "|---|---|---:|---:|---:|---:|---:|"]
    for label, pat in HBM_RATE_KERNELS:
        rx = re.compile(pat)
        fv = [float(r["Counter_Value"]) for r in fetch if rx.search(r["Kernel_Name"])]
        wv = [float(r["Counter_Value"]) for r in write if rx.search(r["Kernel_Name"])]
        tv = [r for r in stats if rx.search(r["Name"])]
        if not fv or not wv or not tv:
            continue
        avg_us = sum(float(r["TotalDurationNs"]) for r in tv) / sum(int(r["Calls"]) for r in tv) / 1e3
        bpl = (sum(fv) / len(fv) * fs + sum(wv) / len(wv) * ws) * 1024.0
        gbs = bpl / (avg_us * 1e-6) / 1e9
        out.append(f"| {label} | `{pat}` | {len(fv)} | {bpl / 1e6:.2f} | {avg_us:.2f} | {gbs:.0f} | "
                   f"{100 * gbs / PEAK_HBM_GBS:.1f}% |")
    out.append("")
    if util_dir:
        util = counters(util_dir)
        out += ["## Matrix-core and LDS utilisation (MfmaUtil / LdsUtil pass)", "",
                "Per-dispatch averages of rocprofv3's derived metrics (percent of the active time of the CUs "
                "that ran the kernel).", "",
                "| class | kernel | dispatches | MfmaUtil % | LdsUtil % |", "|---|---|---:|---:|---:|"]
        for cls, (pat, _files) in CLASS_KERNEL.items():
            rx = re.compile(pat)
            mv = [float(r["Counter_Value"]) for r in util
                  if rx.search(r["Kernel_Name"]) and r["Counter_Name"] == "MfmaUtil"]
            lv = [float(r["Counter_Value"]) for r in util
                  if rx.search(r["Kernel_Name"]) and r["Counter_Name"] == "LdsUtil"]
            if mv:
                out.append(f"| {cls} | `{pat}` | {len(mv)} | {sum(mv) / len(mv):.1f} | "
                           f"{sum(lv) / len(lv) if lv else float('nan'):.1f} |")
        out.append("")
    out += [TRAFFIC_TAG + json.dumps(r) + " -->" for r in recs]
    text = "\n".join(out) + "\n"
    if args.summary_out:
        with open(args.summary_out, "w") as fh:
            fh.write(text)
    else:
        sys.stdout.write(text)


def summarize_trace(args):
    """Top kernels of a traced bench run, and the launches of one step (the
    last step between two commits before the instrumented steps) grouped by
    kernel and grid."""
    import csv
    import glob
    import re
    bench_json, d = args.summarize_trace

    def one(pattern):
        fs = glob.glob(os.path.join(d, pattern))
        if not fs:
            raise SystemExit(f"no {pattern} in {d}")
        return list(csv.DictReader(open(fs[0])))

    def short(nm):
        nm = nm.replace("cdsl::(anonymous namespace)::", "").replace("cdsl::", "")
        return mangled_short(nm) if nm.startswith("_Z") else re.sub(r"\(.*$", "", nm)

    with open(bench_json) as fh:
        b = json.loads([ln for ln in fh.read().splitlines() if ln.startswith("{")][-1])
    cfg = b["config"]
    stats = sorted(one("*_kernel_stats.csv"), key=lambda r: -float(r["TotalDurationNs"]))
    tot = sum(float(r["TotalDurationNs"]) for r in stats)
    out = [f"# rocprofv3 summary: CDSL step, workload {cfg['workload']} (batch {cfg['batch']}, k = {cfg['k']}, "
           f"d = {cfg['d']})", ""]
    if args.commands:
        out += ["Commands (run from /tmp with TMPDIR=/tmp on one MI355X; R = repository root):", "", "```"]
        out += [ln.rstrip() for ln in open(args.commands) if ln.strip()]
        out += ["```", ""]
    out += [f"Bench line of the traced run: {b['ms_per_step']} ms/step, {b['value']:.0f} {b['unit']}.", "",
            "| kernel | calls | total ms | avg us | share |", "|---|---:|---:|---:|---:|"]
    for r in stats[:16]:
        out.append(f"| `{short(r['Name'])}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.2f} | "
                   f"{float(r['AverageNs']) / 1e3:.2f} | {100 * float(r['TotalDurationNs']) / tot:.1f}% |")
    out += ["", "Calls cover the prompt prefill and every warmup, timed, phase-timed and instrumented step.", ""]
    tr = sorted(one("*_kernel_trace.csv"), key=lambda r: int(r["Start_Timestamp"]))
    idx = [i for i, r in enumerate(tr) if "commit_kernel" in r["Kernel_Name"]]
    if len(idx) >= 3:
        a, z = idx[-3] + 1, idx[-2] + 1
        agg = {}
        for r in tr[a:z]:
            g = (f"{int(r['Grid_Size_X']) // int(r['Workgroup_Size_X'])}x{r['Grid_Size_Y']}x{r['Grid_Size_Z']}")
            v = agg.setdefault((short(r["Kernel_Name"]), g), [0, 0.0])
            v[0] += 1
            v[1] += (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        ks = sum(v[1] for v in agg.values()) / 1e3
        wall = (int(tr[z - 1]["End_Timestamp"]) - int(tr[a]["Start_Timestamp"])) / 1e6
        out += [f"One step of the traced run (between two commits): {z - a} launches, {ks:.1f} ms of kernel time "
                f"in {wall:.1f} ms. By kernel and grid (workgroups x y x z):", "",
                "| kernel | grid | launches | ms | avg us |", "|---|---|---:|---:|---:|"]
        for (nm, g), (c, t) in sorted(agg.items(), key=lambda kv: -kv[1][1])[:16]:
            out.append(f"| `{nm}` | {g} | {c} | {t / 1e3:.2f} | {t / c:.1f} |")
    text = "\n".join(out) + "\n"
    if args.summary_out:
        with open(args.summary_out, "w") as fh:
            fh.write(text)
    else:
        sys.stdout.write(text)


def summarize_ranges(args):
    """Per roctx range (one library call): calls, host time, and the kernels
    whose launch API call started inside the range on the same thread, with
    their GPU time (from the kernel trace, matched by correlation id)."""
    import csv
    import glob
    d = args.summarize_ranges

    def one(pattern):
        fs = glob.glob(os.path.join(d, pattern))
        if not fs:
            raise SystemExit(f"no {pattern} in {d}")
        return list(csv.DictReader(open(fs[0])))

    marks, hip, kern = one("*_marker_api_trace.csv"), one("*_hip_api_trace.csv"), one("*_kernel_trace.csv")
    gpu_ns = {r["Correlation_Id"]: int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in kern}
    launches = sorted((int(r["Start_Timestamp"]), r["Thread_Id"], r["Correlation_Id"]) for r in hip
                      if r["Correlation_Id"] in gpu_ns)
    starts = [t for t, _, _ in launches]
    import bisect
    agg = {}
    for m in marks:
        t0, t1, th = int(m["Start_Timestamp"]), int(m["End_Timestamp"]), m["Thread_Id"]
        lo, hi = bisect.bisect_left(starts, t0), bisect.bisect_right(starts, t1)
        ks = [cid for t, tid, cid in launches[lo:hi] if tid == th]
        a = agg.setdefault(m["Function"], [0, 0, 0, 0])
        a[0] += 1
        a[1] += t1 - t0
        a[2] += len(ks)
        a[3] += sum(gpu_ns[c] for c in ks)
    out = ["| library call | calls | host ms per call | kernels per call | GPU ms per call |",
           "|---|---:|---:|---:|---:|"]
    for nm, (n, host, nk, g) in sorted(agg.items(), key=lambda kv: -kv[1][3]):
        out.append(f"| `{nm}` | {n} | {host / n / 1e6:.3f} | {nk / n:.1f} | {g / n / 1e6:.3f} |")
    text = "\n".join(out) + "\n"
    if args.summary_out:
        with open(args.summary_out, "w") as fh:
            fh.write(text)
    else:
        sys.stdout.write(text)


def phase_rooflines(wl, B, k, d, ms, sum_prefix):
    """Algorithmic rates of the rollout (HBM-bound: every draft forward
    streams the draft weights and the prefix KV of every prompt once) and of
    the verification (MFMA-bound: 2 M flops per weight, M = B k d rows).
    The rollout's algorithmic bytes count the KV at bf16 width (2 bytes per
    element, the layout the scope table prices); the library stores each KV
    value as a bf16 hi + lo pair, so the bytes it actually streams count 4
    (``rollout_stored_*``).  The verification's executed MFMA work is twice
    its algorithmic flops (hi and lo products)."""
    dr, tg = wl.draft, wl.target
    kv_tok = lambda m, w: m.n_layers * 2 * m.n_kv_heads * m.head_dim * w   # K + V of one token
    wbytes = dr.n_params(with_embeddings=False) * 2.0
    ro_bytes = d * (wbytes + sum_prefix * kv_tok(dr, 2.0))
    ro_stored = d * (wbytes + sum_prefix * kv_tok(dr, 4.0))
    ve_flops = 2.0 * B * k * d * tg.n_params(with_embeddings=False)
    out = {"rollout_ms": round(ms["rollout"], 3), "verify_ms": round(ms["verify"], 3),
           "tail_ms": round(ms["tail"], 3)}
    if ms["rollout"] > 0:
        sec = ms["rollout"] * 1e-3
        gbs = ro_bytes / sec / 1e9
        out.update({"rollout_GB_per_s": round(gbs, 1), "rollout_hbm_frac": round(gbs / PEAK_HBM_GBS, 4),
                    "rollout_bytes": round(ro_bytes),
                    "rollout_stored_GB_per_s": round(ro_stored / sec / 1e9, 1),
                    "rollout_stored_hbm_frac": round(ro_stored / sec / 1e9 / PEAK_HBM_GBS, 4),
                    "rollout_stored_bytes": round(ro_stored)})
    if ms["verify"] > 0:
        tfs = ve_flops / (ms["verify"] * 1e-3) / 1e12
        out.update({"verify_TFLOP_per_s": round(tfs, 1), "verify_mfma_frac": round(tfs / PEAK_MFMA_BF16_TFS, 4),
                    "verify_gemm_flops": round(ve_flops),
                    "verify_executed_mfma_frac": round(2.0 * tfs / PEAK_MFMA_BF16_TFS, 4)})
    return out


def class_table(stats, step_ms_total):
    out = {}
    for nm, st in stats.items():
        if st["launches"] == 0:
            continue
        sec = st["ms"] / 1e3
        row = {"launches": st["launches"], "ms": round(st["ms"], 3),
               "share": round(st["ms"] / step_ms_total, 4) if step_ms_total else None,
               "avg_launch_us": round(st["ms"] * 1e3 / st["launches"], 2)}
        if sec > 0:
            row["GB/s"] = round(st["bytes"] / sec / 1e9, 1)
            row["hbm_frac"] = round(st["bytes"] / sec / 1e9 / PEAK_HBM_GBS, 4)
            if st["flops"] > 0:
                row["TFLOP/s"] = round(st["flops"] / sec / 1e12, 2)
                row["mfma_frac"] = round(st["flops"] / sec / 1e12 / PEAK_MFMA_BF16_TFS, 4)
        out[nm] = row
    return out


def cpu_baseline(wl, dw, tw, prompt, kws, rw, k, d, min_s=10.0, max_steps=8):
    """The float64 oracle on one prompt of the workload: prefill (untimed),
    then whole CDSL steps (beam heads, rollout of all k beams, tree
    verification, reward, selection, commit) until at least ``min_s`` seconds
    of timed work; rate = k * d * steps / time."""
    import oracle
    threads = os.environ.get("OMP_NUM_THREADS") or str(os.cpu_count())
    od, ot = oracle.Decoder(wl.draft, dw), oracle.Decoder(wl.target, tw)
    t0 = time.perf_counter()
    st = oracle.prefill(od, ot, prompt)
    t_prefill = time.perf_counter() - t0
    log(f"cpu baseline: oracle prefill {t_prefill:.1f}s")
    n, t_steps = 0, 0.0
    while n < max_steps and t_steps < min_s:
        t0 = time.perf_counter()
        res = oracle.step(od, ot, st, k, d, wl.alpha, wl.reward, kws, rw)
        t_steps += time.perf_counter() - t0
        st = res.state
        n += 1
        log(f"cpu baseline: step {n} {t_steps:.1f}s")
    return {"value": round(k * d * n / t_steps, 4), "unit": "lookahead tokens verified/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"1 prompt of workload '{wl.name}' (prompt {len(prompt)} tokens, k={k}, d={d}) in float64: "
                       f"{n} whole CDSL steps in {t_steps:.1f}s; prompt prefill {t_prefill:.1f}s untimed"),
            "s_per_prompt_step": round(t_steps / n, 3)}


# the controller's thresholds in the methods comparison: the paper's
# CommonGen setting for most (draft, target) pairs (d = 3 there; here the
# workload's d), with the concept-coverage reward
METHOD_A_T, METHOD_R_T, METHOD_B = 0.3, 0.3, 1


def measure_methods(eng, wl, prompts, k, d, steps):
    """Wall-clock of the paper's decoding methods on the same models and
    prompts, with the concept-coverage reward (4 seeded concepts per prompt):
    the CDSL step (the timed path above, here with that reward), the same
    step with speculative sampling's soft rejection, one iteration of Alg. 1
    (d tokens drafted from the prefix, the states S1..S4) with hard and with
    soft rejection, and one token of CDLH-appx. (draft lookaheads) and of
    CDLH (target lookaheads).  Each method starts
    from a fresh prefill, runs one untimed iteration, then `steps` timed
    ones.  Tokens per iteration depend on how often the target accepts the
    draft's tokens, which for independent random models is rarely."""
    import numpy as np
    import torch
    import cdsl_inputs as ci
    B = prompts.shape[0]
    kws = torch.from_numpy(ci.keywords(wl.seed, B, 4, wl.target.vocab)).cuda()
    p = torch.from_numpy(prompts).cuda()
    # seeded uniforms of speculative sampling, resident before timing
    U = [(torch.from_numpy(ci.uniforms(wl.seed, 0, t, B, k, d)).cuda(),
          torch.from_numpy(ci.uniforms(wl.seed, 1, t, B, k, d)).cuda()) for t in range(steps + 1)]
    U1 = [torch.from_numpy(np.ascontiguousarray(ci.uniforms(wl.seed, 0, t, B, 1, d)[:, 0])).cuda()
          for t in range(steps + 1)]
    it = [0]

    def soft_step(st):
        u, v = U[it[0] % len(U)]
        it[0] += 1
        return eng.step(st, keywords=kws, k=k, d=d, alpha=math.inf, reward="keyword_coverage", u=u, v=v)

    def alg1_soft(st):
        u = U1[it[0] % len(U1)]
        it[0] += 1
        return eng.controller_step(st, kws, METHOD_A_T, METHOD_R_T, METHOD_B, k=k, d=d, normalize=True, u=u)

    runs = {
        "cdsl_step": lambda st: eng.step(st, keywords=kws, k=k, d=d, alpha=math.inf, reward="keyword_coverage"),
        "cdsl_step_soft": soft_step,
        "alg1": lambda st: eng.controller_step(st, kws, METHOD_A_T, METHOD_R_T, METHOD_B, k=k, d=d, normalize=True),
        "alg1_soft": alg1_soft,
        "cdlh_appx": lambda st: eng.head_step(st, kws, 0, k=k, d=d, normalize=True),
        "cdlh": lambda st: eng.head_step(st, kws, 1, k=k, d=d, normalize=True),
    }
    out = {}
    for name, fn in runs.items():
        it[0] = 0
        st = eng.start(p, k=k)
        fn(st)
        torch.cuda.synchronize()
        before = sum(len(e) for e in st.emitted)
        t0 = time.perf_counter()
        for _ in range(steps):
            fn(st)
        torch.cuda.synchronize()
        sec = time.perf_counter() - t0
        toks = sum(len(e) for e in st.emitted) - before
        out[name] = {"ms_per_iteration": round(sec * 1e3 / steps, 2),
                     "tokens_per_iteration_per_prompt": round(toks / (steps * B), 3),
                     "tokens_per_s": round(toks / sec, 1)}
        st.prefix.free()
    base = out["cdlh"]["tokens_per_s"]
    for name in out:
        out[name]["speedup_vs_cdlh"] = round(out[name]["tokens_per_s"] / base, 2) if base > 0 else None
    out["settings"] = {"reward": "keyword_coverage, 4 concepts per prompt", "k": k, "d": d,
                       "a_t": METHOD_A_T, "r_t": METHOD_R_T, "b": METHOD_B, "timed_iterations": steps}
    return out


def measure_grid(eng, wl, prompts, kw_t, rw_t, points, steps, warmup):
    """Steps per second and lookahead tokens verified per second at each
    (k, d) point, with the rollout / verification split (median over the
    timed steps) and their algorithmic rates."""
    import numpy as np
    import torch
    B = prompts.shape[0]
    rows = []
    for k, d in points:
        st = eng.start(torch.from_numpy(prompts).cuda(), k=k)
        for _ in range(warmup):
            eng.step(st, keywords=kw_t, reward_w=rw_t, k=k, d=d)
        torch.cuda.synchronize()
        ph = {"rollout": [], "verify": [], "tail": []}
        lens = []
        t0 = time.perf_counter()
        for _ in range(steps):
            lens.append(float(np.sum(st.prefix.lengths())))
            marks = []
            eng.step(st, keywords=kw_t, reward_w=rw_t, k=k, d=d, marks=marks)
            ph["rollout"].append(marks)
        torch.cuda.synchronize()
        sec = time.perf_counter() - t0
        med = {"rollout": float(np.median([m[0].elapsed_time(m[1]) for m in ph["rollout"]])),
               "verify": float(np.median([m[1].elapsed_time(m[2]) for m in ph["rollout"]])),
               "tail": float(np.median([m[2].elapsed_time(m[3]) for m in ph["rollout"]]))}
        row = {"k": k, "d": d, "ms_per_step": round(sec * 1e3 / steps, 3),
               "lookahead_tokens_per_s": round(B * k * d * steps / sec, 1),
               "cdsl_steps_per_s": round(steps / sec, 2)}
        row.update(phase_rooflines(wl, B, k, d, med, float(np.mean(lens))))
        log(json.dumps(row))
        rows.append(row)
        st.prefix.free()
    return rows


def main():
    args = parse()
    if args.summarize_profile:
        summarize_profile(args)
        return
    if args.summarize_ranges:
        summarize_ranges(args)
        return
    if args.summarize_trace:
        summarize_trace(args)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the path shards by prompt "
              "across GPUs with no exchange, but only the one-GPU step is built and timed)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch
    import cdsl_inputs as ci
    from paper_2412_10418_amd.engine import Engine

    wl = ci.workload(args.workload)
    if args.batch:
        wl = wl.with_(batch=args.batch)
    k = args.k or wl.k
    d = args.d or wl.d
    points = None
    if args.grid:
        ks, ds = args.grid.split(":")
        points = [(int(a), int(b)) for a in ks.split(",") for b in ds.split(",")]
        k, d = max(p[0] for p in points), max(p[1] for p in points)
    B, L = wl.batch, wl.prompt_len
    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    dw = ci.model_weights(wl.draft, wl.seed, 0, wl.dtype)
    tw = ci.model_weights(wl.target, wl.seed, 1, wl.dtype)
    log(f"weights generated in {time.perf_counter() - t0:.1f}s")
    t0 = time.perf_counter()
    dwd, twd = Engine.upload(wl, dw, tw)
    total_steps = args.warmup + args.steps + args.profile_steps + args.phase_steps
    # the methods comparison restarts from the prompt; its controller
    # iterations emit at most d + 2 tokens each
    total_steps = max(total_steps, 2 * (args.methods_steps + 1) + 1)
    eng = Engine(wl, dwd, twd, max_steps=total_steps + 2, max_batch=B, k=k, d=d)
    del dwd, twd
    torch.cuda.empty_cache()
    log(f"uploaded + cdsl_init in {time.perf_counter() - t0:.1f}s")
    prompts = ci.prompts(wl.seed, B, L, wl.target.vocab)
    kws = ci.keywords(wl.seed, B, wl.n_keywords, wl.target.vocab) if wl.reward.startswith("keyword") else None
    rw = ci.reward_head(wl.seed, wl.target.d_model) if wl.reward == "linear" else None
    kw_t = torch.from_numpy(kws).cuda() if kws is not None else None
    rw_t = torch.from_numpy(rw).cuda() if rw is not None else None

    if points:
        grid = measure_grid(eng, wl, prompts, kw_t, rw_t, points, args.steps, args.warmup)
        eng.close()
        print(json.dumps({"workload": wl.name, "batch": B, "prompt_len": L, "grid": grid}), flush=True)
        return
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    st = eng.start(torch.from_numpy(prompts).cuda(), k=k)
    torch.cuda.synchronize()
    prefill_s = time.perf_counter() - t0
    log(f"prefill {B}x{L}: {prefill_s * 1e3:.1f} ms")

    for _ in range(args.warmup):
        eng.step(st, keywords=kw_t, reward_w=rw_t, k=k, d=d)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        eng.step(st, keywords=kw_t, reward_w=rw_t, k=k, d=d)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_step = elapsed * 1e3 / args.steps
    tok_s = B * k * d * args.steps / elapsed
    log(f"timed {args.steps} steps: {ms_step:.2f} ms/step, {tok_s:.0f} lookahead tokens verified/s")

    # phase timing (rollout | verify | reward + select + commit), median over steps
    phase = {"rollout": [], "verify": [], "tail": []}
    lens = []
    for _ in range(args.phase_steps):
        lens.append(float(np.sum(st.prefix.lengths())))
        marks = []
        eng.step(st, keywords=kw_t, reward_w=rw_t, k=k, d=d, marks=marks)
        torch.cuda.synchronize()
        phase["rollout"].append(marks[0].elapsed_time(marks[1]))
        phase["verify"].append(marks[1].elapsed_time(marks[2]))
        phase["tail"].append(marks[2].elapsed_time(marks[3]))
    phases = None
    if args.phase_steps > 0:
        phases = phase_rooflines(wl, B, k, d, {nm: float(np.median(v)) for nm, v in phase.items()},
                                 float(np.mean(lens)))
        log(json.dumps(phases))

    # instrumented steps: per-kernel-class HIP event timing
    eng.ctx.profile_enable(True)
    t0 = time.perf_counter()
    for _ in range(args.profile_steps):
        eng.step(st, keywords=kw_t, reward_w=rw_t, k=k, d=d)
    stats = eng.ctx.profile_read()
    prof_wall = (time.perf_counter() - t0) * 1e3
    eng.ctx.profile_enable(False)
    kern_ms = sum(v["ms"] for v in stats.values())
    if args.profile_steps > 0 and kern_ms > 0:
        dom, roof = roofline(stats, wl.name)
        table = class_table(stats, kern_ms)
        log(json.dumps(table, indent=1))
        log(f"instrumented: kernel time {kern_ms / args.profile_steps:.2f} ms/step of "
            f"{prof_wall / args.profile_steps:.2f} ms/step wall")
    else:   # no instrumented steps: no roofline object
        dom, roof, table = None, None, {}
    emitted = sum(len(e) for e in st.emitted)
    st.prefix.free()
    methods = measure_methods(eng, wl, prompts, k, d, args.methods_steps) if args.methods_steps > 0 else None
    if methods:
        log(json.dumps(methods))
    if args.calibrate_copy:
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("calibration: 3 copies of 256 MiB (reads 262144 KiB, writes 262144 KiB per copy)")
        del src, dst
    eng.close()
    del eng
    torch.cuda.empty_cache()

    cpu = None
    if not args.no_cpu_baseline:
        try:
            cpu = cpu_baseline(wl, dw, tw, prompts[0], kws[0] if kws is not None else None, rw, k, d)
        except MemoryError:
            cpu = {"value": None, "unit": "lookahead tokens verified/s", "cores": os.cpu_count(),
                   "kind": "oracle", "sample": "skipped: host memory"}

    out = {
        "metric": "lookahead tokens verified/sec",
        "value": round(tok_s, 1),
        "unit": "lookahead tokens verified/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "cdsl_steps_per_s": round(1e3 / ms_step, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 weights, fp32 activations" if wl.dtype == "bf16" else "f32",
        "data": "synthetic (seeded random-init weights, uniform-random prompts)",
        "config": {"workload": wl.name, "draft": f"{wl.draft.n_layers}L/{wl.draft.d_model}/"
                                                  f"{wl.draft.n_heads}H/kv{wl.draft.n_kv_heads}/{wl.draft.ffn_dim}",
                   "target": f"{wl.target.n_layers}L/{wl.target.d_model}/{wl.target.n_heads}H/"
                             f"kv{wl.target.n_kv_heads}/{wl.target.ffn_dim}",
                   "vocab": wl.target.vocab, "batch": B, "prompt_len": L, "k": k, "d": d,
                   "reward": wl.reward, "prefill_ms": round(prefill_s * 1e3, 1),
                   "tokens_emitted": emitted},
        "roofline": roof,
        "phases": phases,
        "methods": methods,
        "kernels": table,
        "launches_per_step": (round(sum(v["launches"] for v in stats.values()) / args.profile_steps)
                              if args.profile_steps > 0 else None),
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
