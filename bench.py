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
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 256 MiB device copy (reference for HBM byte counters)")
    return ap.parse_args()


def roofline(stats):
    """Dominant kernel class of the instrumented steps and its roofline."""
    best = max(stats, key=lambda nm: stats[nm]["ms"])
    st = stats[best]
    sec = st["ms"] / 1e3
    per_launch_ms = st["ms"] / max(1, st["launches"])
    if best in ("gemm_dense",):
        ach = st["flops"] / sec / 1e12
        return best, {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_MFMA_BF16_TFS, "unit": "TFLOP/s",
                      "frac": round(ach / PEAK_MFMA_BF16_TFS, 4), "traffic": None,
                      "kernel": best, "avg_launch_us": round(per_launch_ms * 1e3, 2),
                      "launches": st["launches"]}
    ach = st["bytes"] / sec / 1e9
    return best, {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                  "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": None, "kernel": best,
                  "avg_launch_us": round(per_launch_ms * 1e3, 2), "launches": st["launches"]}


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


def cpu_baseline(wl, dw, tw, prompt, kws, rw, k, d):
    """The float64 oracle on one prompt: prefill (untimed), then the timed
    sample = the full verification of the k*d block + the greedy rollout of
    ONE beam (d draft forwards), scaled to a whole step as
    t_verify + k * t_one_beam + t_reward_select_commit."""
    import numpy as np
    import oracle
    threads = os.environ.get("OMP_NUM_THREADS") or str(os.cpu_count())
    od, ot = oracle.Decoder(wl.draft, dw), oracle.Decoder(wl.target, tw)
    t0 = time.perf_counter()
    st = oracle.prefill(od, ot, prompt)
    t_prefill = time.perf_counter() - t0
    log(f"cpu baseline: oracle prefill {t_prefill:.1f}s")
    heads, hlp, _ = oracle.beam_heads(st, k)
    t0 = time.perf_counter()
    ro = oracle.rollout(od, st, heads[:1], d)
    t_beam = time.perf_counter() - t0
    log(f"cpu baseline: one-beam rollout {t_beam:.1f}s")
    x = np.concatenate([ro.x, np.tile(ro.x[:1], (k - 1, 1))]) if k > 1 else ro.x
    t0 = time.perf_counter()
    ve = oracle.verify(ot, st, heads, hlp, x)
    t_ver = time.perf_counter() - t0
    log(f"cpu baseline: verification {t_ver:.1f}s")
    t0 = time.perf_counter()
    r = oracle.reward_for(wl.reward, st.generated, heads, x, ve.hidden, kws, rw)
    b = oracle.select_beam(ve.scores, r, wl.alpha)
    emitted = [int(heads[b])] + [int(t) for t in x[b, :int(ve.n[b])]]
    oracle.commit(od, ot, st, emitted)
    t_tail = time.perf_counter() - t0
    t_step = t_ver + k * t_beam + t_tail
    return {"value": round(k * d / t_step, 4), "unit": "lookahead tokens verified/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"1 prompt x 1 step of workload '{wl.name}' in float64: verification of the "
                       f"{k}x{d} block {t_ver:.1f}s + rollout of 1 beam {t_beam:.1f}s (x{k} beams) + "
                       f"reward/select/commit {t_tail:.1f}s; prompt prefill {t_prefill:.1f}s untimed"),
            "s_per_prompt_step": round(t_step, 3)}


def main():
    args = parse()
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
    B, L = wl.batch, wl.prompt_len
    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    dw = ci.model_weights(wl.draft, wl.seed, 0, wl.dtype)
    tw = ci.model_weights(wl.target, wl.seed, 1, wl.dtype)
    log(f"weights generated in {time.perf_counter() - t0:.1f}s")
    t0 = time.perf_counter()
    dwd, twd = Engine.upload(wl, dw, tw)
    total_steps = args.warmup + args.steps + args.profile_steps
    eng = Engine(wl, dwd, twd, max_steps=total_steps + 2, max_batch=B, k=k, d=d)
    del dwd, twd
    torch.cuda.empty_cache()
    log(f"uploaded + cdsl_init in {time.perf_counter() - t0:.1f}s")
    prompts = ci.prompts(wl.seed, B, L, wl.target.vocab)
    kws = ci.keywords(wl.seed, B, wl.n_keywords, wl.target.vocab) if wl.reward.startswith("keyword") else None
    rw = ci.reward_head(wl.seed, wl.target.d_model) if wl.reward == "linear" else None
    kw_t = torch.from_numpy(kws).cuda() if kws is not None else None
    rw_t = torch.from_numpy(rw).cuda() if rw is not None else None

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

    # instrumented steps: per-kernel-class HIP event timing
    eng.ctx.profile_enable(True)
    t0 = time.perf_counter()
    for _ in range(args.profile_steps):
        eng.step(st, keywords=kw_t, reward_w=rw_t, k=k, d=d)
    stats = eng.ctx.profile_read()
    prof_wall = (time.perf_counter() - t0) * 1e3
    eng.ctx.profile_enable(False)
    dom, roof = roofline(stats)
    kern_ms = sum(v["ms"] for v in stats.values())
    table = class_table(stats, kern_ms)
    log(json.dumps(table, indent=1))
    log(f"instrumented: kernel time {kern_ms / args.profile_steps:.2f} ms/step of "
        f"{prof_wall / args.profile_steps:.2f} ms/step wall")
    emitted = sum(len(e) for e in st.emitted)
    if args.calibrate_copy:
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("calibration: 3 copies of 256 MiB (reads 262144 KiB, writes 262144 KiB per copy)")
        del src, dst
    st.prefix.free()
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
        "kernels": table,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
