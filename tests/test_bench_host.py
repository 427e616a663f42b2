"""Host logic of the benchmark, without a GPU: the one-GPU contract, the
roofline arithmetic, the phase rates, and the rocprofv3 summary (counter
calibration, bytes per launch, the source-digest gate on stored traffic), and
the per-call summary of a marker trace."""
import csv
import json
import os
import subprocess
import sys
import types

import pytest

import cdsl_inputs as ci

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stdout + r.stderr


def test_roofline_of_the_dominant_class(monkeypatch):
    """frac = algorithmic flops (or bytes) per second over the peak; the
    dense projection's executed fraction is twice the algorithmic one."""
    monkeypatch.setattr(bench, "stored_traffic", lambda cls, wl: None)
    stats = {"gemm_dense": {"ms": 10.0, "launches": 4, "flops": 5e12, "bytes": 4e9},
             "attention": {"ms": 2.0, "launches": 8, "flops": 0.0, "bytes": 8e9}}
    cls, r = bench.roofline(stats, "7b1b")
    assert cls == "gemm_dense" and r["bound"] == "mfma"
    assert r["achieved"] == pytest.approx(500.0)                 # 5e12 flop / 10 ms
    assert r["frac"] == pytest.approx(0.2)
    assert r["executed_frac"] == pytest.approx(0.4)
    assert r["alg_flops_per_launch"] == pytest.approx(1.25e12)
    assert r["avg_launch_us"] == pytest.approx(2500.0)
    assert r["traffic"] is None
    stats["attention"]["ms"] = 20.0
    cls, r = bench.roofline(stats, "7b1b")
    assert cls == "attention" and r["bound"] == "hbm"
    assert r["achieved"] == pytest.approx(400.0)                 # 8e9 B / 20 ms
    assert r["frac"] == pytest.approx(0.05)


def test_phase_rates_count_weights_and_prefix_kv():
    """Rollout bytes: d passes, each streaming the draft weights (bf16, no
    embedding) and every prompt's prefix KV once (bf16; the stored figure
    at 4 bytes for the hi + lo pair).  Verify flops: 2 per target weight
    (no embedding) per fed row."""
    wl = ci.workload("7b1b")
    B, k, d, L = wl.batch, wl.k, wl.d, wl.prompt_len
    dr, tg = wl.draft, wl.target

    def params(m):   # per layer: q, k, v, o, gate, up, down; plus the LM head
        hd = m.d_model // m.n_heads
        per = m.d_model * (m.n_heads * hd + 2 * m.n_kv_heads * hd) + m.n_heads * hd * m.d_model \
            + 3 * m.d_model * m.ffn_dim
        return m.n_layers * per + m.vocab * m.d_model

    hd = dr.d_model // dr.n_heads
    kv_tok = dr.n_layers * 2 * dr.n_kv_heads * hd
    out = bench.phase_rooflines(wl, B, k, d, {"rollout": 10.0, "verify": 20.0, "tail": 1.0}, B * L)
    assert out["rollout_bytes"] == pytest.approx(d * (2.0 * params(dr) + B * L * kv_tok * 2.0), rel=1e-3)
    assert out["rollout_stored_bytes"] == pytest.approx(d * (2.0 * params(dr) + B * L * kv_tok * 4.0), rel=1e-3)
    assert out["verify_gemm_flops"] == pytest.approx(2.0 * B * k * d * params(tg), rel=1e-3)
    assert out["rollout_GB_per_s"] == pytest.approx(out["rollout_bytes"] / 10e-3 / 1e9, rel=1e-3)
    assert out["verify_executed_mfma_frac"] == pytest.approx(2 * out["verify_mfma_frac"], rel=1e-3)


def _write_csv(path, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=list(rows[0].keys()))
        w.writeheader()
        w.writerows(rows)


def test_profile_summary_scales_counters_by_the_copy_calibration(tmp_path, monkeypatch):
    """A synthetic run: the calibration copies read FETCH_SIZE = 131072 KiB
    for 262144 KiB moved (scale 2) and WRITE_SIZE = 262144 KiB (scale 1);
    the dense class reads 1000 KiB and writes 500 KiB per dispatch, so
    (1000 * 2 + 500) KiB per launch.  The summary's traffic record carries
    that figure and the digest of the kernel's sources, and the bench only
    uses a record whose digest matches."""
    trace, fetch, write = (tmp_path / n for n in ("trace", "fetch", "write"))
    for p in (trace, fetch, write):
        p.mkdir()
    dense = "void cdsl::(anonymous namespace)::gemm_bf16_dense<2, 4, 5, 4, 64, 0>(GemmArgs)"
    _write_csv(trace / "bench_kernel_stats.csv",
               [{"Name": dense, "Calls": "10", "TotalDurationNs": "1500000", "AverageNs": "150000"}])
    copy = "__amd_rocclr_copyBuffer"

    def counters(val, cal):
        rows = [{"Kernel_Name": dense, "Counter_Value": str(val)} for _ in range(3)]
        rows += [{"Kernel_Name": copy, "Counter_Value": str(cal)} for _ in range(3)]
        return rows

    _write_csv(fetch / "bench_counter_collection.csv", counters(1000.0, 131072.0))
    _write_csv(write / "bench_counter_collection.csv", counters(500.0, 262144.0))
    line = {"ms_per_step": 37.0, "value": 21600.0, "unit": "lookahead tokens verified/s",
            "config": {"workload": "7b1b", "batch": 16, "k": 5, "d": 10},
            "roofline": {"kernel": "gemm_dense", "alg_bytes_per_launch": 1.5e8},
            "kernels": {"gemm_dense": {"avg_launch_us": 151.0}}}
    bj = tmp_path / "bench.json"
    bj.write_text(json.dumps(line) + "\n")
    out = tmp_path / "summary.md"
    args = types.SimpleNamespace(summarize_profile=[str(bj), str(trace), str(fetch), str(write)],
                                 summary_out=str(out), commands=None)
    bench.summarize_profile(args)
    text = out.read_text()
    assert "scaled by 2.0000 (fetch) and 1.0000 (write)" in text
    recs = [json.loads(ln[len(bench.TRAFFIC_TAG):-len(" -->")]) for ln in text.splitlines()
            if ln.startswith(bench.TRAFFIC_TAG)]
    rec = [r for r in recs if r["class"] == "gemm_dense"][0]
    assert rec["bytes_per_launch"] == round((1000.0 * 2 + 500.0) * 1024)
    assert rec["source"] == bench.source_digest(bench.CLASS_KERNEL["gemm_dense"][1])
    # the gate: a matching digest is used, a stale one is not
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "summary.md").write_text(text)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    real = bench.source_digest
    monkeypatch.setattr(bench, "source_digest", lambda files: rec["source"])
    assert bench.stored_traffic("gemm_dense", "7b1b")["bytes_per_launch"] == rec["bytes_per_launch"]
    assert bench.stored_traffic("gemm_dense", "long") is None
    monkeypatch.setattr(bench, "source_digest", lambda files: "0" * 16)
    assert bench.stored_traffic("gemm_dense", "7b1b") is None
    monkeypatch.setattr(bench, "source_digest", real)


def test_range_summary_attributes_kernels_by_launch_time(tmp_path):
    """A kernel counts for the roctx range (library call) in which its launch
    call started on the same thread; its GPU time is its own duration."""
    def w(name, rows):
        _write_csv(tmp_path / name, rows)

    w("x_marker_api_trace.csv", [
        {"Function": "cdsl_rollout", "Thread_Id": "1", "Start_Timestamp": "100", "End_Timestamp": "200"},
        {"Function": "cdsl_verify", "Thread_Id": "1", "Start_Timestamp": "300", "End_Timestamp": "400"},
        {"Function": "cdsl_rollout", "Thread_Id": "1", "Start_Timestamp": "500", "End_Timestamp": "600"}])
    w("x_hip_api_trace.csv", [
        {"Correlation_Id": "1", "Thread_Id": "1", "Start_Timestamp": "110"},
        {"Correlation_Id": "2", "Thread_Id": "1", "Start_Timestamp": "150"},
        {"Correlation_Id": "3", "Thread_Id": "2", "Start_Timestamp": "160"},   # another thread
        {"Correlation_Id": "4", "Thread_Id": "1", "Start_Timestamp": "350"},
        {"Correlation_Id": "5", "Thread_Id": "1", "Start_Timestamp": "550"},
        {"Correlation_Id": "6", "Thread_Id": "1", "Start_Timestamp": "450"}])  # outside every range
    w("x_kernel_trace.csv", [
        {"Correlation_Id": c, "Start_Timestamp": "0", "End_Timestamp": str(ns)}
        for c, ns in (("1", 1_000_000), ("2", 3_000_000), ("3", 9_000_000), ("4", 5_000_000),
                      ("5", 2_000_000), ("6", 7_000_000))])
    out = tmp_path / "r.md"
    bench.summarize_ranges(types.SimpleNamespace(summarize_ranges=str(tmp_path), summary_out=str(out)))
    rows = {ln.split("|")[1].strip(" `"): [x.strip() for x in ln.split("|")[2:6]]
            for ln in out.read_text().splitlines()[2:]}
    # rollout: 2 calls, kernels 1, 2 (first) and 5 (second): 3 / 2 per call, 6 ms / 2
    assert rows["cdsl_rollout"] == ["2", f"{100 / 1e6:.3f}", "1.5", "3.000"]
    assert rows["cdsl_verify"] == ["1", f"{100 / 1e6:.3f}", "1.0", "5.000"]


def test_trace_summary_groups_one_step_by_kernel_and_grid(tmp_path):
    """The step summarised is the last one between two commits before the
    instrumented step; launches are grouped by kernel and grid, and a name
    the tracer left mangled is shortened."""
    bj = tmp_path / "b.json"
    bj.write_text(json.dumps({"ms_per_step": 5.0, "value": 100.0, "unit": "lookahead tokens verified/s",
                              "config": {"workload": "long", "batch": 64, "k": 8, "d": 8}}) + "\n")
    _write_csv(tmp_path / "x_kernel_stats.csv", [
        {"Name": "void cdsl::(anonymous namespace)::gemm_bf16_dense<2, 4, 5, 4, 64, 0>(GemmArgs)", "Calls": "4",
         "TotalDurationNs": "4000", "AverageNs": "1000"},
        {"Name": "_ZN4cdsl12_GLOBAL__N_110embed_rowsIDF16bEEvNS_8PassDescE", "Calls": "2",
         "TotalDurationNs": "1000", "AverageNs": "500"}])
    seq = ["commit_kernel", "gemm", "gemm", "emb", "commit_kernel", "gemm", "emb", "commit_kernel", "gemm",
           "commit_kernel"]
    names = {"gemm": "void cdsl::(anonymous namespace)::gemm_bf16_dense<2, 4, 5, 4, 64, 0>(GemmArgs)",
             "emb": "_ZN4cdsl12_GLOBAL__N_110embed_rowsIDF16bEEvNS_8PassDescE",
             "commit_kernel": "cdsl::commit_kernel(CommitArgs)"}
    _write_csv(tmp_path / "x_kernel_trace.csv", [
        {"Kernel_Name": names[n], "Start_Timestamp": str(1000 * t), "End_Timestamp": str(1000 * t + 500),
         "Grid_Size_X": "512", "Workgroup_Size_X": "256", "Grid_Size_Y": "1", "Grid_Size_Z": "3" if n == "gemm" else "1"}
        for t, n in enumerate(seq)])
    out = tmp_path / "s.md"
    bench.summarize_trace(types.SimpleNamespace(summarize_trace=[str(bj), str(tmp_path)], summary_out=str(out),
                                                commands=None))
    text = out.read_text()
    assert "workload long (batch 64, k = 8, d = 8)" in text
    assert "| `embed_rows<...>` | 2 |" in text
    # the step between the second and third commits: gemm, emb, commit
    assert "One step of the traced run (between two commits): 3 launches" in text
    assert "| `void gemm_bf16_dense<2, 4, 5, 4, 64, 0>` | 2x1x3 | 1 |" in text


def test_source_digest_ignores_comments_but_not_code(tmp_path, monkeypatch):
    src = tmp_path / "paper_2412_10418_amd" / "csrc"
    src.mkdir(parents=True)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    f = src / "k.hip"
    f.write_text("// header\n__global__ void k(float* x) {\n  x[0] = 1.f;  // one\n}\n")
    d0 = bench.source_digest(["k.hip"])
    f.write_text("/* a block\n comment */\n__global__ void k(float* x) {\n\n    x[0] = 1.f;\n}\n")
    assert bench.source_digest(["k.hip"]) == d0
    f.write_text("__global__ void k(float* x) {\n  x[0] = 2.f;\n}\n")
    assert bench.source_digest(["k.hip"]) != d0
