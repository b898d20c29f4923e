"""CPU checks of bench.py's bookkeeping: the algorithmic byte counts behind
roofline.achieved, Table I's per-node communication, the source digest that
keys the committed counters, and the one-GPU guard."""
import os
import subprocess
import sys
import types

import pytest

import bench
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_algorithmic_bytes_of_the_streaming_stage():
    # 1.1B: N*d*(2 + 12) for bf16 gradients plus the per-worker sketch S.
    w = synth.WORKLOADS["llama1b"]
    got = bench.algorithmic_bytes(w, w.K_global())["sketch_kernel"]
    assert got == w.N * w.d * 14 + 4 * w.N * w.m * w.r == 61_637_086_016
    # 124M: fp32 gradients, 16 bytes per element and worker.
    w = synth.WORKLOADS["gpt2s"]
    assert bench.algorithmic_bytes(w, w.K_global())["sketch_kernel"] == \
        w.N * w.d * 16 + 4 * w.N * w.m * w.r


def test_comparison_compressors_stream_what_they_need():
    w = synth.WORKLOADS["llama1b"]
    arc = bench.algorithmic_bytes(w, w.K_global())["sketch_kernel"]
    randk = bench.algorithmic_bytes(w, w.K_global(), "randk")["sketch_kernel"]
    topk = bench.algorithmic_bytes(w, w.K_global(), "topk")["sketch_kernel"]
    assert randk == w.N * w.d * (2 + 8)  # grad + h read and write only
    assert topk == w.N * w.d * 14 + 4 * w.N * w.m
    assert randk < topk < arc


def test_table1_communication_per_node():
    # Table I: ARC-Top-K 2Kn + 2mr, Rand-K 2Kn, local Top-K (N-1)(nK + K).
    w = synth.WORKLOADS["gpt2s"]
    K, n = 163, w.n
    comp = types.SimpleNamespace(K_total=K, payload=K * n, m=w.m)
    arc = bench.table1_communication(w, comp, "arc")
    assert arc["values"] == 2 * K * n + 2 * w.m * w.r
    assert arc["uncompressed"] == 2 * w.d
    assert bench.table1_communication(w, comp, "randk")["values"] == 2 * K * n
    topk_comp = types.SimpleNamespace(K_total=w.N * K, payload=w.N * K * n, m=w.m)
    assert bench.table1_communication(w, topk_comp, "topk")["values"] == \
        (w.N - 1) * (n * K + K)


def test_kernel_digest_ignores_comments_and_whitespace(tmp_path):
    a = tmp_path / "a.hip"
    b = tmp_path / "b.hip"
    c = tmp_path / "c.hip"
    a.write_text("int f(int x) {\n  return x + 1;  // one\n}\n")
    b.write_text("/* header */\nint f(int x)\n{\n    return x + 1;\n}\n")
    c.write_text("int f(int x) {\n  return x + 2;\n}\n")
    assert bench.kernel_source_digest(str(a)) == bench.kernel_source_digest(str(b))
    assert bench.kernel_source_digest(str(a)) != bench.kernel_source_digest(str(c))


def test_committed_traffic_matches_the_current_kernel_source():
    # profiles/sketch_traffic.json must have been taken on this arc_sketch.hip;
    # otherwise bench.py reports traffic as null.
    import json
    rec = json.load(open(bench.TRAFFIC_FILE))
    assert rec["kernel_source_digest"] == bench.kernel_source_digest()
    for name in ("gpt2s", "llama1b"):
        e = rec["workloads"][name]
        assert e["hbm_bytes_per_launch"] == pytest.approx(e["algorithmic_bytes_per_launch"],
                                                          rel=2e-3)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one MI355X" in r.stderr


def test_host_info_states_cores_and_memory():
    info = bench.host_info()
    assert info["nproc"] == os.cpu_count()
    assert 1 <= info.get("affinity_cpus", 1) <= info["nproc"]
    assert 0 < info["mem_available_GB"] <= info["mem_total_GB"]


def test_unknown_workloads_are_refused():
    for args in (["--workload", "nope"], ["--also", "gpt2s,nope"]):
        r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                           capture_output=True, text=True, timeout=120)
        assert r.returncode == 2 and "unknown workload" in r.stderr, r.stderr
