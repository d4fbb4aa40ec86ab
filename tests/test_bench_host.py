"""Host-side pieces of bench.py (no GPU): the single-GPU guard, the traffic
figure's source check, token sizing and the CPU baseline's report."""
import math
import os
import subprocess
import sys

import bench
import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def _summary(path, digest, traffic="6.5000e+08"):
    with open(path, "w") as f:
        f.write("# HBM traffic\n\n")
        f.write(f"- traffic_bytes_per_launch: `{traffic}`\n")
        f.write(f"- gemm_bf16.hip code sha256[:16]: `{digest}`\n")


def test_measured_traffic_only_for_the_profiled_source(tmp_path, monkeypatch):
    path = tmp_path / "traffic.md"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(path))
    assert bench.measured_traffic() is None                      # no summary
    _summary(path, bench.gemm_source_hash())
    assert bench.measured_traffic() == 6.5e8                     # current source
    _summary(path, "0" * 16)
    assert bench.measured_traffic() is None                      # another source
    _summary(path, bench.gemm_source_hash(), traffic="n/a")
    assert bench.measured_traffic() is None                      # unreadable value


def test_code_hash_ignores_comments_only(tmp_path):
    a, b, c = tmp_path / "a.hip", tmp_path / "b.hip", tmp_path / "c.hip"
    a.write_text("int f() {  // one\n  return 1;\n}\n")
    b.write_text("// header\n\nint f() {  // two\n  return 1;   \n}\n")
    c.write_text("int f() {\n  return 2;\n}\n")
    assert bench.code_hash(a) == bench.code_hash(b)
    assert bench.code_hash(a) != bench.code_hash(c)


def test_needed_tokens_cover_the_timed_passes():
    for name in ("tiny", "small", "8b", "8b-throughput", "8b-long"):
        w = wl.WORKLOADS[name]
        cd = w.codec
        for passes in (1, 4, 131):
            n = bench.needed_tokens(w, passes)
            assert n <= w.n_tokens
            # every chunk lasts at least chunk_len / m_max passes, so these many
            # batches of chunks keep every slot busy for `passes` passes
            want = cd.batch * (math.ceil(passes / math.ceil(cd.chunk_len / cd.m_max)) + 1)
            assert n == min(w.n_tokens, want * cd.chunk_len)


def test_cpu_baseline_reports_the_oracle():
    out = bench.cpu_baseline(wl.WORKLOADS["tiny"])
    assert out["kind"] == "oracle" and out["unit"] == "B/s"
    assert out["value"] > 0 and out["cores"] >= 1
    assert "fp64" in out["sample"]
