"""The benchmark's measurement tooling on the CPU: the roofline-pass summaries
of rocprofv3 trace and counter CSVs (the marker fills delimit the pass, the
per-step work outside the layer calls is left out), the committed traffic
records and their source digest, and the refusal of more than one GPU."""
import csv
import io
import json
import os
import subprocess
import sys
from contextlib import redirect_stdout

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

MARK = "void at::native::vectorized_elementwise_kernel<8, at::native::FillFunctor<short>, std::array<char*, 1ul> >(int, at::native::FillFunctor<short>, std::array<char*, 1ul>)"


def write_trace(path, recs):
    """recs: (kernel name, start ns, end ns)."""
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Kernel_Name", "Start_Timestamp", "End_Timestamp", "Workgroup_Size_X", "Workgroup_Size_Y",
                    "Workgroup_Size_Z", "Grid_Size_X", "Grid_Size_Y", "Grid_Size_Z"])
        for name, t0, t1 in recs:
            w.writerow([name, t0, t1, 256, 1, 1, 256, 1, 1])


def run(fn, *args):
    buf = io.StringIO()
    with redirect_stdout(buf):
        fn(*args)
    return buf.getvalue()


def test_pass_summary_of_a_trace(tmp_path):
    """Only the kernels between the two marker fills count, less the
    compaction, plan and spin kernels; per layer call = their time / calls."""
    p = str(tmp_path / "trace.csv")
    write_trace(p, [
        ("gemm_before", 0, 5000),                       # warm-up: before the first marker
        (MARK, 10000, 11000),
        ("at::cuda::spin_kernel(long)", 12000, 2012000),
        ("compact_weights_kernel<__bf16>", 2013000, 2043000),
        ("plan_tiles_wide_kernel", 2044000, 2050000),
        ("fast_gemm_kernel<A>", 2051000, 2061000),      # 10 us
        ("fast_gemm_kernel<A>", 2062000, 2072000),      # 10 us
        ("splitk_reduce4_kernel<float, 1>", 2073000, 2077000),  # 4 us
        (MARK, 2080000, 2081000),
        ("gemm_after", 2090000, 2190000),               # the comparisons after the pass
    ])
    out = run(bench.summarize_pass, p, 10, 2, "trace")
    assert "roofline pass: 3 kernels, 24.0 us of kernel time, 12.00 us per layer call (2 calls)" in out
    assert "compact" not in out and "plan_tiles" not in out and "spin" not in out
    assert "gemm_before" not in out and "gemm_after" not in out


def test_pass_summary_of_counters(tmp_path):
    p = str(tmp_path / "counters.csv")
    rows = [(1, "gemm_before", 100.0), (2, MARK, 1.0), (3, "compact_weights_kernel<__bf16>", 500.0),
            (4, "fast_gemm_kernel<A>", 30.0), (5, "fast_gemm_kernel<A>", 50.0), (6, MARK, 1.0),
            (7, "gemm_after", 70.0)]
    with open(p, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for d, name, v in rows:
            w.writerow([d, name, "FETCH_SIZE", v])
    out = run(bench.summarize_pass, p, 5, 2, "counters")
    assert "roofline pass: FETCH_SIZE sum 80.0 over 2 dispatches, 40.0 per layer call" in out


def test_pass_summary_needs_both_markers(tmp_path):
    p = str(tmp_path / "trace.csv")
    write_trace(p, [(MARK, 0, 1000), ("fast_gemm_kernel<A>", 2000, 3000)])
    with pytest.raises(AssertionError):
        run(bench.summarize_pass, p, 5, 1, "trace")


def test_traffic_record_follows_the_source_digest(tmp_path, monkeypatch):
    """A record counts only for the kernel sources it was taken on."""
    prof = tmp_path / "profiles"
    prof.mkdir()
    rec = {"workload": "w", "p": 0.7, "steps": 100, "source_digest": bench.source_digest(), "bytes_per_call": 1234}
    stale = dict(rec, source_digest="0" * 64, bytes_per_call=999)
    (prof / "a.md").write_text("text\ntraffic-record: " + json.dumps(stale) + "\n")
    (prof / "b.md").write_text("traffic-record: " + json.dumps(rec) + "\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    # the digest covers the kernel sources under ROOT: give the temporary root the same files
    os.symlink(os.path.join(ROOT, "paper_1805_08939_amd"), tmp_path / "paper_1805_08939_amd")
    os.symlink(os.path.join(ROOT, "include"), tmp_path / "include")
    assert bench.traffic_record("w", 0.7, 100) == 1234
    assert bench.traffic_record("w", 0.5, 100) is None
    assert bench.traffic_record("v", 0.7, 100) is None
    (prof / "b.md").unlink()
    assert bench.traffic_record("w", 0.7, 100) is None  # only the stale record is left


def test_digest_ignores_comments_and_layout():
    """Comments, blank lines and runs of blanks do not change the code a
    record was taken on; a change of the code does."""
    a = "int f(int x) {  // one\n  return x + 1; /* two */\n}\n"
    b = "/* header\n   lines */\nint f(int x) {\n\n  return  x + 1;\n}  // end\n"
    c = "int f(int x) {\n  return x + 2;\n}\n"
    assert bench.code_text(a) == bench.code_text(b) == "int f(int x) {\nreturn x + 1;\n}"
    assert bench.code_text(c) != bench.code_text(a)
    s = 'const char* s = "/* kept */ // kept"; char q = \'"\';'
    assert bench.code_text(s) == s


def test_committed_traffic_records_parse():
    """Every committed profile carries one parsable traffic record with the
    fields the benchmark reads."""
    pdir = os.path.join(ROOT, "profiles")
    n = 0
    for f in sorted(os.listdir(pdir)):
        lines = [l for l in open(os.path.join(pdir, f)) if l.startswith("traffic-record: ")]
        for l in lines:
            rec = json.loads(l[len("traffic-record: "):])
            assert {"workload", "p", "steps", "source_digest", "bytes_per_call"} <= set(rec), f
            assert rec["bytes_per_call"] > 0 and len(rec["source_digest"]) == 64
            n += 1
    assert n >= 5


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
