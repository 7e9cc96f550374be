"""Host logic of bench.py (CPU only): the HBM-traffic summary built from two
rocprofv3 counter CSVs, its copy-calibration scaling, and the rule that a stored
figure is used only while the fused kernel's sources are unchanged."""
import csv
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

KERNEL = "void rlsim_dev::k_cartpole_split<0, true>(rlsim_dev::StepArgs)"
COPY = "__amd_rocclr_copyBuffer"


def _csv(path, counter, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, value in rows:
            w.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": value})


def test_ingest_scales_by_the_copy_and_round_trips(tmp_path, monkeypatch):
    out = tmp_path / "traffic.txt"
    monkeypatch.setattr(bench, "traffic_file", lambda workload: str(out))
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    # the 1 GiB copy reads as half its bytes on FETCH_SIZE and exactly on WRITE_SIZE
    _csv(fetch, "FETCH_SIZE", [(KERNEL, 98.0), (KERNEL, 100.0), (KERNEL, 102.0), (COPY, 524288.0)])
    _csv(write, "WRITE_SIZE", [(KERNEL, 1000.0), (KERNEL, 1000.0), (KERNEL, 1010.0), (COPY, 1048576.0)])
    bench.ingest_pmc(str(fetch), str(write), "wl", bench.HEADLINE_KERNEL_PREFIX)
    kv = bench._read_kv(str(out))
    assert float(kv["copy_fetch_scale"]) == 2.0 and float(kv["copy_write_scale"]) == 1.0
    # medians 100 and 1000 KiB: 100 * 1024 * 2 + 1000 * 1024 * 1
    assert float(kv["hbm_bytes_per_launch"]) == 100 * 1024 * 2 + 1000 * 1024
    assert kv["source_digest"] == bench.kernel_source_digest()
    assert bench.stored_traffic("wl") == 100 * 1024 * 2 + 1000 * 1024
    # a change to the kernel's sources invalidates the stored figure
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: "0" * 16)
    assert bench.stored_traffic("wl") is None


def test_ingest_needs_the_kernel_and_the_copy(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "traffic_file", lambda workload: str(tmp_path / "t.txt"))
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    _csv(fetch, "FETCH_SIZE", [(KERNEL, 100.0)])
    _csv(write, "WRITE_SIZE", [(KERNEL, 1000.0)])
    with pytest.raises(SystemExit):
        bench.ingest_pmc(str(fetch), str(write), "wl", bench.HEADLINE_KERNEL_PREFIX)


def test_missing_summary_gives_no_traffic(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "traffic_file", lambda workload: str(tmp_path / "absent.txt"))
    assert bench.stored_traffic("wl") is None



def test_kernel_digest_ignores_comments_but_not_code():
    """The stored traffic stays valid across comment edits of the kernel sources
    and is dropped when their code changes."""
    src = "int f(int x) { // a comment\n  return x + 1; /* block\n comment */ }\n"
    assert bench.code_text(src) == bench.code_text(src.replace("a comment", "another comment"))
    assert bench.code_text(src) == bench.code_text(src.replace("  return", "\treturn"))
    assert bench.code_text(src) != bench.code_text(src.replace("x + 1", "x + 2"))
    assert "comment" not in bench.code_text(src)
