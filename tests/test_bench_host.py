"""Host-side pieces of the benchmark: the source hash that dates the stored
HBM-traffic counter readings, and the workload bookkeeping (no GPU)."""
import json
import os

import bench


def test_code_only_ignores_comments_and_layout():
    a = "int x = 1;  // one\n/* block\n comment */ float y = x * 2;\n"
    b = "int x=1;\nfloat y=x*2;"
    assert bench._code_only(a) == bench._code_only(b)
    assert bench._code_only("int x = 1;") != bench._code_only("int x = 2;")


def test_kernel_hash_is_stable_and_covers_the_sources():
    h = bench.kernel_hash()
    assert h == bench.kernel_hash() and len(h) == 16
    for f in bench.KERNEL_SOURCES:
        assert os.path.exists(os.path.join(bench.ROOT, "paper_2608_01891_amd", "csrc", f)), f


def test_traffic_file_records_its_commands_and_calibration():
    with open(bench.TRAFFIC_FILE) as fh:
        d = json.load(fh)
    assert d["kernel"] == "gemm_gate_up" and len(d["kernel_hash"]) == 16
    assert any("FETCH_SIZE" in c for c in d["commands"]) and any("WRITE_SIZE" in c for c in d["commands"])
    cal = d["calibration"]
    # a 1 GiB copy: the counters' KiB per dispatch scaled back to the bytes moved
    assert abs(cal["FETCH_SIZE_KiB"] * 1024 * cal["fetch_factor"] - cal["copy_bytes"]) < 0.01 * cal["copy_bytes"]
    assert abs(cal["WRITE_SIZE_KiB"] * 1024 * cal["write_factor"] - cal["copy_bytes"]) < 0.01 * cal["copy_bytes"]
    assert d["bytes_per_launch"] > 0


def test_cpu_model_is_a_string_or_none():
    m = bench.cpu_model()
    assert m is None or (isinstance(m, str) and m)
