"""Host-side logic of bench.py (no GPU): the FLOP counts behind the reported
throughput, the rocprofv3 summary (MFMA busy fractions), the attention HBM
traffic file and its source-hash guard, and the one-GPU guard."""
import csv
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

ATTN = "hsa::(anonymous namespace)::attention_bf16_kernel<128, 8, false>(...)"
COPY = "__amd_rocclr_copyBuffer"


def _counter_csv(path, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (kernel, counter, value) in enumerate(rows):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": kernel, "Counter_Name": counter, "Counter_Value": value})


def test_flop_counts():
    # QK^T and PV, 2 FLOPs per MAC each: 4 |A| N d; the Wan-14B block at 25% active
    assert bench.attention_flops(8190, 32760, 5120) == 4 * 8190 * 32760 * 5120 == 5494874112000
    # Q, K, V (3 d^2 MACs) and the output projection (d^2) per active row
    assert bench.gemm_flops(8190, 5120) == 2 * 8190 * 4 * 5120 * 5120


def test_summary_mfma_busy(tmp_path):
    # two dispatches of a matrix kernel: busy cycles over (1024 SIMDs x GRBM_GUI_ACTIVE / 8 XCDs)
    _counter_csv(str(tmp_path / "p" / "run_counter_collection.csv"), [
        (ATTN, "SQ_VALU_MFMA_BUSY_CYCLES", 1024 * 500), (ATTN, "GRBM_GUI_ACTIVE", 8 * 1000),
        (ATTN, "SQ_VALU_MFMA_BUSY_CYCLES", 1024 * 250), (ATTN, "GRBM_GUI_ACTIVE", 8 * 1000),
        (COPY, "SQ_VALU_MFMA_BUSY_CYCLES", 0), (COPY, "GRBM_GUI_ACTIVE", 8 * 10),
    ])
    lines = bench.summarize(str(tmp_path)).splitlines()
    text = "\n".join(lines)
    k = next(i for i, line in enumerate(lines) if line.startswith("MFMA busy per dispatch"))
    busy = lines[k + 1:]
    assert len(busy) == 1, text  # the copy never used the matrix pipes: not listed
    assert busy[0].split()[:2] == ["0.500", "0.250"]
    means = bench.counter_means(str(tmp_path))
    assert means[(ATTN, "SQ_VALU_MFMA_BUSY_CYCLES")] == (1024 * 375, 2)


def test_traffic_file_scales_and_hash_guard(tmp_path, monkeypatch):
    d = tmp_path / "passes"
    # attention: 100 KiB fetched (counter units), 50 KiB written per dispatch; the 1 GiB copy reads
    # FETCH_SIZE 0.5 GiB and WRITE_SIZE 1 GiB, so fetches scale by 2 and writes by 1
    _counter_csv(str(d / "attn_fetch" / "run_counter_collection.csv"), [(ATTN, "FETCH_SIZE", 100)] * 3)
    _counter_csv(str(d / "attn_write" / "run_counter_collection.csv"), [(ATTN, "WRITE_SIZE", 50)] * 3)
    _counter_csv(str(d / "copy_fetch" / "run_counter_collection.csv"),
                 [(COPY, "FETCH_SIZE", 4), (COPY, "FETCH_SIZE", 512 * 1024)])
    _counter_csv(str(d / "copy_write" / "run_counter_collection.csv"),
                 [(COPY, "WRITE_SIZE", 8), (COPY, "WRITE_SIZE", 1024 * 1024)])
    out = tmp_path / "traffic.txt"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(out))
    text = bench.write_traffic(str(d))
    assert "fetch_scale: 2.0000" in text and "write_scale: 1.0000" in text
    assert bench.traffic_from_profile("wan14b", "scattered", 1) == 100 * 1024 * 2 + 50 * 1024
    # only the launch the counters measured
    assert bench.traffic_from_profile("wan14b", "scattered", 2) is None
    assert bench.traffic_from_profile("wan14b", "contiguous", 1) is None
    # a different kernel source voids the figure
    out.write_text(text.replace("kernel_source_sha256: ", "kernel_source_sha256: 0"))
    assert bench.traffic_from_profile("wan14b", "scattered", 1) is None


def test_committed_traffic_matches_the_current_attention_source():
    # the committed counter summary was taken on this kernel source (else the bench reports no traffic)
    assert bench.traffic_from_profile("wan14b", "scattered", 1) is not None


@pytest.mark.parametrize("n", [2, 8])
def test_more_than_one_gpu_is_refused(n):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
