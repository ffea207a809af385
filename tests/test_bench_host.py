"""Host logic of bench.py (no GPU): the kernel classes its counter summary
sorts rocprofv3 names into, the conversion of FETCH_SIZE / WRITE_SIZE counts
into HBM bytes per launch through a plain copy of known size, the source-hash
gate on the stored traffic, and the one-GPU guard."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]


def _counter_folder(path, rows):
    """A rocprofv3 --pmc -f csv output folder holding (kernel name, value) rows."""
    os.makedirs(os.path.join(path, "host", "1"), exist_ok=True)
    with open(os.path.join(path, "host", "1", "run_counter_collection.csv"), "w",
              newline="") as fh:
        w = csv.DictWriter(fh, FIELDS)
        w.writeheader()
        for i, (name, v) in enumerate(rows):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": name, "Counter_Name": "X",
                        "Counter_Value": v})
    return str(path)


FUSED = "void wd::k_gemm_bf16_fused<2, 3, 4, false, 6, 4, 4>(unsigned short const*, int)"
SPLIT = "void wd::k_gemm_bf16<1, 3, 8, 8, false>(unsigned short const*, int)"
DMA = "void wd::k_gemm_bf16_dma<3, 4, true, 12, 6>(unsigned short const*, int)"
BIG = "void wd::k_gemm_bf16_big<2, false>(unsigned short const*, int)"
ATTN = "wd::k_attn_bf16(unsigned short const*, int)"
COMBINE = "wd::k_attn_combine(float const*, int)"
COPY = "__amd_rocclr_copyBuffer"


def test_kernel_classes():
    assert bench.kernel_class_of(FUSED) == 1
    assert bench.kernel_class_of(SPLIT) == 1
    assert bench.kernel_class_of(DMA) == 2
    assert bench.kernel_class_of(BIG) == 2
    assert bench.kernel_class_of(ATTN) == 4
    assert bench.kernel_class_of(COMBINE) == 4
    assert bench.starts_unit(ATTN) and not bench.starts_unit(COMBINE) and bench.starts_unit(DMA)
    assert bench.kernel_class_of(COPY) is None


def test_pmc_summary_scales_counts_by_the_copy(tmp_path, monkeypatch):
    traffic = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(traffic))
    # a 1 MiB copy reads 2048 and writes 1024 counts: 512 and 1024 bytes per count
    cf = _counter_folder(tmp_path / "cf", [(COPY, 2048.0), (COPY, 2048.0)])
    cw = _counter_folder(tmp_path / "cw", [(COPY, 1024.0)])
    # two attention units: one with a split merge, one without
    gf = _counter_folder(tmp_path / "gf", [(FUSED, 100.0), (SPLIT, 300.0), (DMA, 1000.0),
                                           (ATTN, 7.0), (COMBINE, 3.0), (ATTN, 5.0)])
    gw = _counter_folder(tmp_path / "gw", [(FUSED, 2.0), (SPLIT, 6.0), (DMA, 40.0),
                                           (ATTN, 1.0), (COMBINE, 2.0), (ATTN, 1.0)])
    bench.pmc_summary(gf, gw, cf, cw, copy_mib=1)
    rec = json.loads(traffic.read_text())
    assert rec["fetch_bytes_per_count"] == 512.0 and rec["write_bytes_per_count"] == 1024.0
    few, many = rec["kernels"]["k_gemm_bf16"], rec["kernels"]["k_gemm_bf16_dma"]
    attn = rec["kernels"]["k_attn_bf16"]
    assert few["source_sha256_16"] == bench.source_hash("k_gemm_bf16")
    assert attn["source_sha256_16"] == bench.source_hash("k_attn_bf16")
    assert few["dispatches"] == 2 and many["dispatches"] == 1
    assert few["hbm_fetch_bytes_per_launch"] == round((100 + 300) / 2 * 512)
    assert few["hbm_write_bytes_per_launch"] == round((2 + 6) / 2 * 1024)
    assert many["hbm_bytes_per_launch"] == round(1000 * 512 + 40 * 1024)
    assert attn["units"] == 2 and attn["dispatches"] == 3
    assert attn["hbm_bytes_per_launch"] == round((7 + 3 + 5) / 2 * 512 + (1 + 2 + 1) / 2 * 1024)


def test_pmc_summary_rejects_unpaired_runs(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    cf = _counter_folder(tmp_path / "cf", [(COPY, 2048.0)])
    cw = _counter_folder(tmp_path / "cw", [(COPY, 1024.0)])
    gf = _counter_folder(tmp_path / "gf", [(FUSED, 100.0), (FUSED, 100.0)])
    gw = _counter_folder(tmp_path / "gw", [(FUSED, 2.0)])
    with pytest.raises(SystemExit):
        bench.pmc_summary(gf, gw, cf, cw, copy_mib=1)


def test_traffic_only_for_the_profiled_source(tmp_path, monkeypatch):
    traffic = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(traffic))
    rec = {"kernels": {"k_gemm_bf16": {"hbm_bytes_per_launch": 123,
                                       "source_sha256_16": bench.source_hash("k_gemm_bf16")},
                       "k_attn_bf16": {"hbm_bytes_per_launch": 77,
                                       "source_sha256_16": bench.source_hash("k_attn_bf16")}}}
    traffic.write_text(json.dumps(rec))
    assert bench.measured_traffic("k_gemm_bf16") == 123
    assert bench.measured_traffic("k_attn_bf16") == 77
    assert bench.measured_traffic("k_gemm_bf16_dma") is None
    rec["kernels"]["k_gemm_bf16"]["source_sha256_16"] = "0" * 16
    traffic.write_text(json.dumps(rec))
    assert bench.measured_traffic("k_gemm_bf16") is None
    assert bench.measured_traffic("k_attn_bf16") == 77
    traffic.write_text("not json")
    assert bench.measured_traffic("k_gemm_bf16") is None


def test_more_than_one_gpu_is_refused():
    env = dict(os.environ)
    env.pop("WORLD_SIZE", None)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""
