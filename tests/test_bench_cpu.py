"""Host-side parts of the benchmark and the synthetic workloads (CPU only): the one-GPU contract of bench.py,
the Zipf(1.1) expert loads of the MoE configurations, the padded group offsets of the grouped operands, the
roofline constants, and the rule that a measured traffic figure is only reported for the kernel source it was
measured on."""

import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2606_20381_amd import ufp4 as U  # noqa: E402
from paper_2606_20381_amd import workloads as WL  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


@pytest.mark.parametrize("total,experts,cap", [(98304, 64, 16384), (32768, 8, None), (1000, 7, None),
                                               (640, 8, 100)])
def test_zipf_counts(total, experts, cap):
    c = np.array(WL.zipf_counts(total, experts, 1.1, cap))
    assert c.sum() == total and len(c) == experts
    assert (c >= 0).all() and (np.diff(c) <= 1).all()  # non-increasing up to the rounding of one row
    if cap is not None:
        assert c.max() <= cap
    # uncapped experts keep the Zipf ratios among themselves: load ~ rank^-1.1, up to one row of rounding
    w = np.arange(1, experts + 1, dtype=np.float64) ** -1.1
    free = c < (cap if cap is not None else total + 1)
    share = w[free] / w[free].sum() * c[free].sum()
    assert np.abs(c[free] - share).max() < 1.0


# Expected loads, computed independently by the same rule (rank^-1.1, cap with redistribution, largest
# remainder): 64 experts over 16384 x 6 routed rows with at most 16384 per expert (top-6 routing sends a token
# to an expert at most once), and 8 experts over 32768 rows.
MOE_7_9B_LOADS = [
    16384, 12773, 8177, 5959, 4662, 3815, 3220, 2780, 2442, 2175, 1958, 1780, 1630, 1502, 1392, 1297, 1213, 1139,
    1073, 1015, 962, 914, 870, 830, 794, 760, 729, 701, 674, 649, 626, 605, 585, 566, 548, 531, 516, 501, 487, 473,
    461, 449, 437, 426, 416, 406, 396, 387, 379, 370, 362, 355, 347, 340, 333, 327, 321, 314, 309, 303, 298, 292,
    287, 282]
MOE_124B_LOADS = [13047, 6087, 3897, 2839, 2221, 1818, 1534, 1325]


def test_moe_configurations_loads():
    assert WL.zipf_counts(16384 * 6, 64, 1.1, 16384) == MOE_7_9B_LOADS
    assert WL.zipf_counts(32768, 8, 1.1, None) == MOE_124B_LOADS
    # ragged shapes: almost no expert's rows are a multiple of 16, so padding is exercised everywhere
    assert sum(c % 16 != 0 for c in MOE_7_9B_LOADS) == 61 and all(c % 16 for c in MOE_124B_LOADS)


def test_group_offsets_pad_each_group_to_16():
    off, red = U.group_offsets([0, 1, 16, 17, 33], device="cpu")
    assert off.tolist() == [0, 0, 1, 17, 34, 67]
    assert U.padded_offsets(off.tolist()) == [0, 0, 16, 32, 64, 112]
    assert red == 112


def test_roofline_constants():
    # two 32-cycle MFMAs per 32 x 32 tile and 16-block: 32768 ops per 64 cycles per SIMD, 1024 SIMDs at 2.4 GHz
    assert bench.ATTAINABLE_TOPS == pytest.approx(32768 / 64 * 1024 * 2.4e9 / 1e12)
    assert bench.ATTAINABLE_TOPS == pytest.approx(1258.29, abs=0.01)
    assert bench.QUANT_BYTES_PER_ELEM == 2 + 0.5 + 0.25  # bf16 in, 4-bit code and a fp32 scale per 16 out
    assert bench.DUAL_BYTES_PER_ELEM == 2 + 2 * (0.5 + 0.25)
    # the 1 GiB quantizer tensor at the HBM peak: 1.476 GB in 184.5 us; 70% of the peak is 264 us
    t = 32768 * 16384 * bench.QUANT_BYTES_PER_ELEM / (bench.HBM_PEAK_GBPS * 1e9)
    assert t * 1e6 == pytest.approx(184.5, abs=0.1)


def test_traffic_is_reported_only_for_the_measured_source(tmp_path, monkeypatch):
    good = bench._source_digest("ufp4_quant.hip")
    table = {"quant": {"w-good": {"source_sha256": good, "bytes_per_launch": 123},
                       "w-stale": {"source_sha256": "0" * 64, "bytes_per_launch": 456}}}
    path = tmp_path / "traffic.json"
    path.write_text(json.dumps(table))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(path))
    assert bench.measured_traffic("quant", "w-good") == 123
    assert bench.measured_traffic("quant", "w-stale") is None
    assert bench.measured_traffic("quant", "w-missing") is None
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "absent.json"))
    assert bench.measured_traffic("quant", "w-good") is None


def test_committed_traffic_entries_name_known_sources():
    with open(os.path.join(ROOT, "profiles", "traffic.json")) as f:
        table = json.load(f)
    for kind, entries in table.items():
        if kind.startswith("_"):
            continue
        assert kind in bench.TRAFFIC_SOURCES
        for name, e in entries.items():
            assert len(e["source_sha256"]) == 64 and e["bytes_per_launch"] > 0, name


def test_source_digest_ignores_comments_only(tmp_path, monkeypatch):
    src = tmp_path / "paper_2606_20381_amd" / "csrc"
    src.mkdir(parents=True)
    (src / "k.hip").write_text("// header\nint f(int a) { return a + 1; }  /* block\n comment */\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    d0 = bench._source_digest("k.hip")
    (src / "k.hip").write_text("// another header, longer\n\nint f(int a) {   return a + 1; }\n// trailing note\n")
    assert bench._source_digest("k.hip") == d0
    (src / "k.hip").write_text("// header\nint f(int a) { return a + 2; }\n")
    assert bench._source_digest("k.hip") != d0
