"""The committed rocprofv3 summaries describe the committed grouped-GEMM source:
bench.py reports the HBM traffic of GEMM-1 only while the source hash recorded
beside the counters matches, so a kernel change without new counters would turn
`roofline.traffic` into null.  CPU only."""
import os
import re

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_traffic_counters_match_the_gemm_source():
    assert bench.measured_traffic("mixtral4k") is not None


def test_kernel_trace_summary_names_the_current_source():
    with open(os.path.join(ROOT, "profiles", "moe_layer_mixtral4k_kernel_stats.md")) as f:
        text = f.read()
    hashes = re.findall(r"`([0-9a-f]{64})`", text)
    assert bench.gemm_source_sha256() in hashes
