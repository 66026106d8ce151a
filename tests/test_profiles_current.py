"""The committed rocprofv3 summaries describe the committed grouped-GEMM source:
bench.py reports the L2-egress traffic of GEMM-1 only while the source hash
recorded beside the counters matches, so a kernel change without new counters
would turn `roofline.traffic` into null.  CPU only."""
import os
import re

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_traffic_counters_match_the_gemm_source():
    # the workload bench.py measures by default
    assert bench.measured_traffic("memconstrained") is not None


def test_rocprof_summary_names_the_current_source():
    with open(os.path.join(ROOT, "profiles", "moe_layer_memconstrained_rocprof.md")) as f:
        text = f.read()
    hashes = re.findall(r"source_sha256: ([0-9a-f]{64})", text)
    assert bench.gemm_source_sha256() in hashes
