"""The stored HBM traffic records that bench.py quotes as roofline.traffic.

Each record in profiles/traffic.json is keyed "kernel:workload" and holds the
FETCH_SIZE / WRITE_SIZE counters of one launch (or one call of a kernel pair)
scaled by the device-copy calibration, plus the hash of the kernel source it
was taken on.  These checks run on the CPU: the keys name kernels whose source
bench.py can hash and workloads it can run, the byte fields agree with each
other and with the counters and scales, and the headline's dominant kernel has
a record.
"""
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2608_17379_amd import workloads as wl  # noqa: E402


with open(os.path.join(ROOT, "profiles", "traffic.json"), encoding="utf-8") as f:
    DB = json.load(f)

KNOWN = set(wl.WORKLOADS) | set(wl.PAGED_WORKLOADS) | set(wl.GEMM_WORKLOADS)


def _kib(v):
    return sum(v.values()) if isinstance(v, dict) else v


@pytest.mark.parametrize("key", sorted(DB))
def test_record_is_consistent(key):
    kernel, workload = key.split(":")
    rec = DB[key]
    assert kernel in bench.KERNEL_SOURCES
    assert workload in KNOWN
    assert len(rec["source_sha"]) == 16
    assert rec["read_bytes"] > 0 and rec["write_bytes"] > 0
    assert abs(rec["read_bytes"] + rec["write_bytes"] - rec["bytes_per_launch"]) <= 2
    assert rec["read_bytes"] == pytest.approx(_kib(rec["fetch_kib"]) * 1024 * rec["fetch_scale"],
                                              rel=1e-3)
    assert rec["write_bytes"] == pytest.approx(_kib(rec["write_kib"]) * 1024 * rec["write_scale"],
                                               rel=1e-3)


def test_headline_kernels_have_records():
    for kernel in ("fwd_kernel", "bwd_dq_kernel", "bwd_dkdv4_kernel"):
        assert f"{kernel}:{wl.HEADLINE}" in DB


@pytest.mark.parametrize("kernel", sorted(bench.KERNEL_SOURCES))
def test_hashed_sources_follow_includes(kernel):
    """The source hash that ties a record to the code covers the kernel's
    file and every package header it includes, directly or not."""
    files = bench.kernel_source_files(kernel)
    csrc = os.path.join(ROOT, "paper_2608_17379_amd", "csrc")
    assert files[0] == bench.KERNEL_SOURCES[kernel]
    for name in files:
        for line in open(os.path.join(csrc, name), encoding="utf-8"):
            line = line.strip()
            if line.startswith('#include "'):
                inc = line.split('"')[1]
                if os.path.exists(os.path.join(csrc, inc)):
                    assert inc in files, (kernel, name, inc)
    assert "device_common.hpp" in files and "attn_kernels.hpp" in files
