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


def _dkdv(name):
    w = wl.WORKLOADS[name]
    x = wl.make_inputs(w, 0) if w.varlen else None
    nseg = len(x.cu_seqlens) - 1 if w.varlen else w.B
    total = x.q.shape[0] if w.varlen else 0
    S = x.max_seqlen if w.varlen else w.S
    # the rule of attn_bwd_dkdv_form, without loading the library: the
    # eight-wavefront form for causal grids of fewer than 1,024 key blocks at
    # D = 96 and 128
    blocks = w.Hkv * (total // 128 + nseg) if w.varlen else nseg * w.Hkv * ((S + 127) // 128)
    one = w.D != 64 and w.causal and blocks < 1024
    return "bwd_dkdv_kernel" if one else "bwd_dkdv4_kernel"


# Each measured workload's dominant kernel (the longest, whose roofline the
# benchmark reports), as the kernel traces under profiles/ show.
DOMINANT = {
    "mha_causal_b4_h16_s2048_d128": _dkdv,
    "gqa_causal_b2_hq32_hkv8_s4096_d128": _dkdv,
    "long_causal_b1_h16_s16384_d128_qk2": _dkdv,
    "varlen_causal_n8_l512_8192_h32_d64": _dkdv,
    "ragged_gqa_causal_n33_t16294_hq32_hkv4_d128": _dkdv,
    "mha_b4_h48_s4096_d128": _dkdv,
    "mha_causal_b4_h48_s4096_d128": _dkdv,
    "mha_causal_b4_h48_s4096_d96": _dkdv,
    "paged_prefill_causal_q892_p43676_hq24_hkv8_d128": lambda n: "fwd_kernel",
    "paged_decode_b15_nnz9625_p42784_hq24_hkv8_d128": lambda n: "decode_split_kernel",
    "gemm_bf16_nt_m8192_n7168_k5120": lambda n: "gemm_rounds_kernel",
}


@pytest.mark.parametrize("workload", sorted(DOMINANT))
def test_every_measured_workload_has_current_traffic(workload):
    """The dominant kernel of every measured workload has an HBM traffic
    record taken on the kernel's current source (so the bench line's
    roofline.traffic is not null)."""
    kernel = DOMINANT[workload](workload)
    assert f"{kernel}:{workload}" in DB, kernel
    assert bench.load_traffic(kernel, workload) is not None, (kernel, "stale source hash")


def test_dominant_kernels_agree_with_the_traces():
    """The dominant kernel named above is the longest attention kernel in
    the committed trace of the workload."""
    import re
    for workload, fn in DOMINANT.items():
        kernel = fn(workload).split("+")[0]
        path = os.path.join(ROOT, "profiles", f"kernel_trace_{workload}.md")
        rows = [l for l in open(path, encoding="utf-8") if l.startswith("| ") and "_kernel<" in l]
        avg = {re.match(r"\| (\w+)<", l).group(1): float(l.split("|")[3]) for l in rows}
        assert max(avg, key=avg.get) == kernel, (workload, avg)
