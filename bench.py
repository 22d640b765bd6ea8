#!/usr/bin/env python3
"""Throughput of fused attention forward + backward on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME]

Without --workload it measures the headline workload (B4 H16 S2048 D128
causal).  The paged-cache workloads (paged prefill, paged decode) are forward
only, as in the paper: their step is one attn_fwd_paged call (TFLOP/s; a
prefill far too small to fill the chip is split into key chunks, and the
call's forward and merge kernels are timed together for the roofline) or one
attn_decode_paged call (its split and merge kernels; HBM GB/s, with the
roofline against 8 TB/s since decode reads each key and value once).  The
GEMM workload's step is one attn_gemm_bf16_nt call (2 M N K FLOP).

A step is one forward (attn_fwd) and one backward (attn_bwd_phases with the
Delta/dQ phase, then the dK/dV phase: together exactly attn_bwd) over one
batch of seeded synthetic bf16 inputs already resident in HBM.  After a
five-step probe and W untimed warm-up steps, K steps are timed
("at_requested_warmup", the paper's fixed warm-up count); more back-to-back
steps then run until --warmup-seconds (default 1 s) have passed since the
probe, because the GPU's clock and power management take about a second of
sustained load to settle, and K more steps are timed: that pass is `value`
(the JSON's "warmup" is the count run before it, "warmup_requested" the W
asked for).  "median" is the median per-step time of a further pass with an
event between consecutive steps.  When the host cannot enqueue steps faster
than the GPU runs them (the microsecond-scale paged and small workloads),
the GPU first runs a spin kernel long enough for the host to enqueue all K
steps of a pass, so that they run back to back and the timing is the GPU's,
not the host's launch rate; otherwise a pass's start event is recorded
behind the steps before it, with the launch queue still full.  The timed
passes carry no events inside their steps; a last pass of K steps, not part
of `value`, records an event around every launch for the per-kernel times.
One JSON line is printed.

Two secondary objects: "cold" (fwd+bwd workloads) is the median of
--cold-steps single steps, each started after a 512 MiB write has flushed the
L2 caches and the MALL (the write is not timed); "gpu_state" is the graphics
clock (mean over the XCDs), hotspot temperature and socket power sampled
through amdsmi during an untimed pass of --state-seconds of back-to-back
steps after the timed ones (null when amdsmi is not usable).

FLOP convention: forward 4*B*Hq*S^2*D (halved when causal; packed input sums
L^2 over sequences), backward 2.5x forward.  TFLOP/s = (forward + backward
FLOP) / step time.  Peak: 2516.6 TFLOP/s dense bf16 MFMA (256 CUs x 2.4 GHz
x 4096 FLOP/clock/CU).

The roofline object is for the kernel with the largest average duration.
Each kernel's average duration comes from HIP events recorded between the
launches of the last pass (all on the stream the library launches on).  Its
bound is the roof the kernel's algorithmic work meets first: the MFMA roof
(FLOP / 2516.6 TFLOP/s) or the HBM roof (algorithmic bytes / 8 TB/s, every
input read and every output written once); `achieved` is that work per
second and `frac` its fraction of the roof.
Per-launch algorithmic FLOP of each kernel (the backward's 2.5 F are its
five S^2 D products: the recomputed S, dP, dV, dK and dQ):
  fwd_kernel       2 GEMMs  (S = QK^T, O = PV)            = F
  dK/dV kernel     4 GEMMs  (S, dP = dO V^T, dV = P^T dO, dK = dS^T Q) = 2 F
                   (bwd_dkdv4_kernel or bwd_dkdv_kernel, the form the library
                   picks for the workload, attn_bwd_dkdv_form)
  bwd_dq_kernel    1 GEMM   (dQ = dS K)                   = 0.5 F
with F the forward FLOP above.  The dQ kernel also recomputes S and dP (it
executes 3 GEMMs, 1.5 F, of MFMA work); "kernel_tflops" gives each kernel's
algorithmic and executed rates.  `traffic` (HBM bytes per launch from
rocprofv3 FETCH_SIZE + WRITE_SIZE, scaled by a copy-kernel calibration) is
read from profiles/traffic.json when that file was taken on the current
kernel source (comments aside), else null.

The CPU baseline times the fp64 oracle (test infrastructure, used here only
for this leg) on a bounded sample of the same workload: whole (batch, head)
slices, forward + backward, until about --cpu-seconds have elapsed, on every
usable host thread (the CPU affinity, capped by OMP_NUM_THREADS when set),
with the thread count and the CPU model in the record.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6
PEAK_HBM_GBS = 8000.0
METRIC = "attention fwd/bwd TFLOP/s + % bf16 MFMA peak, B4 H16 S2048 D128 causal"
# S^2 D products per launch (each 2 S^2 D FLOP per head, halved when causal):
# algorithmic (the FLOP convention) and executed (MFMA work actually issued).
GEMMS = {"fwd_kernel": 2, "bwd_dq_kernel": 1, "bwd_dkdv_kernel": 4, "bwd_dkdv4_kernel": 4}
GEMMS_EXECUTED = {"fwd_kernel": 2, "bwd_dq_kernel": 3, "bwd_dkdv_kernel": 4,
                  "bwd_dkdv4_kernel": 4}
# --dkdv-form names -> the attn_bwd_phases bit (include/attn.h), and each
# bit's kernel.
DKDV_FORMS = {"auto": 0, "one_per_cu": 4, "two_per_cu": 8}
DKDV_KERNELS = {4: "bwd_dkdv_kernel", 8: "bwd_dkdv4_kernel"}
RIDGE = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)   # FLOP per byte at both roofs
KERNEL_SOURCES = {"fwd_kernel": "attn_fwd.hip", "fwd_kernel+fwd_merge_kernel": "attn_fwd.hip",
                  "bwd_dq_kernel": "attn_bwd.hip",
                  "bwd_dkdv_kernel": "attn_bwd.hip", "bwd_dkdv4_kernel": "attn_bwd.hip",
                  "decode_split_kernel": "attn_decode.hip",
                  "decode_merge_kernel": "attn_decode.hip", "gemm_rounds_kernel": "gemm.hip"}


def fwd_flops(w, cu_seqlens=None) -> float:
    """4 * Hq * D * sum(L^2) (x1/2 causal), as in the module docstring."""
    if cu_seqlens is not None:
        sq = sum((b - a) ** 2 for a, b in zip(cu_seqlens, cu_seqlens[1:]))
        f = 4.0 * w.Hq * w.D * sq
    else:
        f = 4.0 * w.B * w.Hq * w.S * w.S * w.D
    return f * (0.5 if w.causal else 1.0)


def kernel_source_files(kernel: str) -> list:
    """The kernel's source file followed by every header of the package it
    includes (#include "..."), transitively, in first-inclusion order: an
    edit to any of them changes the compiled kernel."""
    csrc = os.path.join(ROOT, "paper_2608_17379_amd", "csrc")
    order, todo = [], [KERNEL_SOURCES[kernel]]
    while todo:
        name = todo.pop(0)
        if name in order:
            continue
        order.append(name)
        for line in open(os.path.join(csrc, name), encoding="utf-8"):
            line = line.strip()
            if line.startswith("#include \""):
                inc = line.split('"')[1]
                if os.path.exists(os.path.join(csrc, inc)):
                    todo.append(inc)
    return order


def source_sha(kernel: str) -> str:
    """Hash of the kernel's source and its package headers with comments and
    blank lines removed, so that a recorded traffic figure survives
    comment-only edits but not a change of the compiled code."""
    csrc = os.path.join(ROOT, "paper_2608_17379_amd", "csrc")
    code = []
    for name in kernel_source_files(kernel):
        code.append(f"// file {name}")
        for line in open(os.path.join(csrc, name), encoding="utf-8"):
            line = line.split("//", 1)[0].rstrip()
            if line:
                code.append(line)
    return hashlib.sha256("\n".join(code).encode()).hexdigest()[:16]


def load_traffic(kernel: str, workload: str):
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        rec = json.load(open(path))[f"{kernel}:{workload}"]
    except (OSError, KeyError, ValueError):
        return None
    if rec.get("source_sha") != source_sha(kernel):
        return None
    return rec.get("bytes_per_launch")


def attention_bytes(kernel: str, w, x) -> float:
    """Algorithmic HBM bytes of one launch: every input read once and every
    output written once (bf16 rows of D values, fp32 per-row values).
      fwd_kernel        reads Q, K, V; writes O, LSE
      bwd_dq_kernel     reads Q, K, V, O, dO, LSE; writes dQ, Delta, LSE log2 e
      dK/dV kernels     reads Q, K, V, dO, Delta, LSE log2 e; writes dK, dV"""
    rows = x.q.shape[0] if w.varlen else w.B * w.S
    nq, nkv = rows * w.Hq, rows * w.Hkv     # (row, head) pairs
    row = w.D * 2
    if kernel == "fwd_kernel":
        return 2 * nq * row + 2 * nkv * row + 4 * nq
    if kernel == "bwd_dq_kernel":
        return 4 * nq * row + 2 * nkv * row + 3 * 4 * nq
    return 2 * nq * row + 4 * nkv * row + 2 * 4 * nq


def roofline(kernel: str, flop: float, nbytes: float, ms: float, workload: str,
             hbm_work: bool = False) -> dict:
    """Roofline object of one kernel.  The bound is the roof its algorithmic
    work meets first: MFMA (flop / 2516.6 TFLOP/s) or HBM (bytes / 8 TB/s);
    `hbm_work` reports an HBM-bound kernel's rate in GB/s of its algorithmic
    bytes.  `traffic` is the measured HBM bytes per launch (None unless the
    counters were taken on the current source), with the HBM rate they imply."""
    hbm = hbm_work or nbytes / (PEAK_HBM_GBS * 1e9) > flop / (PEAK_BF16_TFLOPS * 1e12)
    if hbm:
        ach, peak, unit = nbytes / (ms * 1e-3) / 1e9, PEAK_HBM_GBS, "GB/s"
    else:
        ach, peak, unit = flop / (ms * 1e-3) / 1e12, PEAK_BF16_TFLOPS, "TFLOP/s"
    traffic = load_traffic(kernel, workload)
    out = {"kernel": kernel, "bound": "hbm" if hbm else "mfma", "achieved": round(ach, 2),
           "peak": peak, "unit": unit, "frac": round(ach / peak, 4), "traffic": traffic,
           "algorithmic_bytes": round(nbytes)}
    if flop:
        out["arith_intensity"] = round(flop / nbytes, 1)
    if traffic:
        out["traffic_hbm_frac"] = round(traffic / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)
    return out


def host_cpu() -> dict:
    """Host threads the CPU leg may use (the process's CPU affinity, capped
    by OMP_NUM_THREADS when that is set, as it is where the host is shared)
    and the CPU model (/proc/cpuinfo, the source lscpu reads)."""
    cpus = len(os.sched_getaffinity(0))
    n = cpus
    omp = os.environ.get("OMP_NUM_THREADS", "")
    if omp.isdigit() and int(omp) > 0:
        n = min(n, int(omp))
    model = None
    try:
        for line in open("/proc/cpuinfo", encoding="utf-8"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"threads": n, "affinity_cpus": cpus, "model": model}


class cpu_threads:
    """Run the CPU leg on every usable host thread (host_cpu()), then
    restore torch's thread count."""

    def __enter__(self):
        import torch
        self.saved = torch.get_num_threads()
        self.info = host_cpu()
        torch.set_num_threads(self.info["threads"])
        return self

    def __exit__(self, *exc):
        import torch
        torch.set_num_threads(self.saved)
        return False

    def fields(self) -> dict:
        import torch
        return {"cores": torch.get_num_threads(), "cpu_model": self.info["model"],
                "affinity_cpus": self.info["affinity_cpus"]}


def cpu_baseline(w, x, seconds: float):
    """Oracle (fp64, CPU) forward + backward on whole head slices."""
    import torch
    import oracle
    n_done, flop, t0 = 0, 0.0, time.perf_counter()
    G = w.Hq // w.Hkv
    slices = [(b, g) for b in range(w.B) for g in range(w.Hkv)] if not w.varlen else \
        [(s, g) for s in range(w.B) for g in range(w.Hkv)]
    # Whole passes over the slices are repeated until the time budget is
    # spent (a small workload's full pass can take well under a second).
    passes = 0
    while n_done == 0 or time.perf_counter() - t0 < seconds:
        for seg, g in slices:
            hs = list(range(g * G, (g + 1) * G))
            if w.varlen:
                a, b = x.cu_seqlens[seg], x.cu_seqlens[seg + 1]
                q, k, v, do = x.q[a:b, hs], x.k[a:b, [g]], x.v[a:b, [g]], x.do[a:b, hs]
                cu = [0, b - a]
                f = 4.0 * G * w.D * (b - a) ** 2 * (0.5 if w.causal else 1.0)
            else:
                q, k, v, do = (x.q[seg:seg + 1, hs], x.k[seg:seg + 1, [g]],
                               x.v[seg:seg + 1, [g]], x.do[seg:seg + 1, hs])
                cu = None
                f = 4.0 * G * w.S * w.S * w.D * (0.5 if w.causal else 1.0)
            oracle.attention_forward(q, k, v, w.causal, w.scale, cu_seqlens=cu)
            oracle.attention_backward(q, k, v, do, w.causal, w.scale, cu_seqlens=cu)
            n_done += 1
            flop += 3.5 * f
            if time.perf_counter() - t0 >= seconds:
                break
        passes += 1
    dt = time.perf_counter() - t0
    return {
        "value": round(flop / dt / 1e12, 6),
        "unit": "TFLOP/s",
        "cores": torch.get_num_threads(),
        "kind": "oracle",
        "flop_convention": "fwd + bwd = 3.5 x the forward's causal-halved FLOP",
        "sample": f"{n_done} key/value-head slices ({G} query heads each; {len(slices)} per "
                  f"pass, {passes} pass(es)) of {w.name}, fp64 forward + backward, {dt:.1f} s",
    }


def hold_gpu_for_enqueue(host_ms_per_step: float, steps: int) -> None:
    """Occupy the GPU with torch's spin kernel for longer than the host needs
    to enqueue `steps` steps, so that the timed steps then run back to back:
    the HIP events between launches measure the kernels, not the host's
    launch rate (which matters for microsecond-scale kernels)."""
    import torch
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    torch.cuda._sleep(1_000_000)
    b.record()
    torch.cuda.synchronize()
    cycles_per_ms = 1_000_000 / max(a.elapsed_time(b), 1e-3)
    want_ms = min(2000.0, 1.0 + 1.5 * host_ms_per_step * steps)
    torch.cuda._sleep(int(cycles_per_ms * want_ms))


class GpuMonitor:
    """Samples the GPU's firmware metrics through amdsmi in a background
    thread: graphics clock (MHz, mean over the XCDs), memory, fabric and SoC
    clocks where the firmware reports them, hotspot temperature (C) and
    socket power (W).  The firmware refreshes them every few hundred
    milliseconds, so they describe a sustained run, not a short one.
    Monitoring never fails the benchmark: without amdsmi, or when a query
    fails, the summary is None or lacks that field."""

    def __init__(self, period_s: float = 0.01):
        self.period = period_s
        self.samples = []   # (gfx activity %, {quantity: value})
        self._stop = None
        self._thread = None
        self._smi = None
        self._h = None

    def _sample(self):
        try:
            m = self._smi.amdsmi_get_gpu_metrics_info(self._h)
        except Exception:
            return
        clks = m.get("current_gfxclks")
        if isinstance(clks, list):
            clks = [c for c in clks if isinstance(c, (int, float)) and 0 < c < 10000]
        vals = {"sclk_mhz": sum(clks) / len(clks) if clks else m.get("current_gfxclk"),
                "temp_c": m.get("temperature_hotspot"), "power_w": m.get("current_socket_power")}
        for key, name in (("uclk_mhz", "current_uclk"), ("fclk_mhz", "current_fclk"),
                          ("socclk_mhz", "current_socclk")):
            v = m.get(name)
            if isinstance(v, list):
                v = [c for c in v if isinstance(c, (int, float)) and 0 < c < 10000]
                v = sum(v) / len(v) if v else None
            vals[key] = v
        if vals.get("fclk_mhz") is None:
            try:   # the fabric clock's current DPM level, where the table lacks it
                f = self._smi.amdsmi_get_clk_freq(self._h, self._smi.AmdSmiClkType.DF)
                vals["fclk_mhz"] = f["frequency"][f["current"]] / 1e6
            except Exception:
                pass
        act = m.get("average_gfx_activity")
        self.samples.append((act if isinstance(act, (int, float)) else None,
                             {k: float(v) for k, v in vals.items()
                              if isinstance(v, (int, float)) and v == v}))

    def __enter__(self):
        import threading
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            self._smi = amdsmi
            self._h = amdsmi.amdsmi_get_processor_handles()[0]
        except Exception:
            self._smi = None
            return self
        self._stop = threading.Event()

        def loop():
            while not self._stop.is_set():
                self._sample()
                self._stop.wait(self.period)
        self._thread = threading.Thread(target=loop, daemon=True)
        self._thread.start()
        return self

    def __exit__(self, *exc):
        if self._thread is not None:
            self._stop.set()
            self._thread.join()
        if self._smi is not None:
            try:
                self._smi.amdsmi_shut_down()
            except Exception:
                pass
        return False

    def summary(self):
        """Mean, min and max of each quantity over the samples in which the
        firmware reports the graphics engine at least half busy (the table
        lags the load by a few hundred milliseconds)."""
        if self._smi is None:
            return None
        busy = [v for a, v in self.samples if a is not None and a >= 50]
        out = {"busy_samples": len(busy), "samples": len(self.samples)}
        for key in ("sclk_mhz", "uclk_mhz", "fclk_mhz", "socclk_mhz", "temp_c", "power_w"):
            v = [d[key] for d in busy if key in d]
            if v:
                out[key] = {"mean": round(sum(v) / len(v), 1), "min": min(v), "max": max(v)}
        return out


def sustained_state(step, seconds: float):
    """Run steps back to back for about `seconds` while sampling the GPU's
    clock, temperature and power; returns GpuMonitor.summary() (not part of
    any timed figure)."""
    import torch
    if seconds <= 0:
        return None
    with GpuMonitor() as mon:
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < seconds:
            for _ in range(10):
                step()
            torch.cuda.synchronize()
    return mon.summary()


def cold_steps(step, steps: int, flush_bytes: int = 512 << 20):
    """Median time per step (ms) of `steps` single steps, each after a write
    of `flush_bytes` (more than the L2 caches and the 256 MB MALL hold) that
    is outside the timed events: every step starts with cold caches."""
    import torch
    buf = torch.empty(flush_bytes, dtype=torch.uint8, device="cuda")
    times = []
    for i in range(steps):
        buf.fill_(i & 0xFF)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        step()
        b.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b))
    del buf
    times.sort()
    return times[len(times) // 2]


def time_steps(step, n_kernels: int, steps: int, warmup: int, warmup_seconds: float = 1.0):
    """Warm up and time `steps` steps several ways.  `step(ev)` records ev[0]
    before its first launch and ev[1 + i] after launch i.

      * "early": `warmup` untimed steps (after a five-step probe), then
        `steps` timed steps: the paper's protocol of a fixed warm-up count.
      * "settled" (the reported value): more back-to-back steps until
        `warmup_seconds` have passed since the probe, then `steps` timed
        steps.  The GPU's clock and power management take about a second of
        sustained load to settle; steps timed earlier run up to 12 % slower.
      * "median": the median of `steps` per-step times, from an event
        recorded between consecutive steps of a further pass (the paper
        reports the median of its timed runs).
      * per-kernel times: a last pass records an event around every launch.

    Each timed pass has no events inside its steps (except the median and
    per-kernel passes, as stated).  If the host enqueues a step in less than
    half the time the GPU takes to run it, a pass's start event is recorded
    right behind the steps before it, with the queue still full, so that it
    starts on a busy GPU; otherwise the GPU is first held by a spin kernel
    while the host enqueues the pass, so that the timing is the GPU's and
    not the host's launch rate.
    Returns a dict: ms_step (settled), early_ms, median_ms, kern (ms per
    launch i), warmed (warm-up steps run before the settled pass),
    early_warmup (before the early pass)."""
    import torch
    # Host enqueue rate against GPU rate, on a few steps that cannot fill the
    # launch queue (once it is full, enqueueing waits for the GPU).
    torch.cuda.synchronize()
    t_probe = time.perf_counter()
    probe = 5
    for _ in range(probe):
        step()
    host_ms = (time.perf_counter() - t_probe) * 1e3 / probe
    torch.cuda.synchronize()
    gpu_ms = (time.perf_counter() - t_probe) * 1e3 / probe
    hold = host_ms >= 0.5 * gpu_ms

    def begin():
        if hold:
            torch.cuda.synchronize()
            hold_gpu_for_enqueue(host_ms, steps)
        ev = torch.cuda.Event(enable_timing=True)
        ev.record()
        return ev

    def timed_pass():
        start, end = begin(), torch.cuda.Event(enable_timing=True)
        for _ in range(steps):
            step()
        end.record()
        torch.cuda.synchronize()
        return start.elapsed_time(end) / steps

    done = probe
    for _ in range(warmup):
        step()
        done += 1
    early_warmup = done
    early_ms = timed_pass()
    done += steps
    while done < warmup or time.perf_counter() - t_probe < warmup_seconds:
        step()
        done += 1
    ms_step = timed_pass()

    marks = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    marks[0] = begin()
    for i in range(steps):
        step()
        if i + 1 < steps:
            marks[i + 1].record()
    last = torch.cuda.Event(enable_timing=True)
    last.record()
    torch.cuda.synchronize()
    marks.append(last)
    per_step = sorted(marks[i].elapsed_time(marks[i + 1]) for i in range(steps))
    median_ms = per_step[steps // 2] if steps % 2 else \
        0.5 * (per_step[steps // 2 - 1] + per_step[steps // 2])

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(n_kernels + 1)]
           for _ in range(max(steps, 1))]
    if hold:
        torch.cuda.synchronize()
        hold_gpu_for_enqueue(host_ms, steps)
    for i in range(steps):
        step(evs[i])
    torch.cuda.synchronize()
    kern = [sum(e[j].elapsed_time(e[j + 1]) for e in evs[:steps]) / steps
            for j in range(n_kernels)]
    return {"ms_step": ms_step, "early_ms": early_ms, "median_ms": median_ms, "kern": kern,
            "warmed": done, "early_warmup": early_warmup}


def timing_fields(t: dict, args, work: float, unit_scale: float) -> dict:
    """The secondary timings of a bench line: `work` per step (FLOP or
    bytes) over unit_scale gives the metric's unit per second."""
    rate = lambda ms: round(work / (ms * 1e-3) / unit_scale, 2)
    return {
        "median": {"ms_per_step": round(t["median_ms"], 5), "value": rate(t["median_ms"]),
                   "note": "median of the per-step times of a separate pass"},
        "at_requested_warmup": {"warmup": t["early_warmup"],
                                "ms_per_step": round(t["early_ms"], 5),
                                "value": rate(t["early_ms"]),
                                "note": "timed right after the requested warm-up count "
                                        "(plus the five-step probe), before the clock settles"},
    }


# ---------------------------------------------------------------------------
# Paged key/value cache workloads (forward only, as in the paper)
# ---------------------------------------------------------------------------

def paged_flops(x) -> float:
    """4 * Hq * D * sum(q_len * kv_len), halved when causal with q_len ==
    kv_len (the same convention as the fixed-length forward)."""
    w = x.workload
    tot = 0.0
    for (qa, qb), (ka, kb) in zip(zip(x.qo_indptr, x.qo_indptr[1:]),
                                  zip(x.kv_indptr, x.kv_indptr[1:])):
        ql, kl = qb - qa, kb - ka
        tot += ql * kl * (0.5 if w.causal and ql == kl and ql > 1 else 1.0)
    return 4.0 * w.Hq * w.D * tot


def decode_bytes(x) -> dict:
    """Algorithmic HBM bytes of one decode step, by kernel: the split kernel
    reads every key and value row of every request once, the queries and the
    page indices; the outputs (bf16 O, fp32 LSE) are counted for the merge."""
    w = x.workload
    nnz, batch = len(x.kv_indices), w.batch
    kv = 2 * nnz * w.Hkv * w.D * 2
    q = batch * w.Hq * w.D * 2
    idx = 4 * (nnz + batch + 1)
    out = batch * w.Hq * (w.D * 2 + 4)
    return {"decode_split_kernel": kv + q + idx, "decode_merge_kernel": out}


def prefill_bytes(x) -> float:
    """Algorithmic HBM bytes of one paged prefill call: the queries, every
    key and value row of every request once (per key/value head), the page
    indices and index pointers, and the outputs (bf16 O, fp32 LSE)."""
    w = x.workload
    tq, nnz = x.q.shape[0], len(x.kv_indices)
    return (2 * tq * w.Hq * w.D * 2 + 2 * nnz * w.Hkv * w.D * 2 + 4 * tq * w.Hq
            + 4 * (nnz + 2 * (w.batch + 1)))


def cpu_baseline_paged(x, seconds: float, unit_of):
    """Oracle (fp64, CPU) on the whole paged workload, repeated until about
    `seconds` have elapsed; `unit_of(passes, dt)` turns it into the metric."""
    import torch
    import oracle
    w = x.workload
    t0, passes = time.perf_counter(), 0
    while passes == 0 or time.perf_counter() - t0 < seconds:
        oracle.attention_forward_paged(x.q, x.k_cache, x.v_cache, x.qo_indptr, x.kv_indptr,
                                       x.kv_indices, w.causal, w.scale)
        passes += 1
    dt = time.perf_counter() - t0
    value, unit = unit_of(passes, dt)
    return {"value": round(value, 6), "unit": unit, "cores": torch.get_num_threads(),
            "kind": "oracle",
            "sample": f"the whole workload {w.name}, {passes} pass(es), fp64 forward, {dt:.1f} s"}


def run_paged(args, w) -> int:
    import torch
    from paper_2608_17379_amd import attn
    from paper_2608_17379_amd import workloads as wl

    x = wl.make_paged_inputs(w, 0)
    dev = torch.device("cuda", 0)
    q, kc, vc = (t.to(dev) for t in (x.q, x.k_cache, x.v_cache))
    qo = torch.tensor(x.qo_indptr, dtype=torch.int32, device=dev)
    kv = torch.tensor(x.kv_indptr, dtype=torch.int32, device=dev)
    idx = torch.tensor(x.kv_indices, dtype=torch.int32, device=dev)
    o = torch.empty_like(q)
    lse = torch.empty(w.Hq, q.shape[0], dtype=torch.float32, device=dev)
    # The index arrays are checked once here; the timed calls skip the
    # binding's host-side checks (they would otherwise dominate the step).
    attn.check_cu_seqlens(x.qo_indptr, q.shape[0], x.max_qlen)
    attn.check_paged_host(x.kv_indptr, x.kv_indices, w.num_pages, x.max_kvlen)
    host = dict(checked=True)
    if w.decode:
        kernels = ("decode_split_kernel", "decode_merge_kernel")
        ws = attn.decode_workspace_for(q, kc, x.max_kvlen)

        def launch(i):
            ph = (attn.ATTN_DECODE_SPLIT, attn.ATTN_DECODE_MERGE)[i]
            attn.attn_decode_paged_phases(q, kc, vc, o, lse, kv, idx, x.max_kvlen, w.scale, ws,
                                          ph, **host)
    else:
        # The call is given the workspace it asks for.  A prefill far too small
        # to fill the chip then runs split (two kernels in one call, timed
        # together); one that leaves CUs idle runs the key-halves form.
        ws = attn.prefill_workspace_for(q, kc, w.batch, x.max_qlen, x.max_kvlen)
        kernels = ("fwd_kernel+fwd_merge_kernel",) if ws is not None else ("fwd_kernel",)
        form = {attn.ATTN_FWD_PAGED_UNSPLIT: "unsplit", attn.ATTN_FWD_PAGED_KEY_HALVES: "key halves",
                attn.ATTN_FWD_PAGED_SPLIT: "split"}[
            attn.attn_fwd_paged_form(w.batch, x.max_qlen, x.max_kvlen, w.Hq, True)]

        def launch(i):
            attn.attn_fwd_paged(q, kc, vc, o, lse, qo, kv, idx, x.max_qlen, x.max_kvlen,
                                w.causal, w.scale, ws, **host)

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        for i in range(len(kernels)):
            launch(i)
            if ev is not None:
                ev[1 + i].record()

    tm = time_steps(step, len(kernels), args.steps, args.warmup, args.warmup_seconds)
    ms_step, warmed = tm["ms_step"], tm["warmed"]
    kern_ms = dict(zip(kernels, tm["kern"]))
    gpu_state = sustained_state(step, args.state_seconds)
    if not (torch.isfinite(o.float()).all() and torch.isfinite(lse).all()):
        print("non-finite output", file=sys.stderr)
        return 1

    F = paged_flops(x)
    cfg = {"workload": w.name, "batch": w.batch, "Hq": w.Hq, "Hkv": w.Hkv, "D": w.D,
           "nnz": w.nnz, "num_pages": w.num_pages, "page_size": 1, "causal": w.causal,
           "decode": w.decode, "seed": 0,
           "kv_lens": [b - a for a, b in zip(x.kv_indptr, x.kv_indptr[1:])]}
    if not w.decode:
        cfg["prefill_form"] = form
    rec = {"n_gpus": 1, "steps": args.steps, "warmup": warmed, "warmup_requested": args.warmup,
           "warmup_seconds": args.warmup_seconds,
           "ms_per_step": round(ms_step, 5), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic (seeded i.i.d. N(0,1) bf16; seeded lengths and pages)",
           "config": cfg, "kernel_ms": {n: round(t, 5) for n, t in kern_ms.items()},
           "gpu_state": gpu_state}
    if w.decode:
        by = decode_bytes(x)
        total = sum(by.values())
        dom = max(kernels, key=lambda n: kern_ms[n])
        rec.update({"metric": f"paged decode HBM GB/s, {w.name}",
                    "value": round(total / (ms_step * 1e-3) / 1e9, 2), "unit": "GB/s",
                    "tflops": round(F / (ms_step * 1e-3) / 1e12, 4),
                    "roofline": roofline(dom, 0.0, by[dom], kern_ms[dom], w.name,
                                         hbm_work=True)})
        rec.update(timing_fields(tm, args, total, 1e9))
        unit_of = lambda n, dt: (total * n / dt / 1e9, "GB/s")
    else:
        kn = kernels[0]
        rec.update({"metric": f"attention fwd TFLOP/s, {w.name}",
                    "value": round(F / (ms_step * 1e-3) / 1e12, 2), "unit": "TFLOP/s",
                    "pct_peak": round(100 * F / (ms_step * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2),
                    "roofline": roofline(kn, F, prefill_bytes(x), kern_ms[kn], w.name)})
        rec.update(timing_fields(tm, args, F, 1e12))
        unit_of = lambda n, dt: (F * n / dt / 1e12, "TFLOP/s")
    if not args.no_cpu_baseline:
        with cpu_threads() as ct:
            rec["cpu_baseline"] = cpu_baseline_paged(x, args.cpu_seconds, unit_of)
            rec["cpu_baseline"].update(ct.fields())
    else:
        rec["cpu_baseline"] = None
    print(json.dumps(rec), flush=True)
    return 0


# ---------------------------------------------------------------------------
# BF16 GEMM C = A B^T
# ---------------------------------------------------------------------------

def run_gemm(args, w) -> int:
    import torch
    import oracle
    from paper_2608_17379_amd import attn
    from paper_2608_17379_amd import workloads as wl

    a_h, b_h = wl.make_gemm_inputs(w, 0)
    dev = torch.device("cuda", 0)
    a, b = a_h.to(dev), b_h.to(dev)
    c = torch.empty(w.M, w.N, dtype=torch.bfloat16, device=dev)
    lib = attn.lib()
    stream = torch.cuda.current_stream().cuda_stream

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        st = lib.attn_gemm_bf16_nt(a.data_ptr(), b.data_ptr(), c.data_ptr(), w.M, w.N, w.K,
                                   stream)
        if st != 0:
            raise attn.AttnError(st, "attn_gemm_bf16_nt")
        if ev is not None:
            ev[1].record()

    attn.attn_gemm_bf16_nt(a, b, c)   # shape and pointer checks once, through the binding
    tm = time_steps(step, 1, args.steps, args.warmup, args.warmup_seconds)
    ms_step, (kern_ms,), warmed = tm["ms_step"], tm["kern"], tm["warmed"]
    gpu_state = sustained_state(step, args.state_seconds)
    if not torch.isfinite(c.float()).all():
        print("non-finite output", file=sys.stderr)
        return 1
    F = 2.0 * w.M * w.N * w.K
    rec = {"metric": f"bf16 GEMM TFLOP/s, {w.name}",
           "value": round(F / (ms_step * 1e-3) / 1e12, 2), "unit": "TFLOP/s", "n_gpus": 1,
           "steps": args.steps, "warmup": warmed, "warmup_requested": args.warmup,
           "warmup_seconds": args.warmup_seconds, "ms_per_step": round(ms_step, 5),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic (seeded i.i.d. N(0,1) bf16)",
           "config": {"workload": w.name, "M": w.M, "N": w.N, "K": w.K, "seed": 0},
           "gpu_state": gpu_state,
           "pct_peak": round(100 * F / (ms_step * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2),
           # The paper's shape runs as one launch of gemm_rounds_kernel (full
           # tiles in rounds, then the remaining tiles' halves).
           "kernel_ms": {"gemm_rounds_kernel": round(kern_ms, 5)},
           "roofline": roofline("gemm_rounds_kernel", F,
                                2.0 * (w.M * w.K + w.N * w.K + w.M * w.N), kern_ms, w.name),
           "cpu_baseline": None}
    rec.update(timing_fields(tm, args, F, 1e12))
    if not args.no_cpu_baseline:
        # The oracle on whole rows of C (64 rows at a time) until the budget is spent.
        with cpu_threads() as ct:
            t0, rows = time.perf_counter(), 0
            while rows == 0 or time.perf_counter() - t0 < args.cpu_seconds:
                r0 = rows % w.M
                oracle.gemm_nt(a_h[r0:r0 + 64], b_h)
                rows += 64
            dt = time.perf_counter() - t0
            rec["cpu_baseline"] = {"value": round(2.0 * rows * w.N * w.K / dt / 1e12, 6),
                                   "unit": "TFLOP/s", "kind": "oracle",
                                   "sample": f"{rows} rows of C ({rows}x{w.N}x{w.K}), fp64, "
                                             f"{dt:.1f} s", **ct.fields()}
    print(json.dumps(rec), flush=True)
    return 0


def copy_calibration(nbytes: int, reps: int) -> None:
    """A plain device copy of known size, for scaling HBM byte counters."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "reps": reps}), flush=True)


def mfma_calibration(iters: int, reps: int, seconds: float) -> None:
    """The chip's sustained bf16 MFMA rate: two 4-wavefront workgroups per CU
    running independent chains of v_mfma_f32_32x32x16_bf16 on registers
    (libcalib.so), timed by events, with the graphics clock sampled over a
    sustained pass.  flop/clk/CU = rate / (CUs x clock); the quoted peak
    assumes 4096 at 2.4 GHz."""
    import ctypes
    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2608_17379_amd", "libcalib.so"))
    lib.calib_mfma_rate.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    chains = lib.calib_mfma_chains()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = 2 * cus
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream

    def launch():
        st = lib.calib_mfma_rate(blocks, iters, ctypes.c_void_p(out.data_ptr()),
                                 ctypes.c_void_p(stream))
        if st != 0:
            raise RuntimeError(f"calib_mfma_rate returned {st}")

    for _ in range(3):
        launch()
    state = sustained_state(launch, seconds)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        launch()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    flop = float(blocks) * 4 * iters * chains * 32768
    tflops = flop / (ms * 1e-3) / 1e12
    rec = {"mfma_calibration": {"blocks": blocks, "wavefronts_per_simd": 2, "iters": iters,
                                "chains": chains, "ms_per_launch": round(ms, 4),
                                "tflops": round(tflops, 1), "cus": cus,
                                "frac_of_quoted_peak": round(tflops / PEAK_BF16_TFLOPS, 4)}}
    sclk = (state or {}).get("sclk_mhz", {}).get("mean") if state else None
    if sclk:
        rec["mfma_calibration"]["sclk_mhz"] = sclk
        rec["mfma_calibration"]["flop_per_clk_per_cu"] = round(
            tflops * 1e12 / (cus * sclk * 1e6), 1)
    rec["gpu_state"] = state
    print(json.dumps(rec), flush=True)


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10,
                    help="minimum untimed warm-up steps (more run until --warmup-seconds)")
    ap.add_argument("--warmup-seconds", type=float, default=1.0,
                    help="minimum length of the warm-up (the GPU's clocks settle under load)")
    ap.add_argument("--workload", default=None)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES")
    ap.add_argument("--mfma-calibration", type=int, default=0, metavar="ITERS",
                    help="measure the sustained MFMA rate (ITERS loop trips per wavefront)")
    ap.add_argument("--cold-steps", type=int, default=10,
                    help="steps of the cold-cache pass (0: none)")
    ap.add_argument("--dkdv-form", choices=sorted(DKDV_FORMS), default="auto",
                    help="form of the dK/dV kernel (auto: the one the library picks)")
    ap.add_argument("--state-seconds", type=float, default=1.5,
                    help="length of the untimed pass that samples clock, temperature and power")
    args = ap.parse_args(argv)

    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the attention path is not sharded across GPUs).", file=sys.stderr)
        return 2

    import torch
    from paper_2608_17379_amd import attn
    from paper_2608_17379_amd import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if args.copy_calibration:
        copy_calibration(args.copy_calibration, max(1, args.steps))
        return 0
    if args.mfma_calibration:
        mfma_calibration(args.mfma_calibration, max(1, args.steps), args.state_seconds)
        return 0

    name = args.workload or wl.HEADLINE
    if name in wl.PAGED_WORKLOADS:
        return run_paged(args, wl.PAGED_WORKLOADS[name])
    if name in wl.GEMM_WORKLOADS:
        return run_gemm(args, wl.GEMM_WORKLOADS[name])
    if name not in wl.WORKLOADS:
        print(f"unknown workload {name}; known: "
              + ", ".join(list(wl.WORKLOADS) + list(wl.PAGED_WORKLOADS)
                          + list(wl.GEMM_WORKLOADS)), file=sys.stderr)
        return 2
    w = wl.WORKLOADS[name]
    x = wl.make_inputs(w, 0)
    dev = torch.device("cuda", 0)
    q, k, v, do = (t.to(dev) for t in (x.q, x.k, x.v, x.do))
    o, dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    cu = None
    if w.varlen:
        cu = torch.tensor(x.cu_seqlens, dtype=torch.int32, device=dev)
        lse = torch.empty(w.Hq, q.shape[0], dtype=torch.float32, device=dev)
    else:
        lse = torch.empty(w.B, w.Hq, w.S, dtype=torch.float32, device=dev)
    ws = attn.workspace_for(q, k, cu)
    ms_len = x.max_seqlen
    form_bit = DKDV_FORMS[args.dkdv_form]

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        if cu is None:
            attn.attn_fwd(q, k, v, o, lse, w.causal, w.scale)
        else:
            attn.attn_fwd_varlen(q, k, v, o, lse, cu, ms_len, w.causal, w.scale,
                                 cu_seqlens_host=x.cu_seqlens)
        if ev is not None:
            ev[1].record()
        for i, ph in enumerate((attn.ATTN_BWD_DQ, attn.ATTN_BWD_DKDV | form_bit)):
            if cu is None:
                attn.attn_bwd_phases(q, k, v, o, lse, do, dq, dk, dv, w.causal, w.scale, ws, ph)
            else:
                attn.attn_bwd_varlen_phases(q, k, v, o, lse, do, dq, dk, dv, cu, ms_len, w.causal,
                                            w.scale, ws, ph, cu_seqlens_host=x.cu_seqlens)
            if ev is not None:
                ev[2 + i].record()

    # The dK/dV phase runs the form the library picks for these shapes, or
    # the one --dkdv-form names.
    nseg = len(x.cu_seqlens) - 1 if w.varlen else w.B
    form = form_bit or attn.attn_bwd_dkdv_form(nseg, w.Hkv, ms_len if w.varlen else w.S,
                                               q.shape[0] if w.varlen else 0, w.D, w.causal,
                                               w.varlen)
    if w.D == 64 and form == attn.ATTN_BWD_DKDV_ONE_PER_CU:
        form = attn.ATTN_BWD_DKDV_TWO_PER_CU   # D = 64 has no eight-wavefront form
    dkdv = DKDV_KERNELS[form]
    kernels = ("fwd_kernel", "bwd_dq_kernel", dkdv)
    tm = time_steps(step, len(kernels), args.steps, args.warmup, args.warmup_seconds)
    ms_step, warmed = tm["ms_step"], tm["warmed"]
    kern_ms = dict(zip(kernels, tm["kern"]))
    ms_cold = cold_steps(step, args.cold_steps) if args.cold_steps > 0 else None
    gpu_state = sustained_state(step, args.state_seconds)
    for t in (o, lse, dq, dk, dv):
        if not torch.isfinite(t.float()).all():
            print("non-finite output", file=sys.stderr)
            return 1

    F = fwd_flops(w, x.cu_seqlens)
    total = 3.5 * F
    value = total / (ms_step * 1e-3) / 1e12
    dom = max(kernels, key=lambda n: kern_ms[n])
    kflop = {n: GEMMS[n] / 2 * F for n in kernels}
    fwd_ms = kern_ms["fwd_kernel"]
    bwd_ms = kern_ms["bwd_dq_kernel"] + kern_ms[dkdv]
    cfg = {"workload": w.name, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "S": w.S, "D": w.D,
           "causal": w.causal, "seed": 0}
    if w.varlen:
        cfg["seq_lens"] = [b - a for a, b in zip(x.cu_seqlens, x.cu_seqlens[1:])]
    rec = {
        "metric": METRIC if w.name == wl.HEADLINE else f"attention fwd/bwd TFLOP/s, {w.name}",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": warmed, "warmup_requested": args.warmup,
        "warmup_seconds": args.warmup_seconds,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded i.i.d. N(0,1) bf16)",
        "config": cfg,
        "pct_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "fwd_tflops": round(F / (fwd_ms * 1e-3) / 1e12, 2),
        "bwd_tflops": round(2.5 * F / (bwd_ms * 1e-3) / 1e12, 2),
        "fwd_pct_peak": round(100 * F / (fwd_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2),
        "bwd_pct_peak": round(100 * 2.5 * F / (bwd_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2),
        "kernel_ms": {n: round(t, 4) for n, t in kern_ms.items()},
        "kernel_tflops": {n: {"algorithmic": round(kflop[n] / (kern_ms[n] * 1e-3) / 1e12, 2),
                              "executed": round(GEMMS_EXECUTED[n] / 2 * F
                                                / (kern_ms[n] * 1e-3) / 1e12, 2)}
                          for n in kernels},
        "roofline": roofline(dom, kflop[dom], attention_bytes(dom, w, x), kern_ms[dom], w.name),
        "cpu_baseline": None,
        "cold": None if ms_cold is None else {
            "ms_per_step": round(ms_cold, 4),
            "value": round(total / (ms_cold * 1e-3) / 1e12, 2),
            "steps": args.cold_steps,
            "note": "median step after a 512 MiB write flushes L2 and MALL (write not timed)"},
        "gpu_state": gpu_state,
    }
    rec.update(timing_fields(tm, args, total, 1e12))
    if not args.no_cpu_baseline:
        with cpu_threads() as ct:
            rec["cpu_baseline"] = cpu_baseline(w, x, args.cpu_seconds)
            rec["cpu_baseline"].update(ct.fields())
    print(json.dumps(rec), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
