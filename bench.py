#!/usr/bin/env python3
"""Throughput of the MI355X GEMM library on the paper-shaped workload sweep.

Default run (one GPU), in this order:

1. `configs`: every other workload of the sweep (int8 256^3, bf16 1024^3, the
   2048^3 / 4096^3 squares, the three rectangles, the twelve skinny shapes),
   each timed with HIP events on the launch stream under a labelled protocol
   (cold for the cache-sized and the memory-bound shapes, warm otherwise), with
   its plan, roofline fraction and sampled oracle rows, and the CPU oracle timed on
   the first rows of the same workload (`cpu_oracle`, those rows also compared);
2. the headline: the int8 -> int32 GEMM at M = N = K = 8192 (`value`, TOPS) and
   the bf16 -> fp32 GEMM at the same size (the `bf16` object), inputs resident
   in HBM, W untimed warm-up launches, then K timed launches bracketed by device
   synchronisation; each with the CPU oracle timed on a bounded sample of the
   same workload (`cpu_baseline`) and the timed output compared with every
   oracle row that sample computed (`parity_full`);
3. the same two GEMMs with B stored column-major, and the sustained MFMA
   ceiling of the chip (only the GEMM's MFMAs, no memory traffic): every
   MFMA-bound row of `configs` also gets its fraction of that ceiling, the
   clock-adjusted peak of the box it ran on.

Prints ONE JSON line on stdout with a roofline object for the dominant kernel.

    python bench.py [--steps K] [--warmup W] [--size S] [--no-configs] [--sweep]
    python bench.py --workload int8:2048x2048x2048 --steps 50   # one workload (profiling)

`--paper-sweep` times the GEMM over every (M, K, N) in multiples of the 256 tile
up to 8192 (512 points per dtype and B layout).  `--reduced` also times the 8192^3
GEMMs with narrowed outputs (int8 -> int8, bf16 -> bf16).  `--sweep` writes one
row per workload to OUT_DIR/sweep.jsonl.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time
import types

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"int8": 5000.0, "bf16": 2500.0}          # dense MFMA, TOPS / TFLOP/s (AMD published)
REDUCE_NAMES = {0: "separate", 1: "last-slice", 2: "atomic", 3: "atomic-flag"}   # split-K reductions (GEMM_REDUCE_*)
PLAN_SOURCES = {0: "model", 1: "measured (table)", 2: "measured (nearest M)", 3: "measured (plan file)", 4: "forced"}   # gemm_plan_info.source (GEMM_PLAN_FROM_*)
CONFIG_ORACLE_SECONDS = 0.25  # CPU oracle work per row of the workload table (`cpu_oracle`)
HBM_GBS = 8000.0
KERNEL_DIR = os.path.join(ROOT, "paper_2512_13282_amd", "csrc")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
COPY_PROBE_BYTES = 512 * 1024 * 1024
REQUANT_SHIFT = 14          # int8 -> int8 output: results / 2^14 (|C| <= 2^21 at K = 8192 for uniform int8)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    # The chip's power management needs a few tens of milliseconds of a new load to settle on
    # its sustained clock: launches timed within that window run up to 1.2x slower.  Every
    # timed workload therefore first runs untimed for --settle-ms, then its W warm-up launches.
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--settle-ms", type=float, default=SETTLE_MS,
                    help="untimed launches of each workload for this long before its warm-up (0: none)")
    ap.add_argument("--size", type=int, default=8192)
    ap.add_argument("--sweep", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-bt", action="store_true", help="skip the column-major-B measurements")
    ap.add_argument("--no-ceiling", action="store_true", help="skip the sustained-MFMA-ceiling probe")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--only", choices=["int8", "bf16"], default=None)
    ap.add_argument("--config", type=int, default=-1,
                    help="force one tile configuration (index into the library's table)")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"), default=None,
                    help="write profiles/traffic.json from two rocprofv3 --pmc counter CSVs "
                         "(FETCH_SIZE, WRITE_SIZE) of a `bench.py --copy-probe` run, then exit")
    ap.add_argument("--reduced", action="store_true",
                    help="also time the 8192^3 GEMMs with narrowed outputs (int8 -> int8, bf16 -> bf16); "
                         "off by default because they run the same kernel instances as the int32 / fp32 "
                         "GEMMs, whose per-kernel profiler averages they would otherwise mix into")
    ap.add_argument("--paper-sweep", action="store_true",
                    help="also time the GEMM over M, K, N in multiples of the 256 tile up to 8192, both "
                         "dtypes and B layouts (the paper's > 400-size sweep); details in "
                         "OUT_DIR/paper_sweep.jsonl, summary in the JSON line")
    ap.add_argument("--sweep-set", choices=("all", "skinny"), default="all",
                    help="workloads --sweep times: all of them, or only the skinny (M <= 64) ones")
    ap.add_argument("--out-dir", default="bench_out",
                    help="directory (relative to the repository root unless absolute) for the "
                         "per-point files of --sweep and --paper-sweep")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 512 MiB device copy (reference for HBM byte counters)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-workload table (every other workload of the sweep, timed before "
                         "the headline)")
    ap.add_argument("--config-steps", type=int, default=50, help="timed launches per workload of the table")
    ap.add_argument("--config-warmup", type=int, default=20, help="untimed launches per workload of the table")
    ap.add_argument("--workload", default=None, metavar="DTYPE:MxKxN",
                    help="time only this workload (e.g. int8:2048x2048x2048) with --steps/--warmup and print "
                         "one JSON line (for profiling one kernel)")
    ap.add_argument("--cold", action="store_true",
                    help="with --workload: rotate the launches through copies of B so that more than 512 MB "
                         "is read between reuses of one (B from HBM, as a layer's weights arrive)")
    return ap.parse_args()


def kernel_sha() -> str:
    """Hash of the device sources (every .hip and .h of the library), in name order."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(KERNEL_DIR)):
        if name.endswith((".hip", ".h")):
            h.update(name.encode() + b"\0" + open(os.path.join(KERNEL_DIR, name), "rb").read())
    return h.hexdigest()


def traffic_for(dtype: str, M: int, N: int, K: int, bt: bool = False):
    """HBM bytes per launch from committed rocprofv3 FETCH_SIZE/WRITE_SIZE counters, or None
    when none were taken for this workload (B layout included) or the kernel source changed since."""
    try:
        t = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != kernel_sha():
        return None
    rec = t.get("workloads", {}).get(f"{dtype}_{M}x{K}x{N}" + ("_bt" if bt else ""))
    return None if rec is None else rec.get("bytes_per_launch")


class Workload:
    """One GEMM with its operands resident on the GPU.  bt=True stores B column-major
    (as Bt, N x K) and calls the *_bt entry points."""

    def __init__(self, dtype, M, N, K, copies=1, seed=0, bt=False, out="native"):
        import torch
        from paper_2512_13282_amd import binding, inputs
        self.dtype, self.M, self.N, self.K, self.bt = dtype, M, N, K, bt
        self.out = out      # "native" (int32 / fp32 C), "i8" (int8 -> int8, shift) or "bf16" (bf16 -> bf16)
        self.b = binding
        A, B = inputs.make_inputs(dtype, M, N, K, seed=seed)
        self.A_host, self.B_host = A, B
        dev = torch.device("cuda:0")
        to = (lambda x: torch.from_numpy(x).to(dev)) if dtype == "int8" else \
             (lambda x: torch.from_numpy(x.view(np.int16)).to(dev))
        self.dA = to(A)
        Bdev = to(np.ascontiguousarray(B.T)) if bt else to(B)
        self.dBs = [Bdev] + [Bdev.clone() for _ in range(copies - 1)]
        self.ldb = K if bt else N
        c_dtype = {"native": torch.int32 if dtype == "int8" else torch.float32, "i8": torch.int8,
                   "bf16": torch.int16}[out]
        self.dC = torch.empty((M, N), dtype=c_dtype, device=dev)
        sfx = "_bt" if bt else ""
        if out == "native":
            self.fn = getattr(binding, ("gemm_i8_i32" if dtype == "int8" else "gemm_bf16_f32") + sfx)
        elif out == "i8":
            assert dtype == "int8"
            f = getattr(binding, "gemm_i8_i8" + sfx)
            self.fn = lambda *a: f(*a[:-1], REQUANT_SHIFT, a[-1])
        else:
            assert dtype == "bf16"
            self.fn = getattr(binding, "gemm_bf16_bf16" + sfx)
        self.stream = torch.cuda.current_stream(dev)
        self.i = 0

    def launch(self):
        dB = self.dBs[self.i % len(self.dBs)]
        self.i += 1
        rc = self.fn(self.M, self.N, self.K, self.dA.data_ptr(), self.K, dB.data_ptr(), self.ldb,
                     self.dC.data_ptr(), self.N, self.stream.cuda_stream)
        if rc != 0:
            raise RuntimeError(self.b.gemm_status_string(rc))

    def plan(self):
        # The plan does not depend on C's element type, but gemm_plan checks an int32 / fp32 C
        # against A and B; narrowed outputs ask with a full-width buffer of the same shape.
        import torch
        c = self.dC if self.out == "native" else torch.empty(
            (self.M, self.N), dtype=torch.int32 if self.dtype == "int8" else torch.float32, device="cuda:0")
        return self.b.gemm_plan(0 if self.dtype == "int8" else 1, self.M, self.N, self.K, self.K, self.ldb,
                                self.N, self.dA.data_ptr(), self.dBs[0].data_ptr(), c.data_ptr(),
                                trans_b=self.bt)


_SPIN_RATE = None


def spin_ahead(launches: int, host_us_per_launch: float = 80.0) -> None:
    """Queues a spin kernel long enough for the host to enqueue `launches` more launches (with
    their events) behind it, so that kernels shorter than one Python launch still run back to
    back and their events time the GPU, not the host.  The spin's rate (cycles per
    microsecond) is measured once."""
    global _SPIN_RATE
    import torch
    if _SPIN_RATE is None:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        torch.cuda._sleep(1_000_000)
        e1.record()
        torch.cuda.synchronize()
        _SPIN_RATE = 1_000_000 / max(e0.elapsed_time(e1) * 1e3, 1.0)
    torch.cuda._sleep(int(_SPIN_RATE * host_us_per_launch * launches))


SETTLE_MS = 100.0   # untimed launches ahead of every timed workload (--settle-ms)


def settle(w: Workload, ms: float) -> None:
    """Untimed launches of the workload for at least `ms` of wall time.  The chip's power
    manager needs that long to settle on the clock it sustains under a new load: timed launches
    that start within a few tens of milliseconds of an idle or lighter phase (a fresh process,
    the CPU oracle, the previous workload) run up to 1.2x slower than the same launches a
    moment later."""
    import torch
    if ms <= 0:
        return
    end = time.perf_counter() + ms / 1e3
    while time.perf_counter() < end:
        for _ in range(8):
            w.launch()
        torch.cuda.synchronize()


def time_back_to_back(w: Workload, steps: int, warmup: int, settle_ms: float = SETTLE_MS):
    """W untimed launches; then, behind a spin kernel that lets the host queue them all,
    `steps` back-to-back launches between two HIP events on the launch stream.  Returns the
    GPU time per launch in ms (kernel plus the GPU's own gap between kernels; events around
    every launch would add their own overhead, a few microseconds per launch)."""
    import torch
    settle(w, settle_ms)
    for _ in range(warmup):
        w.launch()
    torch.cuda.synchronize()
    spin_ahead(steps, 40.0)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(w.stream)
    for _ in range(steps):
        w.launch()
    e1.record(w.stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    return ms, ms, ms


def time_workload(w: Workload, steps: int, warmup: int, settle_ms: float = SETTLE_MS):
    """The settle phase, W untimed launches, then `steps` launches with HIP events on the
    launch stream around each.  Returns (wall ms per step, mean kernel ms, min kernel ms)."""
    import torch
    settle(w, settle_ms)
    for _ in range(warmup):
        w.launch()
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        starts[i].record(w.stream)
        w.launch()
        ends[i].record(w.stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kernel_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    return wall * 1e3 / steps, float(np.mean(kernel_ms)), float(np.min(kernel_ms))


FLUSH_BYTES = 512 * 1024 * 1024      # twice the last-level cache


def time_workload_flushed(w: Workload, steps: int, warmup: int, settle_ms: float = SETTLE_MS):
    """Cold-cache timing for operands that fit in the caches: before every launch a 512 MiB
    scratch buffer is written (evicting A, B and C from the L2s and the 256 MB last-level
    cache), then the launch alone is timed with HIP events on the launch stream."""
    import torch
    scratch = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda:0")
    settle(w, settle_ms)
    for _ in range(warmup):
        w.launch()
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    for i in range(steps):
        scratch.fill_(float(i))
        starts[i].record(w.stream)
        w.launch()
        ends[i].record(w.stream)
    torch.cuda.synchronize()
    kernel_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    del scratch
    k_avg = float(np.mean(kernel_ms))
    return k_avg, k_avg, float(np.min(kernel_ms))


def summarize(w: Workload, ms_step: float, k_avg: float, k_min: float):
    ops = 2.0 * w.M * w.N * w.K
    e = 1 if w.dtype == "int8" else 2
    c_bytes = {"native": 4, "i8": 1, "bf16": 2}[getattr(w, "out", "native")]
    comp_bytes = w.M * w.K * e + w.K * w.N * e + w.M * w.N * c_bytes
    plan = w.plan()
    value = ops / (ms_step * 1e-3) / 1e12
    achieved = ops / (k_avg * 1e-3) / 1e12
    mem_bound = ops / comp_bytes < (PEAK[w.dtype] * 1e12) / (HBM_GBS * 1e9)
    traffic = traffic_for(w.dtype, w.M, w.N, w.K, w.bt)
    if mem_bound:
        ach_gbs = comp_bytes / (k_avg * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach_gbs, 1), "peak": HBM_GBS, "unit": "GB/s",
                "frac": round(ach_gbs / HBM_GBS, 4), "traffic": traffic}
    else:
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK[w.dtype],
                "unit": "TOPS" if w.dtype == "int8" else "TFLOP/s",
                "frac": round(achieved / PEAK[w.dtype], 4), "traffic": traffic}
    return {
        "value": round(value, 2), "unit": "TOPS" if w.dtype == "int8" else "TFLOP/s",
        "ms_per_step": round(ms_step, 5), "kernel_ms_avg": round(k_avg, 5), "kernel_ms_min": round(k_min, 5),
        "pct_dense_peak": round(100.0 * value / PEAK[w.dtype], 2),
        "plan": plan["name"], "split_k": plan["split_k"], "grid": plan["grid"],
        "reduce": REDUCE_NAMES[plan["reduce_in_kernel"]] if plan["split_k"] > 1 else None,
        "plan_source": PLAN_SOURCES.get(plan.get("source"), "?"),
        "algorithmic_ops_per_launch": ops, "algorithmic_bytes_per_launch": comp_bytes,
        "roofline": roof,
    }


def parity_sample(w: Workload, rows):
    """Compares the timed output's sampled rows with the oracle (cheap evidence, not the test)."""
    from oracle import oracle
    o = oracle.get()
    C = w.dC[rows].cpu().numpy()
    Ar = np.ascontiguousarray(w.A_host[rows])
    if w.dtype == "int8":
        ref, ovf = o.gemm_i8_i32(Ar, w.B_host)
        if w.out == "i8":
            ref = o.requant_i32(ref, REQUANT_SHIFT, 8)
        return bool(ovf == 0 and np.array_equal(C, ref))
    if w.out == "bf16":
        # within one bf16 step of the correctly rounded exact result
        from paper_2512_13282_amd import inputs
        ref = inputs.f32_from_bf16_bits(o.round_bf16(o.gemm_bf16_f64(Ar, w.B_host))).astype(np.float64)
        got = inputs.f32_from_bf16_bits(C.view(np.uint16)).astype(np.float64)
        step = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -126))) - 7)
        return bool(np.all(np.abs(got - ref) <= step))
    from paper_2512_13282_amd import inputs
    ref = o.gemm_bf16_f64(Ar, w.B_host)
    err = oracle.normalized_error(C, ref, w.K, float(np.abs(inputs.f32_from_bf16_bits(w.A_host)).max()),
                                  float(np.abs(inputs.f32_from_bf16_bits(w.B_host)).max()))
    return bool(err <= 1e-5)


def parity_full(w: Workload):
    """The timed output against the oracle rows cpu_baseline computed (all M rows when the
    oracle finished the whole product): int8 element for element, bf16 by the normalized
    error.  Returns None when no oracle rows are held."""
    held = getattr(w, "oracle_rows", None)
    if held is None:
        return None
    rows, out = held
    C = w.dC[:rows].cpu().numpy()
    if w.dtype == "int8":
        ref, ovf = out
        bad = int(np.count_nonzero(C != ref))
        return {"rows_compared": rows, "of_rows": w.M, "mismatches": bad, "overflows": int(ovf),
                "ok": bool(bad == 0 and ovf == 0), "rule": "bit-exact"}
    from oracle import oracle
    from paper_2512_13282_amd import inputs
    err = oracle.normalized_error(C, out, w.K, float(np.abs(inputs.f32_from_bf16_bits(w.A_host)).max()),
                                  float(np.abs(inputs.f32_from_bf16_bits(w.B_host)).max()))
    return {"rows_compared": rows, "of_rows": w.M, "normalized_error": float(err), "ok": bool(err <= 1e-5),
            "rule": "max|C - C_ref| / (K max|A| max|B|) <= 1e-5"}


def bare_read_us(w: Workload, steps: int = 50, warmup: int = 10) -> float:
    """Microseconds a plain read of B takes (gemm_probe_read), back to back over the same
    rotating copies of B the GEMM was timed with: what the memory-bound GEMMs are held to."""
    import torch
    from paper_2512_13282_amd import binding
    nbytes = w.dBs[0].numel() * w.dBs[0].element_size()
    threads = torch.cuda.get_device_properties(0).multi_processor_count * 2048
    sink = torch.empty(threads, dtype=torch.int32, device="cuda:0")
    def call(i):
        rc = binding.gemm_probe_read(w.dBs[i % len(w.dBs)].data_ptr(), nbytes, sink.data_ptr(), threads,
                                     w.stream.cuda_stream)
        if rc != 0:
            raise RuntimeError(binding.gemm_status_string(rc))
    for i in range(warmup):
        call(i)
    torch.cuda.synchronize()
    spin_ahead(steps, 40.0)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(w.stream)
    for i in range(steps):
        call(i)
    e1.record(w.stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / steps


def config_table(skip, steps: int, warmup: int, oracle_seconds: float = 0.0, settle_ms: float = SETTLE_MS):
    """Every workload of the sweep (inputs.ALL_CONFIGS) except those in `skip`, timed with
    HIP events on the launch stream.  Shapes whose operands fit in the caches (int8 256^3,
    bf16 1024^3) are timed cold, one launch at a time after a 512 MiB flush; the skinny
    (memory-bound) shapes rotate through enough copies of B that more than 512 MB is read
    between reuses of a copy; the rest are timed warm.  Back-to-back launches are queued behind
    a spin kernel and timed between two events, so that each is timed on the GPU rather than
    waiting on the host's next launch (a Python launch takes longer than the smallest kernels).
    Each row carries its
    protocol, plan, roofline fraction and a parity check of sampled output rows; with
    `oracle_seconds` > 0 also the CPU oracle timed on the first rows of the same workload
    (about that many seconds of work, `cpu_oracle`) and those rows of the timed output compared
    with it (`parity_oracle_rows`)."""
    import torch
    from paper_2512_13282_amd import inputs
    rows, pending = [], []
    for (dtype, M, K, N) in inputs.ALL_CONFIGS:
        if (dtype, M, K, N) in skip:
            continue
        e = 1 if dtype == "int8" else 2
        skinny = M < 256
        copies = max(1, int(np.ceil(512e6 / (K * N * e))) + 1) if skinny else 1
        w = Workload(dtype, M, N, K, copies=copies)
        if (dtype, M, K, N) in inputs.SMALL:
            ms, kavg, kmin = time_workload_flushed(w, steps, warmup, settle_ms)
            proto = "cold: 512 MiB flush before each launch, launches timed one by one"
        else:
            ms, kavg, kmin = time_back_to_back(w, steps, warmup, settle_ms)
            proto = (f"cold: back to back, B rotated over {copies} copies (> 512 MB between reuses)"
                     if skinny else "warm: back to back, operands resident")
        r = summarize(w, ms, kavg, kmin)
        ops = 2.0 * M * N * K
        bare = bare_read_us(w) if skinny else None
        row = {"dtype": dtype, "M": M, "K": K, "N": N, "protocol": proto, "plan": r["plan"],
               "split_k": r["split_k"], "reduce": r["reduce"], "plan_source": r["plan_source"],
               "kernel_us": round(kavg * 1e3, 2),
               "value": round(ops / (kavg * 1e-3) / 1e12, 2), "unit": r["unit"],
               "pct_dense_peak": round(100.0 * ops / (kavg * 1e-3) / 1e12 / PEAK[dtype], 2),
               "roofline": {k: r["roofline"][k] for k in ("bound", "achieved", "unit", "frac")},
               "parity_sample_ok": parity_sample(w, sorted({0, M // 2, M - 1}))}
        if oracle_seconds > 0:
            # the oracle runs after every row is timed: CPU work between rows would leave the
            # GPU idle and let its clock drop before the next row's short warm-up
            pending.append((row, types.SimpleNamespace(dtype=dtype, M=M, N=N, K=K, A_host=w.A_host,
                                                       B_host=w.B_host, dC=w.dC.cpu())))
        if bare is not None:
            # a plain read of B under the same protocol (the GEMM also reads A and writes C)
            row["bare_read_of_B_us"] = round(bare, 2)
            row["frac_of_bare_read"] = round(bare / (kavg * 1e3), 3)
        rows.append(row)
        print(f"[configs] {dtype:4s} M={M:5d} K={K:6d} N={N:6d} {row['kernel_us']:9.1f} us {row['value']:9.2f} "
              f"{row['unit']:7s} {row['roofline']['bound']} frac={row['roofline']['frac']:.3f} plan={row['plan']} "
              f"x{row['split_k']}{' ' + row['reduce'] if row['reduce'] else ''} ok={row['parity_sample_ok']}"
              + (f" bare-read={row['bare_read_of_B_us']}us ({row['frac_of_bare_read']:.2f})" if "bare_read_of_B_us" in row else ""),
              file=sys.stderr, flush=True)
        del w
        torch.cuda.empty_cache()
    for row, hw in pending:
        cb = cpu_baseline(hw, oracle_seconds)
        row["cpu_oracle"] = {k: cb[k] for k in ("value", "unit", "cores", "seconds", "sample")}
        row["parity_oracle_rows"] = parity_full(hw)
        print(f"[oracle] {row['dtype']:4s} M={row['M']:5d} K={row['K']:6d} N={row['N']:6d} "
              f"{cb['value']} {cb['unit']} on {cb['cores']} threads ({cb['sample']}); timed output rows "
              f"ok={row['parity_oracle_rows']['ok']}", file=sys.stderr, flush=True)
    return rows


def cpu_baseline(w: Workload, seconds: float):
    """The oracle (as is) on the first rows of the same workload, sized to ~`seconds`."""
    from oracle import oracle
    o = oracle.get()
    threads = len(os.sched_getaffinity(0))
    cap = os.environ.get("OMP_NUM_THREADS")
    if cap and cap.isdigit():
        threads = min(threads, int(cap))
    fn = o.gemm_i8_i32 if w.dtype == "int8" else o.gemm_bf16_f64
    probe = max(1, min(w.M, threads))
    t0 = time.perf_counter()
    fn(np.ascontiguousarray(w.A_host[:probe]), w.B_host, nthreads=threads)
    t_probe = time.perf_counter() - t0
    rows = int(max(probe, min(w.M, probe * seconds / max(t_probe, 1e-6))))
    rows = max(threads, (rows // threads) * threads) if rows >= threads else rows
    t0 = time.perf_counter()
    out = fn(np.ascontiguousarray(w.A_host[:rows]), w.B_host, nthreads=threads)
    t = time.perf_counter() - t0
    w.oracle_rows = (rows, out)          # kept for the full comparison of the timed output
    ops = 2.0 * rows * w.N * w.K
    cpu = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": round(ops / t / 1e12, 6), "unit": "TOPS" if w.dtype == "int8" else "TFLOP/s",
            "cores": threads, "kind": "oracle", "seconds": round(t, 3), "cpu_model": cpu,
            "sample": f"first {rows} of {w.M} rows of C for the same {w.dtype} {w.M}x{w.K}x{w.N} GEMM "
                      f"({rows * w.N} outputs, {ops:.3g} ops)"}


def mfma_ceiling(dtype: str, iters: int = 20000, launches: int = 3) -> dict:
    """Sustained MFMA rate with random operands in registers and no memory traffic
    (gemm_probe_mfma): the ceiling a GEMM on random inputs can reach at the clock the
    chip holds under that load.  Timed with HIP events on the launch stream."""
    import torch
    from paper_2512_13282_amd import binding
    d = binding.GEMM_DTYPE_I8_I32 if dtype == "int8" else binding.GEMM_DTYPE_BF16_F32
    rc, info = binding.gemm_probe_mfma(d, True, iters)
    if rc != 0:
        raise RuntimeError(binding.gemm_status_string(rc))
    wg = int(info["workgroups"])
    clocks = torch.zeros(2 * wg, dtype=torch.int64, device="cuda:0")
    sink = torch.zeros(wg * int(info["threads_per_workgroup"]), dtype=torch.int32, device="cuda:0")
    stream = torch.cuda.current_stream()
    ms = []
    for i in range(launches + 1):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        rc, _ = binding.gemm_probe_mfma(d, True, iters, clocks.data_ptr(), sink.data_ptr(), stream.cuda_stream)
        e1.record(stream)
        if rc != 0:
            raise RuntimeError(binding.gemm_status_string(rc))
        torch.cuda.synchronize()
        if i > 0:
            ms.append(e0.elapsed_time(e1))
    c = clocks.view(wg, 2).double().cpu()
    ghz = float((c[:, 0] / c[:, 1]).mean()) * info["wall_clock_hz"] / 1e9
    tops = info["ops_per_launch"] / (float(np.mean(ms)) * 1e-3) / 1e12
    return {"value": round(tops, 1), "unit": "TOPS" if dtype == "int8" else "TFLOP/s",
            "clock_ghz": round(ghz, 3), "frac_of_published_peak": round(tops / PEAK[dtype], 4)}


def write_traffic(fetch_csv: str, write_csv: str) -> None:
    """L2 -> fabric bytes (last-level cache and HBM) per launch of the timed GEMM kernels, from
    rocprofv3 counter CSVs.

    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are each scaled by the factor that
    makes them read the known traffic of the plain 512 MiB copy profiled in the same
    run (it reads 512 MiB and writes 512 MiB)."""
    import csv
    import collections

    def per_kernel(path, counter):
        vals = collections.defaultdict(list)
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == counter:
                vals[r["Kernel_Name"]].append(float(r["Counter_Value"]))
        return vals

    def copy_probe(vals):
        # The probe's elementwise launches: the fill of its source (reads nothing) and
        # three copies; the copies are the launches within 10% of the largest value.
        cand = [v for k, vs in vals.items() if "elementwise" in k for v in vs]
        if not cand:
            sys.exit("no copy-probe kernel in the counter CSV (run bench.py --copy-probe under rocprofv3)")
        top = max(cand)
        sel = [v for v in cand if v >= 0.9 * top]
        return sum(sel) / len(sel)

    fetch_v = per_kernel(fetch_csv, "FETCH_SIZE")
    write_v = per_kernel(write_csv, "WRITE_SIZE")
    f_scale = COPY_PROBE_BYTES / (copy_probe(fetch_v) * 1024.0)
    w_scale = COPY_PROBE_BYTES / (copy_probe(write_v) * 1024.0)
    fetch = {k: sum(v) / len(v) for k, v in fetch_v.items()}
    write = {k: sum(v) / len(v) for k, v in write_v.items()}
    S = 8192
    workloads = {}
    for k in fetch:
        # gemm_lds_kernel<dtype, BM, BN, WM, WN, waves/EU, B column-major> and
        # gemm_ring_kernel<..., B column-major, ring depth>: one plan per workload
        if "gemm::gemm_lds_kernel<" not in k and "gemm::gemm_ring_kernel<" not in k:
            continue
        targs = [t.strip() for t in k.split("<", 1)[1].split(">", 1)[0].split(",")]
        dtype = "int8" if targs[0] == "0" else "bf16"
        bt = targs[6] == "true"
        e = 1 if dtype == "int8" else 2
        comp = S * S * e * 2 + S * S * 4
        fb = fetch[k] * 1024.0 * f_scale
        wb = write.get(k, 0.0) * 1024.0 * w_scale
        workloads[f"{dtype}_{S}x{S}x{S}" + ("_bt" if bt else "")] = {
            "kernel": k, "fetch_bytes": round(fb), "write_bytes": round(wb),
            "bytes_per_launch": round(fb + wb), "algorithmic_bytes": comp,
            "traffic_over_algorithmic": round((fb + wb) / comp, 3)}
    out = {"kernel_source_sha256": kernel_sha(), "fetch_scale": round(f_scale, 4),
           "write_scale": round(w_scale, 4), "copy_probe_bytes": COPY_PROBE_BYTES,
           "counters": "rocprofv3 --pmc FETCH_SIZE / --pmc WRITE_SIZE, KiB per dispatch, averaged",
           "what": "bytes the XCD L2 caches request from / write to the fabric behind them, i.e. the "
                   "256 MB last-level cache (MALL) and HBM together: an upper bound on HBM traffic "
                   "(the counters do not separate MALL hits from HBM accesses)",
           "workloads": workloads}
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=2)
        f.write("\n")
    print(json.dumps(out, indent=2))


PAPER_SWEEP_SIZES = (256, 512, 1024, 2048, 3072, 4096, 6144, 8192)


def paper_sweep_run(out_dir: str, iters: int = 10) -> dict:
    """GEMM TOPS over every (M, K, N) in PAPER_SWEEP_SIZES^3 (multiples of the 256 tile up to
    8192), both dtypes and both B layouts, with the selector's plans.  Operands are drawn on the
    device (torch, seed 0) in the sweep's distributions and reused as views; each point is
    `iters` back-to-back launches after two warm-ups, queued behind a spin kernel and timed
    between two HIP events (the GPU's time per launch).  Returns a summary; every point goes to
    out_dir/paper_sweep.jsonl."""
    import torch
    from paper_2512_13282_amd import binding
    dev = torch.device("cuda:0")
    torch.manual_seed(0)
    S = max(PAPER_SWEEP_SIZES)
    st = torch.cuda.current_stream(dev)
    os.makedirs(os.path.join(ROOT, out_dir), exist_ok=True)
    summary = {"sizes": list(PAPER_SWEEP_SIZES), "points_per_series": len(PAPER_SWEEP_SIZES) ** 3}
    with open(os.path.join(ROOT, out_dir, "paper_sweep.jsonl"), "w") as f:
        for dtype in ("int8", "bf16"):
            if dtype == "int8":
                A = torch.randint(-128, 128, (S * S,), dtype=torch.int8, device=dev)
                B = torch.randint(-128, 128, (S * S,), dtype=torch.int8, device=dev)
                C = torch.empty(S * S, dtype=torch.int32, device=dev)
            else:
                A = torch.randn(S * S, device=dev).to(torch.bfloat16)
                B = torch.randn(S * S, device=dev).to(torch.bfloat16)
                C = torch.empty(S * S, dtype=torch.float32, device=dev)
            for bt in (False, True):
                fn = getattr(binding, ("gemm_i8_i32" if dtype == "int8" else "gemm_bf16_f32") + ("_bt" if bt else ""))
                tops = []
                for M in PAPER_SWEEP_SIZES:
                    for K in PAPER_SWEEP_SIZES:
                        for N in PAPER_SWEEP_SIZES:
                            ldb = K if bt else N
                            call = lambda: fn(M, N, K, A.data_ptr(), K, B.data_ptr(), ldb, C.data_ptr(), N,
                                              st.cuda_stream)
                            for _ in range(2):
                                if call() != 0:
                                    raise RuntimeError(f"GEMM failed at {(dtype, M, K, N, bt)}")
                            torch.cuda.synchronize()
                            spin_ahead(iters, 40.0)
                            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                            e0.record(st)
                            for _ in range(iters):
                                call()
                            e1.record(st)
                            torch.cuda.synchronize()
                            ms = e0.elapsed_time(e1) / iters
                            t = 2.0 * M * N * K / (ms * 1e-3) / 1e12
                            tops.append((t, M, K, N))
                            f.write(json.dumps({"dtype": dtype, "b_layout": "col" if bt else "row", "M": M,
                                                "K": K, "N": N, "kernel_ms": round(ms, 5),
                                                "tops": round(t, 2)}) + "\n")
                vals = np.array([x[0] for x in tops])
                best = max(tops)
                key = f"{dtype}_{'col' if bt else 'row'}_major_b"
                summary[key] = {"max": round(best[0], 1), "max_at_MKN": list(best[1:]),
                                "median": round(float(np.median(vals)), 1),
                                "quartiles": [round(float(np.percentile(vals, q)), 1) for q in (25, 75)],
                                "at_or_above_4096_cube_volume_median": round(float(np.median(
                                    [t for t, m_, k_, n_ in tops if m_ * k_ * n_ >= 4096 ** 3])), 1),
                                "points_at_or_above_40pct_peak": int(np.sum(vals >= 0.4 * PEAK[dtype])),
                                "unit": "TOPS" if dtype == "int8" else "TFLOP/s"}
                print(f"[paper-sweep] {key}: max {best[0]:.1f} at M,K,N={best[1:]}, median "
                      f"{np.median(vals):.1f}", file=sys.stderr, flush=True)
            del A, B, C
            torch.cuda.empty_cache()
    return summary


def main():
    args = parse()
    if args.traffic_from:
        write_traffic(*args.traffic_from)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py times one GPU: the library has no multi-GPU path (a GEMM would shard by "
              "output tiles, each GPU computing its own columns of C). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    from paper_2512_13282_amd import binding
    binding.lib()   # fails loudly if the HIP library is not built
    if args.config >= 0:
        for d in (binding.GEMM_DTYPE_I8_I32, binding.GEMM_DTYPE_BF16_F32):
            if binding.gemm_force_plan(d, binding.GEMM_KERNEL_AUTO, args.config, 0) != 0:
                sys.exit(f"cannot force config {args.config}")

    if args.workload:
        dtype, shape = args.workload.split(":")
        M, K, N = (int(x) for x in shape.split("x"))
        e = 1 if dtype == "int8" else 2
        copies = max(1, int(np.ceil(512e6 / (K * N * e))) + 1) if args.cold else 1
        w = Workload(dtype, M, N, K, copies=copies)
        ms, kavg, kmin = time_workload(w, args.steps, args.warmup, args.settle_ms)
        r = summarize(w, ms, kavg, kmin)
        r.update({"workload": args.workload, "b_copies": copies,
                  "parity_sample_ok": parity_sample(w, sorted({0, M // 2, M - 1}))})
        print(json.dumps(r), flush=True)
        return

    S = args.size
    from paper_2512_13282_amd import inputs
    heads = [(d, S, S, S) for d in (["int8", "bf16"] if args.only is None else [args.only])]
    # The per-workload table runs first: besides its own figures, it brings the chip to the
    # clock it holds under sustained GEMM load before the headline's warm-up and timed launches.
    table = None if args.no_configs else config_table(set(heads), args.config_steps, args.config_warmup,
                                                      0.0 if args.no_cpu_baseline else CONFIG_ORACLE_SECONDS,
                                                      args.settle_ms)

    results = {}
    for dtype in (["int8", "bf16"] if args.only is None else [args.only]):
        w = Workload(dtype, S, S, S)
        ms, kavg, kmin = time_workload(w, args.steps, args.warmup, args.settle_ms)
        r = summarize(w, ms, kavg, kmin)
        r["parity_sample_ok"] = parity_sample(w, [0, S // 2, S - 1])
        if not args.no_cpu_baseline:
            r["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
            r["parity_full"] = parity_full(w)
            w.oracle_rows = None
        results[dtype] = (w, r)
        print(f"[bench] {dtype} {S}^3: {r['value']} {r['unit']} ({r['pct_dense_peak']}% of dense peak), "
              f"kernel {r['kernel_ms_avg']} ms, plan {r['plan']}", file=sys.stderr, flush=True)
        del w

    bt_results = {}
    if not args.no_bt:
        for dtype in (["int8", "bf16"] if args.only is None else [args.only]):
            w = Workload(dtype, S, S, S, bt=True)
            ms, kavg, kmin = time_workload(w, args.steps, args.warmup, args.settle_ms)
            r = summarize(w, ms, kavg, kmin)
            r["parity_sample_ok"] = parity_sample(w, [0, S // 2, S - 1])
            bt_results[dtype] = {k: r[k] for k in ("value", "unit", "ms_per_step", "kernel_ms_avg",
                                                   "pct_dense_peak", "plan", "split_k", "parity_sample_ok",
                                                   "roofline")}
            print(f"[bench] {dtype} {S}^3 column-major B: {r['value']} {r['unit']} ({r['pct_dense_peak']}% of "
                  f"dense peak), kernel {r['kernel_ms_avg']} ms, plan {r['plan']}", file=sys.stderr, flush=True)
            del w

    reduced = {}
    if args.reduced:
        for dtype, out in (("int8", "i8"), ("bf16", "bf16")):
            if args.only is not None and args.only != dtype:
                continue
            w = Workload(dtype, S, S, S, out=out)
            ms, kavg, kmin = time_workload(w, args.steps, args.warmup, args.settle_ms)
            r = summarize(w, ms, kavg, kmin)
            r["parity_sample_ok"] = parity_sample(w, [0, S // 2, S - 1])
            key = "int8_to_int8" if dtype == "int8" else "bf16_to_bf16"
            reduced[key] = {k: r[k] for k in ("value", "unit", "ms_per_step", "kernel_ms_avg", "pct_dense_peak",
                                              "plan", "split_k", "parity_sample_ok", "roofline")}
            print(f"[bench] {key} {S}^3: {r['value']} {r['unit']} ({r['pct_dense_peak']}% of dense peak), "
                  f"kernel {r['kernel_ms_avg']} ms, plan {r['plan']}", file=sys.stderr, flush=True)
            del w

    paper_sweep = paper_sweep_run(args.out_dir) if args.paper_sweep else None

    if args.copy_probe:
        # Elementwise copy of 512 MiB: reads 512 MiB, writes 512 MiB.  Profiled beside the
        # GEMM so FETCH_SIZE / WRITE_SIZE can be scaled by what they read for known traffic.
        src = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst

    if args.sweep:
        from paper_2512_13282_amd import inputs
        os.makedirs(os.path.join(ROOT, args.out_dir), exist_ok=True)
        with open(os.path.join(ROOT, args.out_dir, "sweep.jsonl"), "w") as f:
            for (dtype, M, K, N) in (inputs.SKINNY if args.sweep_set == "skinny" else inputs.ALL_CONFIGS):
                e = 1 if dtype == "int8" else 2
                bbytes = K * N * e
                copies = 1 if M >= 256 else max(1, int(np.ceil(512e6 / bbytes)) + 1)
                w = Workload(dtype, M, N, K, copies=copies)
                ms, kavg, kmin = time_workload(w, max(20, args.steps // 2), args.warmup, args.settle_ms)
                r = summarize(w, ms, kavg, kmin)
                r.update({"dtype": dtype, "M": M, "K": K, "N": N, "b_copies": copies})
                r["parity_sample_ok"] = parity_sample(w, sorted({0, M - 1}))
                f.write(json.dumps(r) + "\n")
                print(f"[sweep] {dtype:4s} M={M:5d} K={K:6d} N={N:6d} {r['value']:9.2f} {r['unit']:7s} "
                      f"{r['pct_dense_peak']:6.2f}% kernel {r['kernel_ms_avg']*1e3:9.1f} us "
                      f"{r['roofline']['bound']} frac={r['roofline']['frac']:.3f} plan={r['plan']} "
                      f"split={r['split_k']} ok={r['parity_sample_ok']}", file=sys.stderr, flush=True)
                del w
                torch.cuda.empty_cache()

    ceiling = {}
    if not args.no_ceiling:
        for dtype in results:
            ceiling[dtype] = mfma_ceiling(dtype)
            ceiling[dtype]["gemm_frac_of_ceiling"] = round(results[dtype][1]["roofline"]["achieved"] /
                                                           ceiling[dtype]["value"], 4)
            print(f"[bench] {dtype} sustained MFMA ceiling (random operands, no memory traffic): "
                  f"{ceiling[dtype]['value']} at {ceiling[dtype]['clock_ghz']} GHz; GEMM kernel reaches "
                  f"{ceiling[dtype]['gemm_frac_of_ceiling']:.3f} of it", file=sys.stderr, flush=True)

    if table is not None and ceiling:
        # every MFMA-bound row against the same run's sustained MFMA rate: the clock-adjusted peak
        for row in table:
            c = ceiling.get(row["dtype"])
            if c and row["roofline"]["bound"] == "mfma":
                row["frac_of_mfma_ceiling"] = round(row["value"] / c["value"], 4)
        print("[configs] fraction of the sustained MFMA ceiling: " +
              ", ".join(f"{r['dtype']} {r['M']}x{r['K']}x{r['N']} {r['frac_of_mfma_ceiling']:.3f}"
                        for r in table if "frac_of_mfma_ceiling" in r), file=sys.stderr, flush=True)

    head_dtype = args.only or "int8"
    hw, hr = results[head_dtype]
    line = {
        "metric": f"GEMM {'TOPS int8->int32' if head_dtype == 'int8' else 'TFLOP/s bf16->fp32'} "
                  f"M=N=K={S} on 1 MI355X (% of dense MFMA peak in pct_dense_peak)",
        "value": hr["value"], "unit": hr["unit"], "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "settle_ms": args.settle_ms, "ms_per_step": hr["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None,
        "dtype": "i8" if head_dtype == "int8" else "bf16",
        "data": "synthetic: A, B seeded (PCG64 seed 0 / 1); int8 uniform [-128,127], bf16 N(0,1) rounded RNE",
        "config": {"workload": f"{head_dtype} GEMM M=N=K={S}, row-major A, B, C "
                               f"({'int32' if head_dtype == 'int8' else 'fp32'} output)",
                   "M": S, "N": S, "K": S, "plan": hr["plan"], "split_k": hr["split_k"]},
        "pct_dense_peak": hr["pct_dense_peak"],
        "kernel_ms_avg": hr["kernel_ms_avg"],
        "parity_sample_ok": hr["parity_sample_ok"],
        "parity_full_ok": (hr.get("parity_full") or {}).get("ok"),
        "parity_full": hr.get("parity_full"),
        "roofline": hr["roofline"],
        "cpu_baseline": hr.get("cpu_baseline"),
    }
    for dtype, (w, r) in results.items():
        if dtype != head_dtype:
            line[dtype] = {k: r.get(k) for k in ("value", "unit", "ms_per_step", "kernel_ms_avg", "pct_dense_peak",
                                                "plan", "split_k", "parity_sample_ok", "parity_full", "roofline",
                                                "cpu_baseline")}
    if table is not None:
        line["configs"] = table
    if ceiling:
        line["mfma_ceiling"] = {"method": "gemm_probe_mfma: only the GEMM's MFMA instructions on random "
                                          "operands held in registers, one 8-wave workgroup per CU, no memory "
                                          "traffic; HIP-event timed", **ceiling}
    if bt_results:
        line["column_major_b"] = {"workload": f"the same GEMMs with B stored column-major (N x K), "
                                              f"gemm_*_bt entry points", **bt_results}
    if reduced:
        line["reduced_outputs"] = {"workload": f"the same {S}^3 GEMMs with narrowed outputs: int8 -> int8 "
                                               f"(results / 2^{REQUANT_SHIFT}, nearest-even, saturated) and "
                                               f"bf16 -> bf16 (nearest-even)", **reduced}
    if paper_sweep is not None:
        line["paper_sweep"] = paper_sweep
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
