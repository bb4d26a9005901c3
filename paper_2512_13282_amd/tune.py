"""On-device plan tuning: measure candidate plans and record the fastest.

The selector's analytical model (compute vs memory time, wave quantization,
split-K traffic) gives a starting point; this tool then measures the
candidate (configuration, split-K) plans of each shape on the GPU and writes
the fastest into ``csrc/tuned_plans.inc``, which the selector consults before
its model for an exactly matching, suitably aligned shape -- the paper's
procedure of refining the modelled tile choice by measurement on the device
(Sec. 4.5.2).  Rebuild the library afterwards.  With --plans-out the plans go
instead to a plan file that gemm_load_plans / GEMM_MI355X_PLANS load at run time,
no rebuild needed (--out as well writes both).

    python -m paper_2512_13282_amd.tune [--shapes default|FILE] [--out PATH] [--plans-out PATH] [--iters N]

Every plan is first timed in a short burst (the median of --iters launches); the
fastest --confirm plans, plus the fastest of each split-K reduction, are then
re-timed over several interleaved rounds of 50 launches after 30 untimed ones,
the regime of a long run of GEMMs on a chip whose power manager has settled, and
the choice is made on those times.

Shapes default to the paper-shaped workload sweep (see inputs.py) with B
row-major, plus the skinny and 8192^3 workloads with B stored column-major
(the *_bt entry points), and the decode and prefill rows of transformer
projection sizes with both layouts.  A shapes file lists [dtype, M, K, N] or
[dtype, M, K, N, "bt"].  Memory-bound shapes (M < 256) are timed with B cold:
the launches rotate through enough copies of B to exceed the 256 MB last-level
cache.  So are the decode and prefill rows of the default list at every size
(a layer's weights come from HBM), and with --cold every shape; the square and
rectangle workloads are timed warm, as the benchmark times them.  The two
cache-sized workloads (int8 256^3, bf16 1024^3) are timed as lone launches
after a 512 MiB flush.  Back-to-back launches queue behind a
spin kernel so that short kernels are timed on the GPU, not on the host's
launch rate.
"""
from __future__ import annotations

import argparse
import json
import os
import sys

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(PKG, "csrc", "tuned_plans.inc")
SPLITS_SMALL_M = (1, 2, 3, 4, 6, 8, 12, 16, 24, 32, 48, 64, 96, 128)
SPLITS_LARGE = (1, 2, 3, 4)


_SPIN_RATE = None


def _spin_ahead(launches, host_us_per_launch=80.0):
    """Queues a spin kernel long enough for the host to enqueue `launches` more launches behind
    it, so that short kernels run back to back and are timed on the GPU, not on the host's
    launch rate; the spin's cycles per microsecond are measured once."""
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


def _time(fn, copies, iters):
    import torch
    for i in range(3):
        fn(i % copies)
    torch.cuda.synchronize()
    _spin_ahead(iters)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(iters)]
    for i in range(iters):
        ev[i][0].record()
        fn(i % copies)
        ev[i][1].record()
    torch.cuda.synchronize()
    return float(np.median([a.elapsed_time(b) for a, b in ev])) * 1e3   # us


def _time_flushed(fn, iters):
    """Median time of single launches, each after a 512 MiB write that evicts the operands
    from the L2s and the last-level cache: the protocol for shapes whose operands fit in the
    caches (a lone GEMM of that size finds them cold)."""
    import torch
    scratch = torch.empty(128 * 1024 * 1024, dtype=torch.float32, device="cuda:0")
    fn(0)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(iters)]
    for i in range(iters):
        scratch.fill_(float(i))
        ev[i][0].record()
        fn(0)
        ev[i][1].record()
    torch.cuda.synchronize()
    del scratch
    return float(np.median([a.elapsed_time(b) for a, b in ev])) * 1e3   # us


def _time_sustained(fn, copies, warmup, iters):
    """Average time of `iters` back-to-back launches after `warmup` untimed ones: the regime
    of a long run of GEMMs, in which the chip's power manager has settled."""
    import torch
    for i in range(warmup):
        fn(i % copies)
    _spin_ahead(iters, 40.0)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(iters):
        fn(i % copies)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / iters * 1e3   # us


def tune_shape(dtype: str, M: int, N: int, K: int, iters: int, log=print, bt: bool = False,
               confirm: int = 3, rounds: int = 3, cold_single: bool = False, cold_b: bool = False):
    """cold_b: B comes from HBM at every launch (launches rotate through copies of B past
    the last-level cache), as a layer's weights do in a model's forward pass; always the
    case below 256 rows, where reading B is most of the work."""
    import torch
    from . import binding as b
    d = b.GEMM_DTYPE_I8_I32 if dtype == "int8" else b.GEMM_DTYPE_BF16_F32
    e = 1 if dtype == "int8" else 2
    dev = torch.device("cuda:0")
    copies = int(np.ceil(600e6 / (K * N * e))) if (M < 256 or cold_b) else 1
    b_shape, ldb = ((N, K), K) if bt else ((K, N), N)
    if dtype == "int8":
        A = torch.randint(-128, 128, (M, K), dtype=torch.int8, device=dev)
        Bs = [torch.randint(-128, 128, b_shape, dtype=torch.int8, device=dev) for _ in range(copies)]
        C = torch.empty(M, N, dtype=torch.int32, device=dev)
        fn0 = b.gemm_i8_i32_bt if bt else b.gemm_i8_i32
    else:
        A = torch.randn(M, K, device=dev).to(torch.bfloat16)
        Bs = [torch.randn(*b_shape, device=dev).to(torch.bfloat16) for _ in range(copies)]
        C = torch.empty(M, N, dtype=torch.float32, device=dev)
        fn0 = b.gemm_bf16_f32_bt if bt else b.gemm_bf16_f32
    stream = torch.cuda.current_stream().cuda_stream

    def run(i):
        rc = fn0(M, N, K, A.data_ptr(), K, Bs[i].data_ptr(), ldb, C.data_ptr(), N, stream)
        if rc != 0:
            raise RuntimeError(b.gemm_status_string(rc))

    results = []
    measured = set()
    n_cfg = 0
    while b.gemm_force_plan(d, b.GEMM_KERNEL_AUTO, n_cfg, 0) == 0:
        n_cfg += 1
    try:
        for cfg in range(n_cfg):
            for split in (SPLITS_SMALL_M if M < 256 else SPLITS_LARGE):
                reductions = (0, 1, 2, 3) if dtype == "int8" else (0, 1)   # atomic: int8 only
                for reduce in ((-1,) if split == 1 else reductions):
                    if b.gemm_force_plan(d, b.GEMM_KERNEL_AUTO, cfg, split) != 0:
                        continue
                    b.gemm_force_reduce(d, reduce)
                    try:
                        plan = b.gemm_plan(d, M, N, K, K, ldb, N, A.data_ptr(), Bs[0].data_ptr(),
                                           C.data_ptr(), trans_b=bt)
                    except b.GemmError:
                        continue            # configuration cannot run this shape
                    if plan["kernel"] == b.GEMM_KERNEL_GENERIC:
                        continue
                    key = (cfg, plan["split_k"], plan["reduce_in_kernel"] if plan["split_k"] > 1 else -1)
                    if key in measured:
                        continue            # the split clamped to one already measured
                    measured.add(key)
                    us = _time_flushed(run, iters) if cold_single else _time(run, copies, iters)
                    results.append({"config": cfg, "split": plan["split_k"],
                                    "reduce": plan["reduce_in_kernel"] if plan["split_k"] > 1 else -1,
                                    "name": plan["name"], "us": us})
        # The screening above times each plan in a short burst; a chip that has been busy for
        # a while holds a lower clock, and the plans do not all slow down alike.  The fastest
        # few are therefore timed again, interleaved over several rounds, after a warm-up long
        # enough for the power manager to settle, and the choice is made on those times.
        top = sorted(results, key=lambda r: r["us"])[:max(1, confirm)]
        # The two regimes also rank the split-K reductions differently (the burst puts the
        # atomic reduction's zeroing launch, which runs ahead of the GEMM, 1-2 us behind the
        # separate reduction that it beats in sustained runs), so the fastest screened plan
        # of every reduction is confirmed too.
        for mode in sorted({r["reduce"] for r in results} - {-1}):
            best_of_mode = min((r for r in results if r["reduce"] == mode), key=lambda r: r["us"])
            if best_of_mode not in top:
                top.append(best_of_mode)
        if len(top) > 1:
            times = [[] for _ in top]
            for _ in range(rounds):
                for t, cand in enumerate(top):
                    b.gemm_force_plan(d, b.GEMM_KERNEL_AUTO, cand["config"], cand["split"])
                    b.gemm_force_reduce(d, cand["reduce"] if cand["split"] > 1 else -1)
                    times[t].append(_time_flushed(run, 30) if cold_single else _time_sustained(run, copies, 30, 50))
            for t, cand in enumerate(top):
                cand["us_sustained"] = float(np.median(times[t]))
    finally:
        b.gemm_force_plan(d, b.GEMM_KERNEL_AUTO, -1, 0)
        b.gemm_force_reduce(d, -1)
    best = min(top, key=lambda r: r.get("us_sustained", r["us"]))
    log(f"{dtype} M={M} K={K} N={N}{' (B column-major)' if bt else ''}{' (B cold)' if copies > 1 else ''}: "
        f"best {best['name']} split {best['split']} reduce {best['reduce']} "
        f"{best.get('us_sustained', best['us']):.1f} us sustained, {best['us']:.1f} us burst ({len(results)} plans)")
    del A, Bs, C
    torch.cuda.empty_cache()
    return best, results


def write_inc(entries, path=OUT):
    lines = ["// Generated by `python -m paper_2512_13282_amd.tune` from on-device measurements",
             "// (fastest plan per shape over sustained runs of back-to-back launches).  Fields: dtype, M, N, K, config, split_k, reduce,",
             "// (split-K reduction: 0 separate kernel, 1 in-kernel by the last slice, 2 atomic adds into C zeroed by a fill kernel, 3 atomic adds into C zeroed by the first slice, -1 the model's choice), B layout",
             "// (1: column-major).",
             "// Consulted by select_plan before the analytical model for an exact shape match."]
    for e in entries:
        lines.append(f"    {{{e['dtype']}, {e['M']}, {e['N']}, {e['K']}, {e['config']}, {e['split']}, "
                     f"{e['reduce']}, {e.get('trans_b', 0)}}},  // {e['name']} {e.get('us_sustained', e['us']):.1f} us")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def write_plan_file(entries, path):
    """The run-time plan file format of gemm_load_plans: one plan per line,
    "dtype M N K config split reduce trans_b", '#' comments."""
    lines = ["# gemm_mi355x plans measured by `python -m paper_2512_13282_amd.tune`",
             "# dtype M N K config split reduce trans_b"]
    for e in entries:
        lines.append(f"{e['dtype']} {e['M']} {e['N']} {e['K']} {e['config']} {e['split']} {e['reduce']} "
                     f"{e.get('trans_b', 0)}  # {e['name']} {e.get('us_sustained', e['us']):.1f} us")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def default_shapes():
    """The default shape list, as (dtype, M, K, N[, "bt"]) tuples, and the set of
    (dtype, M, K, N) timed with B warm: the benchmark's square and rectangle workloads,
    which it times warm; every other shape models a layer whose weights come from HBM."""
    from . import inputs
    extra = inputs.DECODE + inputs.PREFILL + inputs.MORE_LAYERS + inputs.PREFILL_LONG + inputs.ODD_LAYERS
    shapes = [tuple(s) for s in inputs.ALL_CONFIGS + extra]
    shapes += [tuple(s) + ("bt",) for s in inputs.SKINNY + extra + [c for c in inputs.SQUARE if c[1] == 8192]]
    shapes = list(dict.fromkeys(shapes))        # the rectangle workloads recur among the prefill rows
    return shapes, set(map(tuple, inputs.SQUARE + inputs.RECT))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--shapes", default="default", help="'default' or a JSON file of [dtype, M, K, N] lists")
    ap.add_argument("--out", default=None,
                    help="compiled plan table to write (default: csrc/tuned_plans.inc, unless --plans-out is given)")
    ap.add_argument("--plans-out", default=None, help="write the plans as a run-time plan file (gemm_load_plans)")
    ap.add_argument("--json", default=None, help="also write every measurement here")
    ap.add_argument("--iters", type=int, default=15, help="launches per plan in the screening burst")
    ap.add_argument("--cold", action="store_true",
                    help="time every shape with B cold (default: below 256 rows, and in the default shape "
                         "list every shape but the benchmark's warm-timed workloads)")
    ap.add_argument("--confirm", type=int, default=3,
                    help="re-time this many of the fastest plans in the sustained regime and choose among them")
    args = ap.parse_args()
    sys.path.insert(0, os.path.dirname(PKG))
    from . import inputs
    if args.shapes == "default":
        shapes, warm = default_shapes()
    else:
        shapes = [tuple(s) for s in json.load(open(args.shapes))]
        warm = None
    entries, everything = [], []
    for shape in shapes:
        dtype, M, K, N = shape[:4]
        bt = len(shape) > 4 and shape[4] == "bt"
        # Shapes whose operands fit in the caches are timed as lone launches on cold caches.
        cold_single = (dtype, M, K, N) in inputs.SMALL
        cold_b = args.cold or (warm is not None and (dtype, M, K, N) not in warm)
        best, res = tune_shape(dtype, M, N, K, args.iters, bt=bt, confirm=args.confirm, cold_single=cold_single,
                               cold_b=cold_b)
        entries.append({"dtype": 0 if dtype == "int8" else 1, "M": M, "N": N, "K": K, "trans_b": int(bt), **best})
        everything.append({"dtype": dtype, "M": M, "K": K, "N": N, "bt": bt, "results": res})
    out = args.out or (None if args.plans_out else OUT)
    if out:
        write_inc(entries, out)
    if args.plans_out:
        write_plan_file(entries, args.plans_out)
    if args.json:
        with open(args.json, "w") as f:
            json.dump(everything, f)
    print(f"wrote {', '.join(p for p in (out, args.plans_out) if p)} ({len(entries)} shapes)")


if __name__ == "__main__":
    main()
