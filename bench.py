#!/usr/bin/env python3
"""Benchmark of the emulated batched SGEMM on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME]
                    [--flow F --ec E --tile T] [--no-cpu-baseline]

A step is one sgemm_emu_batched call over the whole batch of the workload
(every step of the path: operand loads, split, three MFMA products, combine
and store), with inputs already resident in HBM, under the policy the
library picks for it (or the one given).  The default workload is the
largest configuration, one 8192 x 8192 x 8192 product (uniform(-1, 1) FP32,
seed 4): the one bound by the matrix units, where the emulation's rate is
measured against one third of the fp16 MFMA peak.

The roofline's "traffic" is the HBM traffic a counter run measured for this
workload and kernel (profiles/traffic.json), reported only while the
kernel's sources are unchanged since that run.

One JSON line is printed with the emulated TFLOP/s, the roofline of the
dominant kernel (its average duration from HIP events recorded on the stream
the kernel is launched on), the median, minimum and maximum of single
launches (from an event recorded after every call of the timed region) and,
as a reported baseline, the oracle's plain FP32 product timed on the host
cores for a bounded sample of the same workload; the accuracy of the GPU
result on that sample is reported with it.

``--copy-calibration`` instead runs a plain device copy of known size, used
to scale the HBM traffic counters of a profiler run; ``--hbm-probe`` times the
batched workloads' memory traffic without their arithmetic, the reference
their HBM fraction is read against; ``--mfma-probe`` times the 8192^3
product's arithmetic without its data movement, the reference its matrix-unit
fraction is read against at the clock the device holds.
"""
from __future__ import annotations

import argparse
import dataclasses
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import torch  # noqa: E402

import paper_2308_15152_amd as pkg  # noqa: E402
import synth  # noqa: E402

# MI355X published peaks
PEAK_HBM_GBS = 8000.0
PEAK_FP16_MFMA_TFLOPS = 2516.6   # dense
PEAK_FP32_VECTOR_TFLOPS = 157.3

METRIC = "emulated-SGEMM TFLOP/s (batched)"
SCAN_METRIC = "inclusive scan of FP32 rows, elements/s (batched)"

# HBM traffic measured with rocprofv3 counters (FETCH_SIZE, WRITE_SIZE), per
# workload, with the hash of the kernel sources it was taken on
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


KERNEL_SOURCES = {  # the translation unit of each kernel; shared headers are added
    "bgemm_reg_kernel": "bgemm_reg.hip",
    "bgemm_big_kernel": "bgemm_big.hip",
    "bgemm_big_stream_kernel": "bgemm_big.hip",
    "bgemm_emu_kernel": "bgemm.hip",
    "householder64_kernel": "rulebuilt.hip",
    "householder64_lds_kernel": "rulebuilt.hip",
    "givens64_kernel": "rulebuilt.hip",
    "givens64_lds_kernel": "rulebuilt.hip",
    "gemm_acc_kernel": "gemm_acc.hip",
    "scan_kernel": "scan.hip",
}


def _code_text(text: str) -> str:
    """Source text with comments removed and whitespace collapsed, so that a
    change to comments alone does not count as a change of the kernel."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash(kernel: str) -> str:
    """SHA-256 over the code (comments and layout ignored) a kernel is built
    from: its translation unit and every header it includes (transitively,
    quoted includes found in the package's csrc/ or in include/)."""
    csrc = os.path.join(ROOT, "paper_2308_15152_amd", "csrc")
    inc = os.path.join(ROOT, "include")
    seen, todo = set(), [os.path.join(csrc, KERNEL_SOURCES[kernel])]
    while todo:
        f = todo.pop()
        if f in seen:
            continue
        seen.add(f)
        with open(f) as fh:
            for name in re.findall(r'^\s*#\s*include\s+"([^"]+)"', fh.read(), flags=re.M):
                for d in (os.path.dirname(f), csrc, inc):
                    cand = os.path.normpath(os.path.join(d, name))
                    if os.path.exists(cand):
                        todo.append(cand)
                        break
    h = hashlib.sha256()
    for f in sorted(seen):
        h.update(os.path.relpath(f, ROOT).encode())
        with open(f) as fh:
            h.update(_code_text(fh.read()).encode())
    return h.hexdigest()


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch from the committed counter runs, or None if there
    are none for this workload and kernel or the kernels changed since."""
    try:
        with open(TRAFFIC_FILE) as fh:
            table = json.load(fh)
    except (OSError, ValueError):
        return None
    e = table.get(workload)
    if not e or e.get("kernel") != kernel or e.get("source_sha256") != kernel_source_hash(kernel):
        return None
    return int(round((e["fetch_kib"] * e["fetch_scale"] + e["write_kib"] * e["write_scale"])
                     * 1024))




GIVENS_MODES = {"auto": pkg.GIVENS_AUTO, "map": pkg.GIVENS_MAP,
                "embedded": pkg.GIVENS_EMBEDDED, "lds": pkg.GIVENS_LDS}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="gemm_8192", choices=sorted(synth.WORKLOADS))
    ap.add_argument("--flow", type=int, default=pkg.FLOW_AUTO)
    ap.add_argument("--ec", type=int, default=1)
    ap.add_argument("--tile", type=int, default=pkg.TILE_AUTO)
    ap.add_argument("--givens-mode", default="auto", choices=sorted(GIVENS_MODES),
                    help="how a Givens workload builds G: map with (i, j) as kernel "
                         "arguments, map with (i, j) compiled in, G stored in LDS, or the "
                         "library's choice")
    ap.add_argument("--householder-mode", default="rule", choices=["rule", "lds"],
                    help="Householder workload: reflector built in registers (rule) or the "
                         "baseline through LDS")
    ap.add_argument("--batch", type=int, default=None,
                    help="override the workload's batch size (a measurement variant, "
                         "recorded in config; the default line uses the workload's own)")
    ap.add_argument("--graph", action="store_true",
                    help="capture the K timed steps in one HIP graph (torch.cuda.CUDAGraph) "
                         "and time one replay of it: per-step time without the host's "
                         "launch overhead, for launch-bound workloads")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-launch-spread", action="store_true",
                    help="record no event between the timed calls (each adds about 2 us of host "
                         "time per call, which shows only where the host's launch rate sets the "
                         "step time); per_launch is then null")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="target host time of the CPU-baseline sample")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--fp16-reference", action="store_true",
                    help="time the vendor library's plain fp16 and bf16 GEMM (torch.mm) on the "
                         "workload's shape: the matrix-unit rate a tuned GEMM reaches on this "
                         "device and clock, context for the emulation's three products (one line "
                         "per dtype; not the benchmark's value)")
    ap.add_argument("--mfma-probe", action="store_true",
                    help="time the full-tile kernel's products alone on the workload's shape "
                         "(sgemm_emu_mfma_probe): the rate the matrix units reach for them at the "
                         "clock the device holds; one line, not the benchmark's value")
    ap.add_argument("--hbm-probe", action="store_true",
                    help="time the read-A, read-B, write-C traffic of the batched square "
                         "workloads without their arithmetic (sgemm_emu_stream_probe) at 256, 512 "
                         "and 1024 threads per item; one line per case")
    ap.add_argument("--paper-sweep", action="store_true",
                    help="time the batched experiment of Sec. 4.4.2 (256 products of "
                         "1024 x k . k x 1024) for every k of the sweep; one line per k")
    return ap.parse_args()


def copy_calibration(steps: int):
    """Plain device-to-device copy of 1 GiB, for counter calibration."""
    n = 1 << 28
    x = torch.rand(n, device="cuda")
    y = torch.empty_like(x)
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        y.copy_(x)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "steps": steps,
                      "ms_per_copy": dt * 1e3, "GBps": 8 * n / dt / 1e9}), flush=True)


def hbm_probe(steps: int, warmup: int):
    """The HBM rate the batched products' access pattern reaches without
    arithmetic: items of A, B, C with the workload's item sizes, one
    workgroup per item reading A and B and writing C (nontemporal), timed
    with HIP events on the stream the probe runs on."""
    for name in ("gemm_128", "gemm_256e"):
        w = synth.WORKLOADS[name]
        assert w.m == w.n == w.k
        A = torch.rand((w.batch, w.m, w.k), device="cuda")
        B = torch.rand((w.batch, w.k, w.n), device="cuda")
        C = torch.empty((w.batch, w.m, w.n), device="cuda")
        nbytes = 3 * A.numel() * 4
        for threads in (256, 512, 1024):
            for _ in range(warmup):
                pkg.sgemm_emu_stream_probe(A, B, C, threads=threads)
            stream = torch.cuda.current_stream()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(steps):
                pkg.sgemm_emu_stream_probe(A, B, C, threads=threads)
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / steps
            ok = bool(torch.equal(C[-1], A[-1] + B[-1]))
            print(json.dumps({"probe": "read A, read B, write C", "items_like": name,
                              "items": w.batch, "item_bytes": A[0].numel() * 4,
                              "threads_per_item": threads, "bytes": nbytes, "steps": steps,
                              "us_per_launch": ms * 1e3, "GBps": nbytes / (ms * 1e-3) / 1e9,
                              "frac_of_8TBps": nbytes / (ms * 1e-3) / 8e12, "checked": ok}),
                  flush=True)
        del A, B, C
        torch.cuda.empty_cache()


def fp16_reference(name: str, steps: int, warmup: int, dtypes=("fp16", "bf16"), quiet=False):
    """The vendor library's plain half-precision GEMM on the workload's
    shape (one product of each item, as a batched matmul), timed with HIP
    events: how fast a tuned single fp16 product runs here.  The emulation
    issues three such products, so a third of this rate is what it would
    reach at the same matrix-unit efficiency.  Returns the records."""
    w = synth.WORKLOADS[name]
    assert w.kind == "gemm"
    out = []
    for label in dtypes:
        dt = {"fp16": torch.float16, "bf16": torch.bfloat16}[label]
        A = torch.rand((w.batch, w.m, w.k), device="cuda", dtype=dt)
        B = torch.rand((w.batch, w.k, w.n), device="cuda", dtype=dt)
        C = torch.empty((w.batch, w.m, w.n), device="cuda", dtype=dt)

        def call():
            if w.batch == 1:
                torch.mm(A[0], B[0], out=C[0])
            else:
                torch.bmm(A, B, out=C)
        for _ in range(warmup):
            call()
        stream = torch.cuda.current_stream()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(steps):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        tf = w.flops / (ms * 1e-3) / 1e12
        rec = {"reference": f"torch {'mm' if w.batch == 1 else 'bmm'} {label}",
               "workload": name, "steps": steps, "ms_per_step": ms, "TFLOPs": tf,
               "frac_of_dense_peak": tf / PEAK_FP16_MFMA_TFLOPS,
               "emulation_at_same_efficiency_TFLOPs": tf / 3}
        out.append(rec)
        if not quiet:
            print(json.dumps(rec), flush=True)
        del A, B, C
        torch.cuda.empty_cache()
    return out


def mfma_ceiling(name: str, steps: int, warmup: int, quiet=False):
    """The full-tile kernel's three products alone on the workload's shape
    (sgemm_emu_mfma_probe: same grid, waves and MFMA sequence on 128 x 256
    tiles, operand fragments held in registers, no loads, split or LDS
    traffic in the k loop), timed with HIP events: the rate the matrix units
    reach for these products at the clock the device holds under them.
    Returns the record."""
    w = synth.WORKLOADS[name]
    if w.kind != "gemm" or w.batch != 1 or w.m % 128 or w.n % 256 or w.k % 32:
        raise SystemExit(f"--mfma-probe needs one product of full 128 x 256 tiles, not {name}")
    g = torch.Generator(device="cuda").manual_seed(w.seed)
    A = torch.rand((w.m, 32), device="cuda", generator=g) * 2 - 1
    B = torch.rand((32, w.n), device="cuda", generator=g) * 2 - 1
    C = torch.empty((w.m, w.n), device="cuda")

    def call():
        pkg.sgemm_emu_mfma_probe(A, B, w.k, C)
    for _ in range(warmup):
        call()
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    tf = w.flops / (ms * 1e-3) / 1e12
    rec = {"reference": "the products alone (sgemm_emu_mfma_probe, kernel mfma_probe_kernel)",
           "workload": name, "steps": steps, "ms_per_step": ms, "TFLOPs": tf,
           "fp16_mfma_TFLOPs": 3 * tf, "frac_of_dense_peak": 3 * tf / PEAK_FP16_MFMA_TFLOPS}
    if not quiet:
        print(json.dumps(rec), flush=True)
    del A, B, C
    torch.cuda.empty_cache()
    return rec


def make_call(w, inputs, policy, givens_mode=pkg.GIVENS_AUTO, hh_mode=pkg.HOUSEHOLDER_RULE):
    if w.kind == "givens":
        c, s, B = inputs
        C = torch.empty((w.batch, w.m, w.n), dtype=torch.float32, device="cuda")
        i, j = w.plane

        def call():
            pkg.givens_emu_batched(i, j, c, s, B, C, mode=givens_mode)
        return call, C
    if w.kind == "scan":
        (X,) = inputs
        Y = torch.empty_like(X)

        def call():
            pkg.sgemm_emu_scan(X, Y)
        return call, Y
    if w.kind == "gemm_acc":
        At, B, Cin = inputs
        D = torch.empty((w.batch, w.m, w.n), dtype=torch.float32, device="cuda")

        def call():
            pkg.sgemm_emu_batched_acc(At, B, Cin, D, op_a=pkg.OP_T)
        return call, D
    if w.kind == "householder":
        u, B = inputs
        C = torch.empty((w.batch, w.m, w.n), dtype=torch.float32, device="cuda")

        def call():
            pkg.householder_emu_batched(u, B, C, mode=hh_mode)
        return call, C
    A, B = inputs
    C = torch.empty((w.batch, w.m, w.n), dtype=torch.float32, device="cuda")

    def call():
        pkg.sgemm_emu_batched(A, B, C, policy=policy)
    return call, C


def inputs_sha256(host_inputs) -> str:
    """SHA-256 of the input tensors' bytes, in the order they are drawn (the
    oracle and the device path see exactly these bytes)."""
    h = hashlib.sha256()
    for t in host_inputs:
        h.update(t.contiguous().numpy().tobytes())
    return h.hexdigest()


def cpu_baseline(w, host_inputs, C_dev, target_s: float):
    """The oracle's plain FP32 product on a bounded sample of the workload,
    timed on the host cores; the same sample gives the accuracy of the GPU
    result against the FP64 product."""
    import numpy as np

    import oracle

    threads = oracle.num_threads()
    if w.kind == "givens":
        c, s, B = host_inputs
        cn, sn, Bn = c.numpy(), s.numpy(), B.numpy()
        i, j = w.plane

        def run(items):
            return oracle.givens(i, j, cn, sn, Bn, items=items, want=("c32",))

        def ref(items):
            return oracle.givens(i, j, cn, sn, Bn, items=items, want=("c64", "n64", "c32"))
    elif w.kind == "scan":
        (X,) = host_inputs

        def run(items):
            return oracle.scan(X[items].numpy(), want=("c32",))

        def ref(items):
            return oracle.scan(X[items].numpy(), want=("c64", "n64", "c32"))
    elif w.kind == "gemm_acc":
        At, B, Cin = host_inputs

        def run(items):
            return oracle.gemm_acc(At[items].numpy(), B[items].numpy(), Cin[items].numpy(),
                                   "T", "N", want=("c32",))

        def ref(items):
            return oracle.gemm_acc(At[items].numpy(), B[items].numpy(), Cin[items].numpy(),
                                   "T", "N", want=("c64", "n64", "c32"))
    elif w.kind == "householder":
        u, B = host_inputs
        un, Bn = u.numpy(), B.numpy()

        def run(items):
            return oracle.householder(un, Bn, items=items, want=("c32",))

        def ref(items):
            return oracle.householder(un, Bn, items=items, want=("c64", "n64", "c32"))
    else:
        A, B = host_inputs

        def run(items):
            return oracle.gemm(A[items].numpy(), B[items].numpy(), want=("c32",))

        def ref(items):
            return oracle.gemm(A[items].numpy(), B[items].numpy(), want=("c64", "n64", "c32"))

    per_item = w.flops / w.batch
    scale, unit = (1e9, "Gelem/s") if w.kind == "scan" else (1e12, "TFLOP/s")
    if w.batch == 1:
        # one huge product: sample whole output rows instead of items,
        # calibrated at full parallelism (at least one row per thread) and
        # grown until the calibration takes an eighth of the target
        A, B = host_inputs
        rows = min(w.m, threads)
        while True:
            t0 = time.perf_counter()
            oracle.gemm(A[0, :rows].numpy()[None], B[0].numpy()[None], want=("c32",))
            dt = time.perf_counter() - t0
            if dt >= target_s / 8 or rows >= w.m:
                break
            rows = min(w.m, rows * 4)
        rows = min(w.m, max(rows, int(rows * target_s / max(dt, 1e-6))))
        t0 = time.perf_counter()
        oracle.gemm(A[0, :rows].numpy()[None], B[0].numpy()[None], want=("c32",))
        dt = time.perf_counter() - t0
        flops = 2.0 * rows * w.n * w.k
        g = np.random.default_rng(0)
        ri = g.integers(0, w.m, 256)
        ci = g.integers(0, w.n, 256)
        r = oracle.dots(A[0].numpy()[ri], np.ascontiguousarray(B[0].numpy()[:, ci].T),
                        want=("c64", "n64", "c32"))
        Cs = C_dev[0].cpu().numpy()[ri, ci]
        acc = {"max_rel_err_emu": oracle.max_rel_err(Cs, r["c64"], r["n64"]),
               "max_rel_err_fp32": oracle.max_rel_err(r["c32"], r["c64"], r["n64"]),
               "sample": "256 random elements"}
        sample = f"{rows} of {w.m} output rows of the {w.m}x{w.n}x{w.k} product"
        return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads,
                "kind": "oracle", "sample": sample, "seconds": dt, "host": host_cpu()}, acc

    # calibrate at full parallelism (at least one item per thread), growing
    # the sample until it takes an eighth of the target
    n = min(w.batch, threads)
    while True:
        t0 = time.perf_counter()
        run(list(range(n)))
        dt = time.perf_counter() - t0
        if dt >= target_s / 8 or n >= w.batch:
            break
        n = min(w.batch, n * 4)
    n = int(min(w.batch, max(n, n * target_s / max(dt, 1e-6))))
    items = list(range(n))
    # when the whole batch takes less than the target, time whole passes
    # until the target is reached
    reps = 0
    t0 = time.perf_counter()
    while True:
        run(items)
        reps += 1
        dt = time.perf_counter() - t0
        if n < w.batch or dt >= target_s:
            break
    acc_items = items[:min(n, 16)]
    r = ref(acc_items)
    Cs = C_dev[acc_items].cpu().numpy()
    acc = {"max_rel_err_emu": oracle.max_rel_err(Cs, r["c64"], r["n64"]),
           "max_rel_err_fp32": oracle.max_rel_err(r["c32"], r["c64"], r["n64"]),
           "sample": f"items 0..{len(acc_items) - 1}"}
    sample = f"{n} of {w.batch} batch items" + (f", {reps} passes" if reps > 1 else "")
    return {"value": per_item * n * reps / dt / scale, "unit": unit, "cores": threads,
            "kind": "oracle", "sample": sample, "seconds": dt, "host": host_cpu()}, acc


def host_cpu():
    """The host the CPU baseline ran on: CPU model, logical CPUs, and the CPUs
    this process may run on."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = None
    return {"model": model, "logical_cpus": os.cpu_count(), "usable_cpus": usable}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU (--gpus 1): the library runs on a single GPU; "
              "its batched workloads would shard by batch item with no communication, "
              "so each GPU would run this same measurement on its share", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    pkg.load()
    if args.copy_calibration:
        copy_calibration(args.steps)
        return
    if args.hbm_probe:
        hbm_probe(args.steps, args.warmup)
        return
    if args.fp16_reference:
        fp16_reference(args.workload, args.steps, args.warmup)
        return
    if args.mfma_probe:
        mfma_ceiling(args.workload, args.steps, args.warmup)
        return

    if args.paper_sweep:
        for k in synth.PAPER_SWEEP_K:
            out = bench_workload(args, f"paper_k{k}", cpu=False)
            print(json.dumps(out), flush=True)
            torch.cuda.empty_cache()
        return
    print(json.dumps(bench_workload(args, args.workload, cpu=not args.no_cpu_baseline)),
          flush=True)


def bench_workload(args, name: str, cpu: bool) -> dict:
    """Time one workload; the JSON record of the benchmark contract."""
    w = synth.WORKLOADS[name]
    if args.batch is not None and args.batch != w.batch:
        w = dataclasses.replace(w, batch=args.batch)
    host_inputs = synth.workload_inputs(w)
    dev_inputs = tuple(t.to("cuda") for t in host_inputs)
    policy = None
    if (args.flow, args.ec, args.tile) != (pkg.FLOW_AUTO, 1, pkg.TILE_AUTO):
        policy = pkg.Policy(args.flow, args.ec, args.tile)
    givens_mode = GIVENS_MODES[args.givens_mode]
    hh_mode = pkg.HOUSEHOLDER_LDS if args.householder_mode == "lds" else pkg.HOUSEHOLDER_RULE
    call, C = make_call(w, dev_inputs, policy, givens_mode, hh_mode)

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    launches = args.steps  # host calls in the timed region
    if args.graph:
        # the K steps captured in one graph on a side stream (default
        # priority) and replayed once: one graph launch per K steps instead
        # of K kernel launches (a graph launch costs more than a kernel
        # launch, so a graph of one step would be slower).  The library
        # launches on the capturing stream and allocates nothing, so the
        # graph holds the steps' kernels only.
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            with torch.cuda.graph(graph, stream=side):
                for _ in range(args.steps):
                    call()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        call = graph.replay
        launches = 1
        call()  # one untimed replay
        torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    # one event before the first call and one after every call (a marker on
    # the stream, no work): the first and last bound the timed region, the
    # ones between give the spread of single launches
    spread = not (args.graph or args.no_launch_spread)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(launches + 1 if spread else 2)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record(stream)
    if spread:
        for i in range(launches):
            call()
            evs[i + 1].record(stream)
    else:
        for _ in range(launches):
            call()
        evs[1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_events = evs[0].elapsed_time(evs[-1])
    ms_step = ms_events / args.steps
    per_launch = None
    if spread:
        d = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(launches))
        h = len(d) // 2
        median = d[h] if len(d) % 2 else 0.5 * (d[h - 1] + d[h])
        per_launch = {"median_ms": median, "min_ms": d[0], "max_ms": d[-1],
                      "value_at_median": (w.flops / (median * 1e-3)
                                          / (1e9 if w.kind == "scan" else 1e12))}

    flops = w.flops
    tflops = flops / (ms_step * 1e-3) / 1e12
    metric, value, unit = METRIC, tflops, "TFLOP/s"
    if w.kind == "scan":
        # one addition per element; the matrix form's MFMA work (12 MFMAs
        # of 32x32x16 per 2048 elements) is far below the HBM floor
        metric, value, unit = SCAN_METRIC, flops / (ms_step * 1e-3) / 1e9, "Gelem/s"
    # dominant (and only) kernel: one launch per step.  The bound is the
    # roof with the longer floor: HBM bytes at 8 TB/s or fp16 MFMA flops (3
    # per emulated flop) at the dense peak.
    bytes_alg = w.algorithmic_bytes
    t_hbm = bytes_alg / (PEAK_HBM_GBS * 1e9)
    t_mfma = 3 * flops / (PEAK_FP16_MFMA_TFLOPS * 1e12)
    if t_mfma > t_hbm and w.kind != "scan":
        roof = {"bound": "mfma", "achieved": 3 * flops / (ms_step * 1e-3) / 1e12,
                "peak": PEAK_FP16_MFMA_TFLOPS, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": bytes_alg / (ms_step * 1e-3) / 1e9,
                "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    resolved, kernel = None, ("householder64_lds_kernel" if hh_mode == pkg.HOUSEHOLDER_LDS
                              else "householder64_kernel")
    if w.kind == "givens":
        kernel = "givens64_lds_kernel" if givens_mode == pkg.GIVENS_LDS else "givens64_kernel"
    elif w.kind == "gemm_acc":
        kernel = "gemm_acc_kernel"
    elif w.kind == "scan":
        kernel = "scan_kernel"
    elif w.kind == "gemm":
        A, B = dev_inputs
        resolved, kernel = pkg.sgemm_emu_resolve_policy(A, B, C, policy=policy)
    roof["kernel"] = kernel
    tkey = w.name
    if w.kind == "givens" and args.givens_mode != "auto":
        tkey += ":" + args.givens_mode
    if w.kind == "householder" and args.householder_mode != "rule":
        tkey += ":" + args.householder_mode
    if w.batch != synth.WORKLOADS[name].batch:
        tkey += f":batch{w.batch}"
    roof["traffic"] = measured_traffic(tkey, roof["kernel"])

    out = {
        "metric": metric,
        "value": value,
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp16x3-mfma-fp32acc",
        "data": "synthetic",
        "config": {"workload": w.name, "kind": w.kind, "batch": w.batch, "m": w.m, "n": w.n,
                   "k": w.k, "dist": w.dist, "seed": w.seed,
                   "inputs_sha256": inputs_sha256(host_inputs),
                   "graph": bool(args.graph),
                   "policy": None if resolved is None else
                   {"flow": resolved.flow, "ec": resolved.ec, "tile": resolved.tile,
                    "requested": "auto" if policy is None else "explicit"},
                   **({"givens": {"plane": list(w.plane), "mode": args.givens_mode}}
                      if w.kind == "givens" else {}),
                   **({"householder_mode": args.householder_mode}
                      if w.kind == "householder" else {})},
        "frac_fp32_vector_peak": tflops / PEAK_FP32_VECTOR_TFLOPS,
        "frac_fp16_mfma_over_3": tflops / (PEAK_FP16_MFMA_TFLOPS / 3),
        "hbm_GBps_algorithmic": bytes_alg / (ms_step * 1e-3) / 1e9,
        "wall_s_timed": wall,
        "per_launch": per_launch,
        "roofline": roof,
        "cpu_baseline": None,
    }
    if w.kind == "gemm" and w.name == "gemm_8192" and args.batch is None:
        # context, measured after the timed region on the same device: the
        # vendor's fp16 GEMM on this shape (the clock the chip holds under
        # matrix load keeps even it far below the nominal peak)
        ref = fp16_reference(w.name, 10, 3, dtypes=("fp16",), quiet=True)[0]
        out["context_fp16_gemm"] = {
            "what": "torch.mm fp16 on the same shape, same device, after the timed region",
            "TFLOPs": ref["TFLOPs"], "frac_of_dense_peak": ref["frac_of_dense_peak"],
            "emulated_rate_over_a_third_of_it": tflops / (ref["TFLOPs"] / 3)}
        # and the same products with their operands held in registers
        cei = mfma_ceiling(w.name, 10, 3, quiet=True)
        out["context_mfma_ceiling"] = {
            "what": "the same three products alone (operands in registers, no loads, split or "
                    "LDS traffic; sgemm_emu_mfma_probe), same device, after the timed region",
            "TFLOPs": cei["TFLOPs"], "frac_of_dense_peak": cei["frac_of_dense_peak"],
            "emulated_rate_over_it": tflops / cei["TFLOPs"]}
    if cpu:
        cb, acc = cpu_baseline(w, host_inputs, C, args.cpu_seconds)
        out["cpu_baseline"] = cb
        out["accuracy"] = acc
    return out




if __name__ == "__main__":
    main()
