#!/usr/bin/env python3
"""Throughput of libhadacore's batched Walsh-Hadamard transform on one MI355X.

One step = one call of the transform over one batch of synthetic input that is
already resident in HBM.  Steps cycle through a rotating set of buffers of at
least 1 GiB so that no call finds its data in the 256 MiB Infinity Cache.

The default run measures every named workload and the size sweep:
  * the four named workloads: fp16 1024x256 out of place; bf16 1,048,576x128 in
    place with 0.1% outliers (the attention head_dim rotation, the headline);
    fp16 16384x4096 out of place with 16 outlier columns; bf16 4096x32768 in
    place;
  * the sweep n = 2^7 .. 2^15 at 2^28 elements per call, fp16 and bf16, in place
    and out of place (36 points; each input serves both modes).
Each point warms the GPU up for a fixed time, then times `--steps` back-to-back
calls in `--regions` separately synchronized regions (the headline's first
region is the reported step time), and also times two device copies of the same
bytes: the library's 16-byte copy kernel and the runtime's hipMemcpyAsync.  The CPU-baseline leg then runs the fp64 oracle over every row of the
named workloads and over sampled rows of the sweep points, compares it with one
fresh-copy call of the transform per point, and times the oracle on the
headline workload on the host cores.

Prints ONE JSON line; per-point results are in config.points.
``--workload NAME`` measures one workload only (used for profiling).
``--sweep FILE`` additionally writes one JSON line per extended point
(n = 2^0..2^20, FP8 and INT8 outputs) to FILE.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time
from pathlib import Path

ROOT = Path(__file__).resolve().parent
if str(ROOT) not in sys.path:
    sys.path.insert(0, str(ROOT))

METRIC = "FWHT elements/s and achieved HBM GB/s (% of peak) per n, fp16/bf16"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
ROTATING_BYTES = 1 << 30       # rotating buffer set per workload (>> 256 MiB MALL)
SOURCE = ROOT / "paper_2412_08832_amd" / "csrc" / "hadacore.hip"
PROFILES = ROOT / "profiles"
HEADLINE = "bf16_1048576x128_inplace"
NAMED = (HEADLINE, "fp16_1024x256", "fp16_16384x4096", "bf16_4096x32768_inplace")
SWEEP_LOG2 = range(7, 16)
SWEEP_SAMPLE_ELEMS = 1 << 22   # oracle-checked elements per sweep point (whole rows)


def parse_args(argv=None):
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50, help="timed calls per region")
    p.add_argument("--warmup", type=int, default=20,
                   help="untimed calls before each point's timing (at least)")
    p.add_argument("--warm-seconds", type=float, default=0.05,
                   help="keep warming up until this much time has passed (the GPU needs "
                        "~10 ms of sustained load to reach its steady clock)")
    p.add_argument("--regions", type=int, default=5,
                   help="timed regions per point (median and min reported)")
    p.add_argument("--workload", default=None,
                   help="measure one workload only: a named workload or "
                        "sweep:<dtype>:<log2 n>:<in|out>")
    p.add_argument("--sweep", metavar="FILE", help="also time the extended points, one JSON line each")
    p.add_argument("--fp8", action="store_true",
                   help="with --workload: the fused transform + e4m3 quantization")
    p.add_argument("--int8", action="store_true",
                   help="with --workload: the fused transform + int8 quantization")
    p.add_argument("--cpu-seconds", type=float, default=10.0,
                   help="target duration of the oracle timing on the headline workload")
    p.add_argument("--no-cpu-baseline", action="store_true",
                   help="skip the CPU leg (oracle timing and the per-point oracle checks)")
    return p.parse_args(argv)


def workload_by_name(name: str):
    from paper_2412_08832_amd import workloads as W
    if name in W.WORKLOADS:
        return W.WORKLOADS[name]
    m = re.fullmatch(r"sweep:(fp16|bf16):(\d+):(in|out)", name)
    if not m:
        raise SystemExit(f"unknown workload {name!r}")
    return W.sweep_point(int(m.group(2)), m.group(1), m.group(3) == "in")


def target_fraction(w) -> float | None:
    """Throughput target as a fraction of the HBM peak: 70% for n <= 4096 and 55%
    at n = 32768; none for n = 8192/16384, and none for the 1 MiB fp16 1024x256
    call, which is launch-bound and judged on parity (its size's target is read
    off the sweep's n = 256 points)."""
    if w.name == "fp16_1024x256":
        return None
    if w.n <= 4096:
        return 0.70
    if w.n == 32768:
        return 0.55
    return None


def source_digest() -> str:
    return hashlib.sha256(SOURCE.read_bytes()).hexdigest()


def measured_traffic(workload: str, digest: str):
    """HBM bytes per launch from a committed rocprofv3 PMC summary, or None.

    A summary counts only while the kernel source it was taken on is unchanged.
    """
    for path in sorted(PROFILES.glob("*.txt")):
        text = path.read_text()
        fields = dict(re.findall(r"^([a-z_0-9]+):\s*(\S+)\s*$", text, flags=re.M))
        if fields.get("workload") == workload and fields.get("source_sha256") == digest:
            try:
                return int(float(fields["traffic_bytes_per_launch"]))
            except (KeyError, ValueError):
                return None
    return None


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


class Device:
    def __init__(self):
        import torch
        from paper_2412_08832_amd import hadacore
        if not torch.cuda.is_available():
            raise SystemExit("bench.py needs a ROCm GPU")
        self.torch = torch
        self.H = hadacore
        hadacore.library()  # raises if the HIP library is missing: there is no fallback
        self.dev = torch.device("cuda:0")
        torch.cuda.set_device(self.dev)
        self.stream = torch.cuda.current_stream(self.dev)

    def upload(self, bits, dtype: str):
        import numpy as np
        torch = self.torch
        t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(self.dev)
        return t.view(torch.float16 if dtype == "fp16" else torch.bfloat16)

    def download(self, t):
        import numpy as np
        return t.view(self.torch.int16).cpu().numpy().view(np.uint16)

    def warm(self, calls, warmup: int, min_warm_s: float) -> None:
        """At least `warmup` calls, and more until `min_warm_s` seconds of them have run."""
        torch = self.torch
        t0 = time.perf_counter()
        i = 0
        while i < warmup or (min_warm_s > 0 and time.perf_counter() - t0 < min_warm_s):
            calls[i % len(calls)]()
            i += 1
            if i % 50 == 0:
                torch.cuda.synchronize(self.dev)
        torch.cuda.synchronize(self.dev)

    def region(self, calls, steps: int, first: int = 0) -> float:
        """Seconds for exactly `steps` back-to-back calls (cycling through `calls`),
        bracketed by device synchronizations, with HIP events recorded on the stream
        the kernels are launched on."""
        torch = self.torch
        torch.cuda.synchronize(self.dev)
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        start.record(self.stream)
        for i in range(steps):
            calls[(first + i) % len(calls)]()
        end.record(self.stream)
        end.synchronize()
        torch.cuda.synchronize(self.dev)
        return start.elapsed_time(end) / 1e3


def _median(xs):
    s = sorted(xs)
    k = len(s)
    return s[k // 2] if k % 2 else 0.5 * (s[k // 2 - 1] + s[k // 2])


def time_point(d: Device, w, pristine, args, quant: str | None = None) -> tuple[dict, object]:
    """Time one workload on device input `pristine` (left unchanged), then run one
    fresh-copy call.  Returns (record, fresh output on the host: 16-bit bits, or
    (codes, scales) for quant)."""
    H, torch = d.H, d.torch
    code = H.FP16 if w.dtype == "fp16" else H.BF16
    nbytes = w.m * w.n * 2
    per_set = nbytes + (w.m * w.n + 4 * w.m if quant else (0 if w.inplace else nbytes))
    nbuf = max(2, math.ceil(ROTATING_BYTES / per_set))
    ins = [pristine.clone() for _ in range(nbuf)]
    s = d.stream.cuda_stream
    ws = None
    if quant:
        entry = {"fp8": H.hadamard_transform_fp8, "int8": H.hadamard_transform_int8}[quant]
        codes = [torch.empty((w.m, w.n), dtype=torch.uint8, device=d.dev) for _ in range(nbuf)]
        scales = [torch.empty((w.m,), dtype=torch.float32, device=d.dev) for _ in range(nbuf)]

        def call(x, i):
            entry(x.data_ptr(), w.n, codes[i].data_ptr(), w.n, scales[i].data_ptr(), w.m, w.n,
                  code, w.scale, s)
        alg_bytes = w.m * w.n * 3 + 4 * w.m          # 16-bit read, 1-byte code write, row scales
        outs = codes
    elif w.n > 1 << 16:
        # two passes through an fp32 workspace (shared: the calls run in stream order)
        outs = ins if w.inplace else [torch.empty_like(pristine) for _ in range(nbuf)]
        need = H.hadamard_transform_workspace_size(w.m, w.n)
        ws = torch.empty(need, dtype=torch.uint8, device=d.dev)

        def call(x, i):
            y = x if w.inplace else outs[i]
            H.hadamard_transform_ws(x.data_ptr(), w.n, y.data_ptr(), w.n, w.m, w.n, code, w.scale,
                                    ws.data_ptr(), need, s)
        alg_bytes = 2 * nbytes                      # one read + one write of every element
    else:
        outs = ins if w.inplace else [torch.empty_like(pristine) for _ in range(nbuf)]

        def call(x, i):
            y = x if w.inplace else outs[i]
            H.hadamard_transform(x.data_ptr(), y.data_ptr(), w.m, w.n, code, w.scale, s)
        alg_bytes = 2 * nbytes                      # one read + one write of every element
    calls = [(lambda i=i: call(ins[i], i)) for i in range(nbuf)]
    d.warm(calls, args.warmup, args.warm_seconds)
    secs = [d.region(calls, args.steps, first=r * args.steps) for r in range(args.regions)]
    per_call = [x / args.steps for x in secs]

    # device copy of the same element bytes: the achievable-bandwidth reference
    dsts = [torch.empty_like(pristine) for _ in range(nbuf)] if (w.inplace or quant) else outs
    copies = [
        (lambda i=i: H.hadacore_stream_copy(ins[i].data_ptr(), dsts[i].data_ptr(), nbytes, s))
        for i in range(nbuf)
    ]
    d.warm(copies, 0, 0.02)
    csec = _median([d.region(copies, args.steps) for _ in range(3)]) / args.steps
    copy_gbs = 2 * nbytes / csec / 1e9
    # the runtime's device-to-device copy of the same bytes (torch's copy_ between
    # contiguous same-dtype tensors on one device is a hipMemcpyAsync): the memcpy
    # bound the paper compares against (App. B)
    memcpys = [(lambda i=i: dsts[i].copy_(ins[i])) for i in range(nbuf)]
    d.warm(memcpys, 0, 0.02)
    msec = _median([d.region(memcpys, args.steps) for _ in range(3)]) / args.steps
    memcpy_gbs = 2 * nbytes / msec / 1e9
    del dsts, copies, memcpys, calls, outs, ins

    # one call on a fresh copy of the input, for the oracle check
    x = pristine.clone()
    if quant:
        c = torch.empty((w.m, w.n), dtype=torch.uint8, device=d.dev)
        sc = torch.empty((w.m,), dtype=torch.float32, device=d.dev)
        entry(x.data_ptr(), w.n, c.data_ptr(), w.n, sc.data_ptr(), w.m, w.n, code, w.scale, s)
        torch.cuda.synchronize(d.dev)
        fresh = (c.cpu().numpy(), sc.cpu().numpy())
        del c, sc, codes, scales
    else:
        y = x if w.inplace else torch.empty_like(pristine)
        if ws is not None:
            H.hadamard_transform_ws(x.data_ptr(), w.n, y.data_ptr(), w.n, w.m, w.n, code, w.scale,
                                    ws.data_ptr(), ws.numel(), s)
        else:
            H.hadamard_transform(x.data_ptr(), y.data_ptr(), w.m, w.n, code, w.scale, s)
        torch.cuda.synchronize(d.dev)
        fresh = d.download(y)
        del y
    del x, ws

    med = _median(per_call)
    gbs = alg_bytes / med / 1e9
    rec = {
        "workload": w.name + (f"_{quant}" if quant else ""), "dtype": w.dtype, "m": w.m,
        "n": w.n, "inplace": w.inplace and not quant, "output": quant or w.dtype,
        "steps_per_region": args.steps, "regions": args.regions, "rotating_buffers": nbuf,
        "ms_per_call": med * 1e3, "ms_per_call_min": min(per_call) * 1e3,
        "ms_per_call_first_region": per_call[0] * 1e3,
        "elements_per_s": w.m * w.n / med, "gbs": gbs, "frac_hbm_peak": gbs / HBM_PEAK_GBS,
        "gbs_best_region": alg_bytes / min(per_call) / 1e9,
        "copy_gbs": copy_gbs, "frac_of_copy": gbs / copy_gbs,
        "memcpy_gbs": memcpy_gbs, "frac_of_memcpy": gbs / memcpy_gbs,
        "alg_bytes_per_call": alg_bytes,
    }
    if not quant:
        tgt = target_fraction(w)
        rec["target_frac"] = tgt
        rec["meets_target"] = None if tgt is None else rec["frac_hbm_peak"] >= tgt
    return rec, fresh


# ---- CPU leg: the oracle (test infrastructure), timed and used as the checker ----

def host_info() -> dict:
    try:
        visible = len(os.sched_getaffinity(0))
    except AttributeError:
        visible = os.cpu_count() or 1
    cpu = ""
    try:
        for line in Path("/proc/cpuinfo").read_text().splitlines():
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"cpus_visible": visible, "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
            "cpu_model": cpu}


def _checker():
    tests = str(ROOT / "tests")
    if tests not in sys.path:
        sys.path.insert(0, tests)
    import oracle
    from gpu_util import compare_with_oracle, oracle_threads
    return oracle.get(), compare_with_oracle, oracle_threads


def check_point(w, in_bits, out_bits, rows=None) -> dict:
    """Compare one fresh-copy GPU output with the oracle (all rows, or `rows`)."""
    orc, compare_with_oracle, threads = _checker()
    t0 = time.perf_counter()
    c = compare_with_oracle(orc, out_bits, in_bits, w.dtype, w.scale, w.n, rows=rows,
                            threads=threads())
    return {"rows_checked": int(w.m if rows is None else len(rows)), "elements_checked": c.count,
            "rel_l2": c.rel_l2, "max_ulp_floored": c.max_ulp_floored,
            "max_ulp_unfloored": c.max_ulp_unfloored, "above_4ulp_unfloored": c.n_above_4ulp_unfloored,
            "nonfinite_mismatch": c.nonfinite_mismatch, "ok": bool(c.ok),
            "check_s": round(time.perf_counter() - t0, 2)}


def sweep_rows(w):
    """Sampled rows of a sweep point: the first, the last and random ones, about
    SWEEP_SAMPLE_ELEMS elements in all."""
    import numpy as np
    k = max(64, SWEEP_SAMPLE_ELEMS // w.n)
    rng = np.random.default_rng(w.n + (0 if w.dtype == "fp16" else 1))
    return np.unique(np.r_[0, w.m - 1, rng.integers(0, w.m, k)])


def cpu_baseline(w, target_seconds: float, quant: str | None = None) -> dict:
    """The fp64 oracle on the host cores, timed on a bounded row sample of the workload
    (with quant, the oracle's fused transform + quantization, which runs on one thread)."""
    import numpy as np
    from paper_2412_08832_amd import workloads as W
    orc, _, threads = _checker()
    info = host_info()
    cores = 1 if quant else threads()

    def run(b):
        if quant == "fp8":
            orc.fwht_fp8(b, w.dtype, w.scale)
        elif quant == "int8":
            orc.fwht_int8(b, w.dtype, w.scale)
        else:
            orc.fwht(b, w.dtype, w.scale, nthreads=cores)

    probe_rows = max(1, min(w.m, (1 << 20) // w.n // (16 if quant else 1)))
    bits = W.generate(w, rows=probe_rows)
    t0 = time.perf_counter()
    run(bits)
    rate = probe_rows * w.n / max(time.perf_counter() - t0, 1e-6)
    rows = int(min(w.m, max(probe_rows, target_seconds * rate / w.n)))
    bits = W.generate(w, rows=rows) if rows != probe_rows else bits
    # repeat the pass when the whole sample is shorter than the target duration
    passes = 0
    t0 = time.perf_counter()
    while True:
        run(bits)
        passes += 1
        sec = time.perf_counter() - t0
        if sec >= target_seconds or passes >= 1000:
            break
    single = None
    if not quant and cores > 1:
        # the same oracle on one thread, over a sample sized for ~1/4 of the target
        rows1 = max(1, min(rows, int(rows * passes / cores / 4)))
        t1 = time.perf_counter()
        orc.fwht(np.ascontiguousarray(bits[:rows1]), w.dtype, w.scale, nthreads=1)
        single = rows1 * w.n / max(time.perf_counter() - t1, 1e-6)
    threads_note = (f"fp64 iterative FWHT + {quant} quantization in C on 1 thread (the oracle's "
                    "quantizing path is single-threaded)" if quant
                    else f"fp64 iterative FWHT in C on {cores} threads")
    out = {
        "value": passes * rows * w.n / sec, "unit": "elements/s", "cores": cores, "kind": "oracle",
        "sample": f"{passes} pass(es) over the first {rows} of {w.m} rows of {w.name} "
                  f"({rows * w.n} elements each), {sec:.1f} s, {threads_note}; host: "
                  f"{info['cpu_model']}, {info['cpus_visible']} CPUs visible, "
                  f"OMP_NUM_THREADS={info['omp_num_threads']}",
        **info,
    }
    if single is not None:
        out["value_1_thread"] = single
    return out


# The paper's own performance claims (abstract; Sec. 5): speedups of its CUDA kernel
# over the Dao AI Lab fast-hadamard-transform kernel, fp16, n = 2^7 ... 2^15, on
# other hardware.  Context only: they are ratios between two kernels on A100 and
# H100, not a rate on this GPU, so vs_baseline stays null.
PAPER_CONTEXT = {
    "kind": "speedup over the paper's baseline FWHT kernel, other hardware, context only",
    "a100_pcie": {"typical": "1.1-1.4x", "peak": "3.5x"},
    "h100_pcie": {"typical": "1.0-1.3x", "peak": "3.6x"},
    "source": "abstract and Sec. 5",
}


def headline_line(args, w, rec, quant=None) -> dict:
    digest = source_digest()
    first = rec["ms_per_call_first_region"] / 1e3
    gbs = rec["alg_bytes_per_call"] / first / 1e9
    return {
        "metric": METRIC,
        "value": w.m * w.n / first,
        "unit": "elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": first * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": rec["workload"], "m": w.m, "n": w.n, "io_dtype": w.dtype,
            "inplace": rec["inplace"],
            "output": f"{'e4m3' if quant == 'fp8' else 'int8'} codes + fp32 row scales" if quant
            else w.dtype,
            "scale": w.scale, "rotating_buffers": rec["rotating_buffers"],
            "achieved_gbs": gbs, "frac_hbm_peak": gbs / HBM_PEAK_GBS,
            "copy_gbs": rec["copy_gbs"], "frac_of_copy": gbs / rec["copy_gbs"],
            "memcpy_gbs": rec["memcpy_gbs"], "frac_of_memcpy": gbs / rec["memcpy_gbs"],
            "timing": f"value and ms_per_step from the first timed region ({args.steps} calls after "
                      f">= {args.warmup} calls and >= {args.warm_seconds} s of warm-up); "
                      f"points report the median of {args.regions} regions",
        },
        "roofline": {
            "bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": gbs / HBM_PEAK_GBS, "traffic": measured_traffic(rec["workload"], digest),
        },
        "paper_context": PAPER_CONTEXT,
        "source_sha256": digest,
    }


def run_single(args, d: Device) -> dict:
    from paper_2412_08832_amd import workloads as W
    quant = "fp8" if args.fp8 else ("int8" if args.int8 else None)
    w = workload_by_name(args.workload)
    bits = W.generate(w)
    pristine = d.upload(bits, w.dtype)
    rec, fresh = time_point(d, w, pristine, args, quant=quant)
    del pristine
    d.torch.cuda.empty_cache()
    line = headline_line(args, w, rec, quant)
    line["config"]["point"] = rec
    if not args.no_cpu_baseline:
        if not quant:
            rows = None if w.name in NAMED else sweep_rows(w)
            line["config"]["point"]["parity"] = check_point(w, bits, fresh, rows=rows)
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds, quant=quant)
    return line


def run_all(args, d: Device) -> dict:
    from paper_2412_08832_amd import workloads as W
    points = []
    head_rec = None
    check = not args.no_cpu_baseline

    def record(w, bits, rec, fresh, rows):
        if check:
            rec["parity"] = check_point(w, bits, fresh, rows=rows)
        points.append(rec)
        par = rec.get("parity")
        log(f"[bench] {rec['workload']}: {rec['gbs']:.0f} GB/s ({100 * rec['frac_hbm_peak']:.1f}% of "
            f"peak, {100 * rec['frac_of_copy']:.1f}% of copy)"
            + (f"; oracle check {'ok' if par['ok'] else 'FAILED'} rel_l2={par['rel_l2']:.2e} "
               f"max_ulp_floored={par['max_ulp_floored']:.2f}" if par else ""))

    for name in NAMED:
        w = W.WORKLOADS[name]
        bits = W.generate(w)
        pristine = d.upload(bits, w.dtype)
        rec, fresh = time_point(d, w, pristine, args)
        del pristine
        d.torch.cuda.empty_cache()
        if name == HEADLINE:
            head_rec = rec
        record(w, bits, rec, fresh, None)
        del bits, fresh
    for dt in ("fp16", "bf16"):
        for k in SWEEP_LOG2:
            w_in = W.sweep_point(k, dt, True)
            w_out = W.sweep_point(k, dt, False)
            bits = W.generate(w_in)          # one input for both modes
            pristine = d.upload(bits, dt)
            rows = sweep_rows(w_in)
            for w in (w_in, w_out):
                rec, fresh = time_point(d, w, pristine, args)
                record(w, bits, rec, fresh, rows)
                del fresh
            del pristine, bits
            d.torch.cuda.empty_cache()
    w = W.WORKLOADS[HEADLINE]
    line = headline_line(args, w, head_rec)
    fr = [p["frac_hbm_peak"] for p in points]
    line["config"]["points"] = points
    line["config"]["summary"] = {
        "points": len(points),
        "parity_checked": sum(1 for p in points if "parity" in p),
        "parity_ok": sum(1 for p in points if p.get("parity", {}).get("ok")),
        "targets_checked": sum(1 for p in points if p.get("meets_target") is not None),
        "targets_met": sum(1 for p in points if p.get("meets_target")),
        "frac_hbm_peak_min": min(fr), "frac_hbm_peak_max": max(fr),
        "sweep_frac_n_le_4096_min": min(p["frac_hbm_peak"] for p in points
                                        if p["workload"].startswith("sweep") and p["n"] <= 4096),
        "sweep_frac_n_32768_min": min(p["frac_hbm_peak"] for p in points
                                      if p["workload"].startswith("sweep") and p["n"] == 32768),
    }
    if check:
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    return line


def run_extended(args, d: Device, path: str) -> None:
    """Extended points (outside the metric's configs): n = 2^0..2^6 and 2^16..2^20 (bf16),
    and the fused FP8/INT8 outputs at n = 2^0..2^16 and on the two outlier workloads."""
    from paper_2412_08832_amd import workloads as W
    pts = [W.sweep_point(k, "bf16", ip) for ip in (True, False) for k in range(0, 7)]
    pts += [W.sweep_point(16, dt, ip) for dt in ("fp16", "bf16") for ip in (True, False)]
    pts += [W.sweep_point(k, "bf16", True) for k in range(17, 21)]
    q_pts = [W.sweep_point(k, "bf16", False) for k in range(0, 17)]
    q_pts += [W.WORKLOADS[HEADLINE], W.WORKLOADS["fp16_16384x4096"]]
    jobs = [(p, None) for p in pts] + [(p, q) for q in ("fp8", "int8") for p in q_pts]
    with open(path, "w") as f:
        for p, q in jobs:
            pristine = d.upload(W.generate(p), p.dtype)
            rec, _ = time_point(d, p, pristine, args, quant=q)
            del pristine
            d.torch.cuda.empty_cache()
            f.write(json.dumps(rec) + "\n")
            f.flush()
            log(f"[extended] {rec['workload']}: {rec['gbs']:.0f} GB/s "
                f"({100 * rec['frac_hbm_peak']:.1f}% of peak, {100 * rec['frac_of_copy']:.1f}% of copy)")


def main(argv=None) -> int:
    t_start = time.perf_counter()
    args = parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); rows are "
              "independent, so N GPUs would each run this kernel on m/N rows.", file=sys.stderr)
        return 2
    if args.fp8 and args.int8:
        raise SystemExit("--fp8 and --int8 are exclusive")
    if (args.fp8 or args.int8) and args.workload is None:
        raise SystemExit("--fp8/--int8 need --workload")
    if args.steps < 1 or args.regions < 1:
        raise SystemExit("--steps and --regions must be >= 1")
    d = Device()
    line = run_single(args, d) if args.workload else run_all(args, d)
    if args.sweep:
        run_extended(args, d, args.sweep)
    line["bench_wall_s"] = round(time.perf_counter() - t_start, 1)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
