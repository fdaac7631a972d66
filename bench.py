#!/usr/bin/env python3
"""Throughput of libhadacore's batched Walsh-Hadamard transform on one MI355X.

One step = one call of the transform over one batch of synthetic input that is
already resident in HBM.  Steps cycle through a rotating set of buffers of at
least 1 GiB so that no call finds its data in the 256 MiB Infinity Cache.

Default workload: bf16, m = 8 x 32 x 4096 = 1,048,576 rows of n = 128 (the
attention head_dim rotation), in place, scale fp32(1/sqrt(128)).

Prints ONE JSON line.  ``--sweep FILE`` additionally times every named
workload and the n = 2^7..2^16 sweep (both dtypes, both modes) and writes one
JSON line per point to FILE.
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


def parse_args(argv=None):
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    # the GPU needs ~10 ms of sustained load to reach its steady clock; the
    # defaults warm up for ~25 ms and time ~17 ms of back-to-back calls
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=300)
    p.add_argument("--workload", default="bf16_1048576x128_inplace",
                   help="a named workload (workloads.WORKLOADS) or sweep:<dtype>:<log2 n>:<in|out>")
    p.add_argument("--sweep", metavar="FILE", help="also time every workload, one JSON line each")
    p.add_argument("--fp8", action="store_true",
                   help="time the fused transform + e4m3 quantization instead of the transform")
    p.add_argument("--int8", action="store_true",
                   help="time the fused transform + int8 quantization instead of the transform")
    p.add_argument("--cpu-seconds", type=float, default=10.0,
                   help="target duration of the CPU oracle baseline sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    return p.parse_args(argv)


def workload_by_name(name: str):
    from paper_2412_08832_amd import workloads as W
    if name in W.WORKLOADS:
        return W.WORKLOADS[name]
    m = re.fullmatch(r"sweep:(fp16|bf16):(\d+):(in|out)", name)
    if not m:
        raise SystemExit(f"unknown workload {name!r}")
    return W.sweep_point(int(m.group(2)), m.group(1), m.group(3) == "in")


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

    def time_calls(self, calls, steps: int, warmup: int, min_warm_s: float = 0.0) -> float:
        """Seconds for `steps` back-to-back calls (cycling through `calls`), HIP events
        recorded on the stream the kernels are launched on.  At least `warmup` untimed
        calls run first, and more until `min_warm_s` seconds of them have run."""
        torch = self.torch
        t0 = time.perf_counter()
        i = 0
        while i < warmup or (min_warm_s > 0 and time.perf_counter() - t0 < min_warm_s):
            calls[i % len(calls)]()
            i += 1
            if min_warm_s > 0 and i % 50 == 0:
                torch.cuda.synchronize(self.dev)
        torch.cuda.synchronize(self.dev)
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        start.record(self.stream)
        for i in range(steps):
            calls[i % len(calls)]()
        end.record(self.stream)
        end.synchronize()
        torch.cuda.synchronize(self.dev)
        return start.elapsed_time(end) / 1e3


def time_workload(d: Device, w, steps: int, warmup: int, min_warm_s: float = 0.0,
                  quant: str | None = None) -> dict:
    """Time one workload: the transform (16-bit out, in place or not) or, with quant
    "fp8" / "int8", the fused transform + per-row quantization (codes + scales out)."""
    from paper_2412_08832_amd import workloads as W
    H, torch = d.H, d.torch
    bits = W.generate(w)
    code = H.FP16 if w.dtype == "fp16" else H.BF16
    nbytes = w.m * w.n * 2
    per_set = nbytes + (w.m * w.n + 4 * w.m if quant else (0 if w.inplace else nbytes))
    nbuf = max(2, math.ceil(ROTATING_BYTES / per_set))
    first = d.upload(bits, w.dtype)
    del bits
    ins = [first] + [first.clone() for _ in range(nbuf - 1)]
    s = d.stream.cuda_stream
    if quant:
        entry = {"fp8": H.hadamard_transform_fp8, "int8": H.hadamard_transform_int8}[quant]
        codes = [torch.empty((w.m, w.n), dtype=torch.uint8, device=d.dev) for _ in range(nbuf)]
        scales = [torch.empty((w.m,), dtype=torch.float32, device=d.dev) for _ in range(nbuf)]
        calls = [
            (lambda i=i: entry(ins[i].data_ptr(), w.n, codes[i].data_ptr(), w.n,
                               scales[i].data_ptr(), w.m, w.n, code, w.scale, s))
            for i in range(nbuf)
        ]
        alg_bytes = w.m * w.n * 3 + 4 * w.m          # 16-bit read, 1-byte code write, row scales
        outs = codes
    elif w.n > 1 << 16:
        # two passes through an fp32 workspace (shared: the calls run in stream order)
        outs = ins if w.inplace else [torch.empty_like(first) for _ in range(nbuf)]
        need = H.hadamard_transform_workspace_size(w.m, w.n)
        ws = torch.empty(need, dtype=torch.uint8, device=d.dev)
        calls = [
            (lambda i=i: H.hadamard_transform_ws(ins[i].data_ptr(), w.n, outs[i].data_ptr(), w.n,
                                                 w.m, w.n, code, w.scale, ws.data_ptr(), need, s))
            for i in range(nbuf)
        ]
        alg_bytes = 2 * nbytes                      # one read + one write of every element
    else:
        outs = ins if w.inplace else [torch.empty_like(first) for _ in range(nbuf)]
        calls = [
            (lambda i=i: H.hadamard_transform(ins[i].data_ptr(), outs[i].data_ptr(), w.m, w.n, code,
                                              w.scale, s))
            for i in range(nbuf)
        ]
        alg_bytes = 2 * nbytes                      # one read + one write of every element
    sec = d.time_calls(calls, steps, warmup, min_warm_s)
    per_launch = sec / steps
    gbs = alg_bytes / per_launch / 1e9

    # device copy of the same element bytes: the achievable-bandwidth reference
    dsts = [torch.empty_like(first) for _ in range(nbuf)] if (w.inplace or quant) else outs
    copies = [
        (lambda i=i: H.hadacore_stream_copy(ins[i].data_ptr(), dsts[i].data_ptr(), nbytes, s))
        for i in range(nbuf)
    ]
    csec = d.time_calls(copies, steps, warmup, min_warm_s) / steps
    copy_gbs = 2 * nbytes / csec / 1e9
    # the runtime's device-to-device copy of the same bytes (torch's copy_ between
    # contiguous same-dtype tensors on one device is a hipMemcpyAsync)
    memcpys = [(lambda i=i: dsts[i].copy_(ins[i])) for i in range(nbuf)]
    msec = d.time_calls(memcpys, steps, warmup, min_warm_s) / steps
    memcpy_gbs = 2 * nbytes / msec / 1e9
    del ins, outs, dsts, first, calls
    torch.cuda.empty_cache()
    return {
        "workload": w.name + (f"_{quant}" if quant else ""), "dtype": w.dtype, "m": w.m,
        "n": w.n, "inplace": w.inplace and not quant, "output": quant or w.dtype,
        "steps": steps, "rotating_buffers": nbuf, "ms_per_step": per_launch * 1e3,
        "elements_per_s": w.m * w.n / per_launch, "gbs": gbs, "frac_hbm_peak": gbs / HBM_PEAK_GBS,
        "copy_gbs": copy_gbs, "frac_of_copy": gbs / copy_gbs, "memcpy_gbs": memcpy_gbs,
        "alg_bytes_per_launch": alg_bytes,
    }


# The paper's own performance claims (abstract; §5): speedups of its CUDA kernel
# over the Dao AI Lab fast-hadamard-transform kernel, fp16, n = 2^7 ... 2^15, on
# other hardware.  Context only: they are ratios between two kernels on A100 and
# H100, not a rate on this GPU, so vs_baseline stays null.
PAPER_CONTEXT = {
    "kind": "speedup over the paper's baseline FWHT kernel, other hardware, context only",
    "a100_pcie": {"typical": "1.1-1.4x", "peak": "3.5x"},
    "h100_pcie": {"typical": "1.0-1.3x", "peak": "3.6x"},
    "source": "abstract and Sec. 5",
}


def cpu_baseline(w, target_seconds: float, quant: str | None = None) -> dict:
    """The fp64 oracle on the host cores, timed on a bounded row sample of the workload
    (with quant, the oracle's fused transform + quantization, which runs on one thread)."""
    import numpy as np
    import oracle
    from paper_2412_08832_amd import workloads as W
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    cores = 1 if quant else max(1, min(cores, 16))
    orc = oracle.get()

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
    cpu = ""
    try:
        for line in Path("/proc/cpuinfo").read_text().splitlines():
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    out = {
        "value": passes * rows * w.n / sec, "unit": "elements/s", "cores": cores, "kind": "oracle",
        "sample": f"{passes} pass(es) over the first {rows} of {w.m} rows ({rows * w.n} "
                  f"elements each), {sec:.1f} s, "
                  + (f"fp64 iterative FWHT + {quant} quantization in C on 1 thread, " if quant
                     else f"fp64 iterative FWHT in C on {cores} threads, ") + cpu,
    }
    if single is not None:
        out["value_1_thread"] = single
    return out


def main(argv=None) -> int:
    args = parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); rows are "
              "independent, so N GPUs would each run this kernel on m/N rows.", file=sys.stderr)
        return 2
    if args.fp8 and args.int8:
        raise SystemExit("--fp8 and --int8 are exclusive")
    quant = "fp8" if args.fp8 else ("int8" if args.int8 else None)
    w = workload_by_name(args.workload)
    d = Device()
    r = time_workload(d, w, args.steps, args.warmup, quant=quant)
    digest = source_digest()
    traffic = measured_traffic(r["workload"], digest)
    line = {
        "metric": METRIC,
        "value": r["elements_per_s"],
        "unit": "elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": r["workload"], "m": w.m, "n": w.n, "io_dtype": w.dtype,
            "inplace": r["inplace"],
            "output": f"{'e4m3' if quant == 'fp8' else 'int8'} codes + fp32 row scales" if quant
            else w.dtype,
            "scale": w.scale, "rotating_buffers": r["rotating_buffers"],
            "achieved_gbs": r["gbs"], "frac_hbm_peak": r["frac_hbm_peak"],
            "copy_gbs": r["copy_gbs"], "frac_of_copy": r["frac_of_copy"],
            "memcpy_gbs": r["memcpy_gbs"],
        },
        "roofline": {
            "bound": "hbm", "achieved": r["gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": r["frac_hbm_peak"], "traffic": traffic,
        },
        "paper_context": PAPER_CONTEXT,
    }
    if args.sweep:
        from paper_2412_08832_amd import workloads as W
        points = [W.WORKLOADS[k] for k in ("fp16_1024x256", "bf16_1048576x128_inplace", "fp16_16384x4096", "bf16_4096x32768_inplace")]
        for inplace in (True, False):
            for dt in ("fp16", "bf16"):
                points += [W.sweep_point(k, dt, inplace) for k in range(7, 17)]
        # sizes below and above the one-pass range: bf16 (above: in place, two passes)
        points += [W.sweep_point(k, "bf16", ip) for ip in (True, False) for k in range(0, 7)]
        points += [W.sweep_point(k, "bf16", True) for k in range(17, 21)]
        q_points = [W.sweep_point(k, "bf16", False) for k in range(0, 17)]
        q_points += [W.WORKLOADS["bf16_1048576x128_inplace"], W.WORKLOADS["fp16_16384x4096"]]
        jobs = [(p, None) for p in points] + [(p, q) for q in ("fp8", "int8") for p in q_points]
        with open(args.sweep, "w") as f:
            for p, q in jobs:
                pr = time_workload(d, p, args.steps, args.warmup, min_warm_s=0.03, quant=q)
                f.write(json.dumps(pr) + "\n")
                f.flush()
                print(f"[sweep] {pr['workload']}: {pr['gbs']:.0f} GB/s ({100 * pr['frac_hbm_peak']:.1f}% "
                      f"of peak, {100 * pr['frac_of_copy']:.1f}% of copy)", file=sys.stderr,
                      flush=True)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds, quant=quant)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
