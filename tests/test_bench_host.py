"""Host logic of bench.py, checked on the CPU: the one-GPU rule, workload names,
the traffic figure read from the committed rocprofv3 summaries, and the
paper-context object of the JSON line."""
from __future__ import annotations

import re
import subprocess
import sys

import pytest

import bench
from paper_2412_08832_amd import workloads as W


def _profile_fields(path):
    return dict(re.findall(r"^([a-z_0-9]+):\s*(\S+)\s*$", path.read_text(), flags=re.M))


PROFILES = sorted(p for p in bench.PROFILES.glob("*.txt")
                  if "algorithmic_bytes_per_launch" in _profile_fields(p))
COUNTER_SUMMARIES = sorted(p for p in bench.PROFILES.glob("*.txt") if p not in PROFILES)


def test_more_than_one_gpu_exits_with_a_message():
    res = subprocess.run([sys.executable, str(bench.ROOT / "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout == ""


def test_workload_names():
    w = bench.workload_by_name("sweep:bf16:16:in")
    assert (w.n, w.m, w.dtype, w.inplace) == (65536, 4096, "bf16", True)
    w = bench.workload_by_name("sweep:fp16:7:out")
    assert (w.n, w.m, w.dtype, w.inplace) == (128, 1 << 21, "fp16", False)
    assert bench.workload_by_name("bf16_1048576x128_inplace") is W.WORKLOADS["bf16_1048576x128_inplace"]
    with pytest.raises(SystemExit):
        bench.workload_by_name("sweep:fp32:7:in")


def test_default_run_covers_every_configuration():
    """No flags: one GPU, every named workload (the headline first) and the
    n = 2^7..2^15 sweep in both dtypes and modes."""
    args = bench.parse_args([])
    assert args.workload is None and args.gpus == 1
    w = W.WORKLOADS[bench.HEADLINE]
    assert (w.m, w.n, w.dtype, w.inplace) == (1048576, 128, "bf16", True)
    assert bench.NAMED[0] == bench.HEADLINE
    assert set(bench.NAMED) == set(W.WORKLOADS)
    assert list(bench.SWEEP_LOG2) == list(range(7, 16))
    assert args.warm_seconds > 0 and args.regions >= 1


def test_targets():
    """70% of the HBM peak for n <= 4096, 55% at n = 32768, none stated for
    8192/16384 or for the launch-bound 1 MiB call."""
    assert bench.target_fraction(W.WORKLOADS["fp16_1024x256"]) is None
    assert bench.target_fraction(W.WORKLOADS["bf16_1048576x128_inplace"]) == 0.70
    assert bench.target_fraction(W.WORKLOADS["fp16_16384x4096"]) == 0.70
    assert bench.target_fraction(W.WORKLOADS["bf16_4096x32768_inplace"]) == 0.55
    for k in range(7, 16):
        t = bench.target_fraction(W.sweep_point(k, "fp16", True))
        assert t == (0.70 if k <= 12 else 0.55 if k == 15 else None)


def test_sweep_sample_rows():
    for k in (7, 12, 15):
        w = W.sweep_point(k, "bf16", True)
        rows = bench.sweep_rows(w)
        assert rows[0] == 0 and rows[-1] == w.m - 1
        assert (rows >= 0).all() and (rows < w.m).all() and (rows[1:] > rows[:-1]).all()
        assert len(rows) * w.n >= min(w.m * w.n, bench.SWEEP_SAMPLE_ELEMS) // 2


def test_check_point_flags_a_wrong_output(oracle):
    """The per-point oracle check of the CPU leg accepts the oracle's own rounded
    result and rejects one element moved by 8 ulp."""
    import numpy as np
    w = W.sweep_point(7, "fp16", True)
    bits = W.generate(w, rows=300)
    ref = oracle.fwht(bits, "fp16", w.scale)
    good = ref.astype(np.float16).view(np.uint16)
    small = W.Workload(w.name, w.dtype, 300, w.n, w.inplace, w.scale, w.description)
    assert bench.check_point(small, bits, good)["ok"]
    bad = good.copy()
    bad[17, 5] = np.uint16(int(bad[17, 5]) + 8)
    r = bench.check_point(small, bits, bad, rows=np.array([0, 17, 299]))
    assert not r["ok"] and r["rows_checked"] == 3 and r["max_ulp_floored"] > 4


@pytest.mark.parametrize("path", PROFILES, ids=[p.stem for p in PROFILES])
def test_profile_summary_is_consistent(path):
    """Each summary names its command, and its figures agree with each other:
    achieved GB/s = algorithmic bytes / average duration, and the counted HBM
    traffic is within 1% of the algorithmic bytes (no re-reads)."""
    f = _profile_fields(path)
    text = path.read_text()
    assert "rocprofv3" in text and "bench.py" in text
    assert re.fullmatch(r"[0-9a-f]{64}", f["source_sha256"])
    alg = float(f["algorithmic_bytes_per_launch"])
    avg = float(f["kernel_avg_ns_timed_calls"])
    assert float(f["achieved_gbs_timed_calls"]) == pytest.approx(alg / avg, rel=2e-3)
    if "traffic_bytes_per_launch" in f:
        # per-dispatch constants (code and argument fetches of every XCD) are a
        # visible fraction only of the 1 MiB call
        tol = 0.01 if alg >= 1 << 26 else 0.03
        assert float(f["traffic_bytes_per_launch"]) / alg == pytest.approx(1.0, abs=tol)


@pytest.mark.parametrize("path", [p for p in PROFILES if "traffic_bytes_per_launch" in
                                  _profile_fields(p)], ids=lambda p: p.stem)
def test_traffic_is_read_only_for_the_profiled_source(path):
    f = _profile_fields(path)
    got = bench.measured_traffic(f["workload"], f["source_sha256"])
    assert got == int(float(f["traffic_bytes_per_launch"]))
    assert bench.measured_traffic(f["workload"], "0" * 64) is None


@pytest.mark.parametrize("path", COUNTER_SUMMARIES, ids=[p.stem for p in COUNTER_SUMMARIES])
def test_counter_summary_names_its_command_and_source(path):
    """Counter-only summaries (no timing) name the rocprofv3 command, the source
    they were taken on and per-kernel shares between 0 and 1."""
    text = path.read_text()
    f = _profile_fields(path)
    assert "rocprofv3 --pmc" in text and "bench.py" in text
    assert re.fullmatch(r"[0-9a-f]{64}", f["source_sha256"])
    shares = [float(v) for k, v in re.findall(r"^([a-z_]+_share):\s*(\S+)$", text, flags=re.M)]
    assert shares and all(0.0 <= x <= 1.0 for x in shares)


def test_default_command_summary_agrees_with_the_bench_line():
    """The trace of the default bench command: the headline kernel's first timed
    region, averaged from the trace, agrees with the step time the same run
    printed (HIP events around that region) within 3%."""
    paths = [p for p in PROFILES if p.stem.endswith("_default_command")]
    assert len(paths) == 1
    f = _profile_fields(paths[0])
    assert "--steps 20 --warmup 5" in paths[0].read_text()
    trace_ms = float(f["kernel_avg_ns_first_region"]) / 1e6
    assert trace_ms == pytest.approx(float(f["bench_ms_per_step_same_run"]), rel=0.03)


def test_counter_summaries_cover_both_front_ends():
    text = (bench.PROFILES / "sq_counters_front_ends_bf16.txt").read_text()
    for L in (7, 11, 12, 13, 15):
        for front in ("valu", "mfma"):
            assert f"HADACORE_VARIANT={front}" in text and f"sweep:bf16:{L}:in" in text
    blocks = re.findall(r"front: (valu|mfma)\nkernel: \S+\ndispatches: \d+\nvalu_insts_per_512_elements: ([\d.]+)", text)
    assert len(blocks) == 10
    # the matrix-core front issues fewer VALU instructions at every size
    for i in range(0, 10, 2):
        assert blocks[i][0] == "valu" and blocks[i + 1][0] == "mfma"
        assert float(blocks[i + 1][1]) < float(blocks[i][1])


def test_every_summary_is_checked():
    assert len(PROFILES) + len(COUNTER_SUMMARIES) == len(list(bench.PROFILES.glob("*.txt")))
    assert PROFILES, "no kernel-trace summaries"


def test_paper_context_is_context_only():
    ctx = bench.PAPER_CONTEXT
    assert ctx["a100_pcie"] == {"typical": "1.1-1.4x", "peak": "3.5x"}
    assert ctx["h100_pcie"] == {"typical": "1.0-1.3x", "peak": "3.6x"}
    assert "context" in ctx["kind"]


def test_cpu_baseline_fields():
    """The oracle baseline on a small workload: the contract's fields, plus the
    one-thread rate when more than one core is used."""
    r = bench.cpu_baseline(W.WORKLOADS["fp16_1024x256"], 0.2)
    assert r["kind"] == "oracle" and r["unit"] == "elements/s"
    assert r["value"] > 0 and r["cores"] >= 1
    assert "pass(es) over the first" in r["sample"]
    assert r["cpus_visible"] >= 1 and "CPUs visible" in r["sample"]
    if r["cores"] > 1:
        assert r["value_1_thread"] > 0
    q = bench.cpu_baseline(W.WORKLOADS["fp16_1024x256"], 0.2, quant="fp8")
    assert q["cores"] == 1 and "value_1_thread" not in q
