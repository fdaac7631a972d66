"""The binding in a fresh process: loading the library before torch has been
imported must still bind it to torch's HIP runtime (one runtime per process),
so that torch's pointers and streams work with it."""
from __future__ import annotations

import subprocess
import sys
from pathlib import Path

import pytest

pytestmark = pytest.mark.gpu

ROOT = Path(__file__).resolve().parent.parent

SCRIPT = r"""
import sys
sys.path.insert(0, {root!r})
from paper_2412_08832_amd import hadacore as H
H.library()                      # before any explicit import of torch
import torch
x = torch.ones((4, 128), dtype=torch.bfloat16, device="cuda")
st = H.hadamard_transform(x.data_ptr(), x.data_ptr(), 4, 128, H.BF16, 1.0,
                          torch.cuda.current_stream().cuda_stream, check=False)
torch.cuda.synchronize()
row = x[0].float().cpu()
ok = st == 0 and row[0].item() == 128.0 and bool((row[1:] == 0).all())
maps = sorted({{l.split()[-1] for l in open("/proc/self/maps") if "libamdhip64" in l}})
print("status", st, "ok", ok, "runtimes", maps, flush=True)
sys.exit(0 if ok and len(maps) == 1 else 1)
"""


def test_library_loaded_before_torch_uses_torch_runtime():
    res = subprocess.run([sys.executable, "-c", SCRIPT.format(root=str(ROOT))],
                         capture_output=True, text=True, timeout=240)
    print(res.stdout, res.stderr[-2000:], flush=True)
    assert res.returncode == 0, res.stdout + res.stderr[-2000:]
