"""The Python binding in a fresh process that loads the library before any
torch import: the distillation loss, a forward and a backward call still run,
on one HIP runtime, and match the same calls made after torch was imported."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

SCRIPT = r"""
import sys
sys.path.insert(0, {root!r})
import paper_2606_27748_amd as F
if {lib_first}:
    F.load()
import numpy as np
import torch
import workloads as W
from tests.gpu_util import to_device, desc_of
F.load()
out = []
wl = W.Workload("order", 1, 2, 130, 64, 64, "nonstationary", True, "bf16", True, 5)
t = to_device(W.generate(wl))
d = desc_of(wl)
O, den = F.flex_linattn_fwd(d, t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"])
g = F.flex_linattn_bwd(d, t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"], O, den, t["dO"])
aw = W.AWD_WORKLOADS[W.AWD_HEADLINE].scaled(B=1, H=2, N=100)
xa = to_device(W.generate_awd(aw))
da = F.make_desc(aw.B, aw.H, aw.N, aw.d, aw.m, aw.variant, False, aw.io)
r = F.flex_awd_loss(da, xa["Q"], xa["K"], xa["W1"], xa["W2"], xa["tau"], grads=True)
torch.cuda.synchronize()
vals = [O.float(), den, g["dK"], g["dW1"], r["loss"], r["dW1"]]
print("SUMS", " ".join(repr(float(v.double().abs().sum())) for v in vals), flush=True)
"""


def _run(lib_first):
    code = SCRIPT.format(root=ROOT, lib_first=lib_first)
    p = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=240, cwd=ROOT)
    assert p.returncode == 0, p.stderr[-3000:]
    line = [l for l in p.stdout.splitlines() if l.startswith("SUMS")]
    assert line, p.stdout[-2000:]
    return [float(v) for v in line[0].split()[1:]]


def test_library_loaded_before_torch():
    """Regression: loaded before torch, the library once bound to a second
    HIP runtime and its launches on torch's streams failed.  Results must be
    bitwise those of the torch-first order (the computation is deterministic)."""
    a = _run(lib_first=True)
    b = _run(lib_first=False)
    assert a == b
