"""MDGEMM_LOG: one stderr line per product or QR call, naming the plan, the path
the call took and its status; nothing without the variable.

The CPU tests call entry points that refuse their arguments before any HIP call
(negative sizes, a workspace passed to the allocation-free entry); the GPU test
runs a fused small product, a staged product and a QR in a child process.
"""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CPU_CHILD = r"""
import ctypes, sys
sys.path.insert(0, ROOT)
from paper_2607_06881_amd import mdgemm as md
L = md.lib()
o = md.mdgemm_opts()
L.mdgemm_opts_init(ctypes.byref(o))
print("st", L.mdgemm_ex(-1, 4, 4, 2, None, None, None, ctypes.byref(o)), flush=True)
o.workspace = ctypes.c_void_p(4096)
o.workspace_bytes = 1 << 20
print("st", L.mdgemm_ex_noalloc(8, 8, 8, 2, None, None, None, ctypes.byref(o)), flush=True)
"""


def _run(child, level, timeout):
    env = dict(os.environ)
    env.pop("MDGEMM_LOG", None)
    if level is not None:
        env["MDGEMM_LOG"] = str(level)
    code = "ROOT = %r\n" % ROOT + child
    return subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=timeout)


def test_log_lines_for_refused_calls():
    p = _run(CPU_CHILD, 1, 120)
    assert p.returncode == 0, p.stderr
    lines = [ln for ln in p.stderr.splitlines() if ln.startswith("[mdgemm]")]
    assert len(lines) == 2, p.stderr
    assert "mdgemm_ex m=-1 n=4 k=4 limbs=2 unplanned" in lines[0] and "path=refused -> invalid argument" in lines[0]
    assert lines[1].startswith("[mdgemm] mdgemm_ex_noalloc m=8 n=8 k=8 limbs=2 w=13 S=8 T=7")
    assert "workspace=scratch array" in lines[1] and "-> invalid argument" in lines[1]


def test_no_log_without_the_variable():
    p = _run(CPU_CHILD, None, 120)
    assert p.returncode == 0, p.stderr
    assert "[mdgemm]" not in p.stderr
    assert p.stdout.split() == ["st", str(-1), "st", str(-1)]


GPU_CHILD = r"""
import sys
sys.path.insert(0, ROOT)
import numpy as np, torch
from paper_2607_06881_amd import mdgemm as md, workloads
dev = torch.device("cuda:0")
rng = np.random.default_rng(3)
A = torch.from_numpy(workloads.make_operand(rng, 2, 40, 30, "normal")).to(dev)
B = torch.from_numpy(workloads.make_operand(rng, 2, 30, 50, "normal")).to(dev)
md.mdgemm_ex(A, B)
md.mdgemm_ex(A, B, flags=md.MDGEMM_STAGED)
Q = torch.from_numpy(workloads.make_operand(rng, 2, 300, 40, "normal")).to(dev)
md.mdgemm_qr_dd(Q, nb=16)
torch.cuda.synchronize()
print("done", flush=True)
"""


@pytest.mark.gpu
def test_log_lines_name_the_path():
    print("[case] MDGEMM_LOG=1 and 2 in a child process", flush=True)
    p = _run(GPU_CHILD, 1, 240)
    assert p.returncode == 0 and "done" in p.stdout, p.stderr[-2000:]
    lines = [ln for ln in p.stderr.splitlines() if ln.startswith("[mdgemm]")]
    assert len(lines) == 3, lines
    assert "m=40 n=50 k=30 limbs=2 w=13 S=8 T=7" in lines[0] and "path=fused small product -> success" in lines[0]
    assert "flags=0x40" in lines[1] and "path=staged: pair levels -> success" in lines[1]
    assert lines[2].startswith("[mdgemm] mdgemm_qr_dd m=300 n=40 nb=16") and lines[2].endswith("-> success")
    # level 2 adds the QR's own products, before its line
    p2 = _run(GPU_CHILD, 2, 240)
    assert p2.returncode == 0, p2.stderr[-2000:]
    lines2 = [ln for ln in p2.stderr.splitlines() if ln.startswith("[mdgemm]")]
    assert len(lines2) > 3 and lines2[-1].startswith("[mdgemm] mdgemm_qr_dd")
    assert all("-> success" in ln for ln in lines2)
