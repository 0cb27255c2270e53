"""The allocation-free entry point mdgemm_ex_noalloc, called through the C ABI.

Its output must equal mdgemm_ex's (the entry point it is a variant of) bit for
bit, on two calls in a row, the second with a smaller product (the scratch array
keeps the first call's contents, so anything read before it is written would
show up), and also for the int8 level products and under HIP graph capture.
Requests it cannot serve without allocating are refused on the host.
"""

import ctypes

import numpy as np
import pytest
import torch

from oracle import pipeline
from paper_2607_06881_amd import mdgemm as md
from paper_2607_06881_amd import workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _operands(L, m, k, n, seed):
    rng = np.random.default_rng(seed)
    A = workloads.make_operand(rng, L, m, k, "normal", row_exp=9)
    B = workloads.make_operand(rng, L, k, n, "normal", col_exp=9)
    return torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV), A, B


def _noalloc(A, B, C, **opts):
    L, m, k = A.shape
    n = B.shape[2]
    o = md.make_opts(**opts)
    return md.lib().mdgemm_ex_noalloc(m, n, k, L, A.data_ptr(), B.data_ptr(), C.data_ptr(), ctypes.byref(o))


@pytest.mark.parametrize("flags", [0, md.MDGEMM_INT8])
def test_noalloc_equals_mdgemm_ex_on_two_calls_second_smaller(flags):
    for L, m, k, n, seed in [(3, 300, 160, 270, 1), (2, 70, 45, 33, 2)]:
        print(f"[case] noalloc flags={flags} L={L} {m}x{k}x{n}", flush=True)
        assert md.mdgemm_workspace_bytes(m, n, k, L, flags=flags) <= md.MDGEMM_NOALLOC_MAX_BYTES
        Ag, Bg, A, B = _operands(L, m, k, n, seed)
        want = md.mdgemm_ex(Ag, Bg, flags=flags)
        C = torch.full((L, m, n), 7.0, dtype=torch.float64, device=DEV)
        assert _noalloc(Ag, Bg, C, flags=flags) == md.MDGEMM_OK
        torch.cuda.synchronize()
        assert torch.equal(C, want)
    # the smaller product is also the oracle's (digits, levels and rounding)
    w, S, T = md.mdgemm_plan(m, n, k, L, flags=flags)
    assert np.array_equal(C.cpu().numpy(), pipeline.full_reference(A, B, S, T, w)["C"])


def test_noalloc_refusals_and_capture():
    print("[case] noalloc refusals and graph capture", flush=True)
    Ag, Bg, _, _ = _operands(2, 64, 64, 64, 3)
    C = torch.empty((2, 64, 64), dtype=torch.float64, device=DEV)
    E = md.MDGEMM_EINVAL
    # no caller workspace, no timing events, no finiteness check
    ws = torch.empty(md.mdgemm_workspace_bytes(64, 64, 64, 2), dtype=torch.uint8, device=DEV)
    assert _noalloc(Ag, Bg, C, workspace=ws) == E
    assert _noalloc(Ag, Bg, C, flags=md.MDGEMM_TIME_STAGES) == E
    assert _noalloc(Ag, Bg, C, flags=md.MDGEMM_CHECK_FINITE) == E
    # a product whose workspace exceeds the scratch array: refused before any launch
    m, k, n = 2048, 64, 2048
    assert md.mdgemm_workspace_bytes(m, n, k, 2) > md.MDGEMM_NOALLOC_MAX_BYTES
    o = md.make_opts()
    assert md.lib().mdgemm_ex_noalloc(m, n, k, 2, Ag.data_ptr(), Bg.data_ptr(), C.data_ptr(),
                                      ctypes.byref(o)) == md.MDGEMM_EWORKSPACE
    # captured in a HIP graph: every replay (eager calls in between) equals mdgemm_ex
    want = md.mdgemm_ex(Ag, Bg)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        assert _noalloc(Ag, Bg, C, stream=s) == md.MDGEMM_OK  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        assert _noalloc(Ag, Bg, C) == md.MDGEMM_OK
    other = torch.empty_like(C)
    for r in range(3):
        C.fill_(5.0)
        assert _noalloc(Ag, Bg, other) == md.MDGEMM_OK  # eager use of the same scratch between replays
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(C, want), r
        assert torch.equal(other, want), r
