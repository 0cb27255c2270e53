"""GPU parity of the fused small-product kernel (all five steps in one launch
per 16 x 16 tile of C).

Every case is checked three ways, bit for bit: against the staged kernels
(MDGEMM_STAGED, the same product through the exponent, split, level-GEMM and
accumulation kernels) and against the oracle's chain (digits on the shared
grids, int64 levels, exact sum, greedy rounding).  The shapes cover ragged
tiles, a single element, k not a multiple of 4, k longer than one LDS chunk
(up to 1024, four chunks),
one to four limbs, every cutoff form, the adaptive width, range balancing,
zero lines and subnormal products; that the fused path is the one that ran is
read from mdgemm_workspace_layout, which refuses products it takes.
"""

import numpy as np
import pytest
import torch

from oracle import exact, pipeline
from paper_2607_06881_amd import mdgemm as md
from paper_2607_06881_amd import workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _fused(m, n, k, L, **opts):
    try:
        md.mdgemm_workspace_layout(m, n, k, L, **opts)
    except md.MdgemmError as e:
        return e.status == md.MDGEMM_EINVAL
    return False


CASES = [
    (2, 64, 64, 64, {"cutoff": md.MDGEMM_CUTOFF_ALL}, 0),
    (2, 17, 300, 33, {}, 1),
    (1, 1, 1, 1, {}, 2),
    (3, 200, 37, 150, {"cutoff": md.MDGEMM_CUTOFF_ALL}, 3),
    (4, 45, 130, 60, {}, 4),
    (2, 256, 200, 256, {}, 5),
    (2, 100, 64, 90, {"slice_bits": md.MDGEMM_SLICE_BITS_AUTO}, 6),
    (2, 70, 48, 65, {"range_bits": 60}, 7),
    (4, 33, 20, 45, {"cutoff": md.MDGEMM_CUTOFF_ALL}, 8),
    (3, 31, 5, 47, {"cutoff": 4}, 9),
    (2, 16, 129, 16, {"slices": 9, "cutoff": 10}, 10),
    (2, 40, 6, 20, {"slice_bits": 24, "slices": 5}, 11),  # the widest digit FP32 holds
    # long k, where the time estimates pick the fused kernel over a k-split staged GEMM
    (3, 100, 400, 100, {}, 12),
    (4, 45, 300, 60, {}, 13),
    (2, 256, 800, 256, {}, 14),
    (2, 17, 512, 33, {}, 15),
    (1, 128, 1024, 128, {}, 16),
    (2, 128, 1024, 128, {"slice_bits": md.MDGEMM_SLICE_BITS_AUTO}, 17),
]


def test_small_product_refused_where_fp32_digits_are_not_exact():
    # 25-bit digits are not exact in the fused kernel's FP32 LDS: the staged path runs
    assert not _fused(129, 65, 1, 2, slice_bits=25, slices=5)
    assert _fused(129, 65, 1, 2, slice_bits=24, slices=5)


@pytest.mark.parametrize("L,m,k,n,opts,seed", CASES)
def test_small_product_fused_equals_staged_and_oracle(L, m, k, n, opts, seed):
    w, S, T = md.mdgemm_plan(m, n, k, L, **opts)
    print(f"[case] fused small product L={L} {m}x{k}x{n} {opts}: w={w} S={S} T={T}", flush=True)
    assert _fused(m, n, k, L, **opts)
    assert not _fused(m, n, k, L, flags=md.MDGEMM_STAGED, **opts)
    rng = np.random.default_rng(seed)
    A = workloads.make_operand(rng, L, m, k, "normal" if seed % 2 else "uniform", row_exp=12)
    B = workloads.make_operand(rng, L, k, n, "normal", col_exp=12)
    if m > 3:
        A[:, 3, :] = 0.0  # a zero row
    if n > 5:
        B[:, :, 5] = 0.0  # a zero column
    Ag, Bg = torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV)
    C = md.mdgemm_ex(Ag, Bg, **opts)
    Cs = md.mdgemm_ex(Ag, Bg, flags=md.MDGEMM_STAGED, **opts)
    torch.cuda.synchronize()
    assert torch.equal(C, Cs)
    ref = pipeline.full_reference(A, B, S, T, w)
    assert np.array_equal(C.cpu().numpy(), ref["C"])


def test_small_product_extremes_timing_and_capture():
    # extreme magnitudes (products far below 2^-1022 give +0.0 limbs), the
    # stage timing of the fused kernel, and graph capture without a workspace
    print("[case] fused small product: extremes, timing, capture", flush=True)
    rng = np.random.default_rng(40)
    L, m, k, n = 2, 50, 30, 40
    A = workloads.make_operand(rng, L, m, k, "normal")
    B = workloads.make_operand(rng, L, k, n, "normal")
    A[:, 10:15] *= 2.0**-600
    B[:, :, 20:24] *= 2.0**500
    A[:, 30:33] *= 2.0**-520
    B[:, :, 30:33] *= 2.0**-520
    Ag, Bg = torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV)
    assert _fused(m, n, k, L)
    C = md.mdgemm_ex(Ag, Bg, flags=md.MDGEMM_TIME_STAGES)
    ms = md.mdgemm_stage_times()
    torch.cuda.synchronize()
    assert ms[2] > 0.0 and ms[0] < ms[2] and ms[3] < ms[2]
    want = md.mdgemm_ex(Ag, Bg, flags=md.MDGEMM_STAGED).cpu().numpy()
    assert np.array_equal(C.cpu().numpy(), want)
    ref = pipeline.full_reference(A, B, 8, 7)
    assert np.array_equal(want, ref["C"])
    assert not np.signbit(want[want == 0.0]).any()
    # no workspace and no library buffer: capturable as it is
    out = torch.empty_like(C)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        md.mdgemm_ex(Ag, Bg, out)  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        md.mdgemm_ex(Ag, Bg, out)
    for r in range(3):
        out.fill_(3.0)
        md.mdgemm_ex(Ag, Bg)  # eager work in between
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy(), want), r


def test_small_product_workload_c0_tolerance():
    # the 64^3 workload with all slice pairs: every entry bit-exact and within
    # the stated tolerance of the exact product (sampled)
    w = workloads.WORKLOADS["c0"]
    A, B = workloads.make_workload(w)
    print("[case] fused small product: workload c0", flush=True)
    assert _fused(w.m, w.n, w.k, w.limbs, **w.options())
    C = md.mdgemm_ex(torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV), **w.options()).cpu().numpy()
    assert np.array_equal(C, pipeline.full_reference(A, B, w.slices, w.cutoff)["C"])
    for (i, j) in [(0, 0), (63, 63), (17, 40), (40, 17)]:
        want, mag = exact.exact_product(A, B, i, j)
        assert abs(exact.value(C[:, i, j]) - want) <= exact.tolerance(w.k, w.limbs, mag)
