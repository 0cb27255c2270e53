"""GPU parity of the int8 level products (MDGEMM_INT8).

With digits of at most 7 bits every level of section 2 is formed exactly by
int8 matrix products with int32 sums, so the digits, the levels and the limbs
must equal the oracle's chain at the same width bit for bit, and equal the
FP64 path run with the same width, digit count and cutoff.  Sizes span ragged
shapes (n not a multiple of 16, k not a multiple of 16) and every limb count
the option supports.  The level products run on the hand-written int8 kernel;
the shape tests cover odd stage counts, ragged tiles and many levels.
"""

import ctypes
import random

import numpy as np
import pytest
import torch

from oracle import exact, pipeline
from paper_2607_06881_amd import mdgemm as md
from paper_2607_06881_amd import workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
I8 = md.MDGEMM_INT8


def _gpu(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _operands(L, m, k, n, seed, range_bits=0):
    rng = np.random.default_rng(seed)
    if range_bits:
        A = workloads.make_operand(rng, L, m, k, "normal")
        B = workloads.make_operand(rng, L, k, n, "normal")
        e = rng.integers(0, range_bits + 1, k)  # the wide-range recipe of workload c7
        A *= np.ldexp(1.0, -e)[None, None, :]
        B *= np.ldexp(1.0, e - range_bits)[None, :, None]
        return A, B
    base = "normal" if seed % 2 else "uniform"
    A = workloads.make_operand(rng, L, m, k, base, row_exp=15)
    B = workloads.make_operand(rng, L, k, n, base, col_exp=15)
    return A, B


def _fp64_same_digits(A, B, w, S, T, range_bits):
    D = -(-range_bits // w) if range_bits else 0
    return _host(md.mdgemm_ex(_gpu(A), _gpu(B), slice_bits=w, slices=S - D, cutoff=T, range_bits=range_bits))


@pytest.mark.parametrize("L,m,k,n,cutoff,range_bits,seed", [
    (2, 130, 64, 129, -1, 0, 40), (1, 65, 200, 17, -1, 0, 41), (3, 40, 100, 70, -1, 0, 42),
    (4, 33, 64, 45, -2, 0, 43), (8, 9, 40, 5, -1, 0, 44), (2, 1, 1, 1, -1, 0, 45),
    (2, 70, 48, 65, -1, 60, 46), (2, 17, 33, 300, 5, 0, 47), (4, 20, 17, 33, -1, 26, 48)])
def test_int8_end_to_end(L, m, k, n, cutoff, range_bits, seed):
    w, S, T = md.mdgemm_plan(m, n, k, L, flags=I8, cutoff=cutoff, range_bits=range_bits)
    assert (w, S, T) == exact.plan(L, k, int8=True, cutoff=cutoff, range_bits=range_bits)
    print(f"[case] int8 L={L} {m}x{k}x{n} w={w} S={S} T={T} range={range_bits}", flush=True)
    A, B = _operands(L, m, k, n, seed, range_bits)
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B), flags=I8, cutoff=cutoff, range_bits=range_bits))
    ref = pipeline.full_reference(A, B, S, T, w)
    assert np.array_equal(C, ref["C"])
    assert np.array_equal(C, _fp64_same_digits(A, B, w, S, T, range_bits))
    if cutoff == -1 and L <= 4:
        for i in range(0, m, max(1, m // 3)):
            for j in range(0, n, max(1, n // 3)):
                want, mag = exact.exact_product(A, B, i, j)
                assert abs(exact.value(C[:, i, j]) - want) <= exact.tolerance(k, L, mag), (i, j)


@pytest.mark.parametrize("L,m,k,n,bits,seed", [(2, 16, 8877, 8, 0, 50), (2, 40, 300, 33, 4, 51),
                                               (3, 9, 64, 70, 3, 52)])
def test_int8_narrow_digits(L, m, k, n, bits, seed):
    # k beyond the 7-bit budget (w = 6), and explicit narrow widths
    w, S, T = md.mdgemm_plan(m, n, k, L, flags=I8, slice_bits=bits)
    assert (w, S, T) == exact.plan(L, k, int8=True, slice_bits=bits)
    assert w < 7
    print(f"[case] int8 narrow L={L} {m}x{k}x{n} w={w} S={S} T={T}", flush=True)
    A, B = _operands(L, m, k, n, seed)
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B), flags=I8, slice_bits=bits))
    assert np.array_equal(C, pipeline.full_reference(A, B, S, T, w)["C"])


@pytest.mark.parametrize("L,m,k,n,seed", [(2, 1000, 2000, 777, 60), (4, 300, 1000, 260, 61), (3, 513, 1537, 129, 62)])
def test_int8_larger_products(L, m, k, n, seed):
    w, S, T = md.mdgemm_plan(m, n, k, L, flags=I8)
    print(f"[case] int8 larger L={L} {m}x{k}x{n} w={w} S={S} T={T}", flush=True)
    A, B = _operands(L, m, k, n, seed)
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B), flags=I8))
    assert np.array_equal(C, _fp64_same_digits(A, B, w, S, T, 0))
    pick = random.Random(seed)
    entries = [(pick.randrange(m), pick.randrange(n)) for _ in range(6)] + [(m - 1, n - 1), (0, 0)]
    ref = pipeline.reference_entries(A, B, S, T, entries, w)
    for (i, j), r in ref.items():
        assert list(C[:, i, j]) == r["limbs"], (i, j)


@pytest.mark.parametrize("L,m,k,n,seed", [(2, 300, 700, 257, 70), (3, 520, 1100, 300, 71), (2, 1000, 2000, 777, 60),
                                          (8, 64, 128, 8192, 72), (4, 257, 129, 513, 73), (1, 3, 5, 2, 74)])
def test_int8_shapes(L, m, k, n, seed):
    w, S, T = md.mdgemm_plan(m, n, k, L, flags=I8)
    print(f"[case] int8 L={L} {m}x{k}x{n} w={w} S={S} T={T}", flush=True)
    A, B = _operands(L, m, k, n, seed)
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B), flags=I8))
    assert np.array_equal(C, _fp64_same_digits(A, B, w, S, T, 0))
    pick = random.Random(seed)
    entries = [(pick.randrange(m), pick.randrange(n)) for _ in range(4)] + [(m - 1, n - 1)]
    ref = pipeline.reference_entries(A, B, S, T, entries, w)
    for (i, j), r in ref.items():
        assert list(C[:, i, j]) == r["limbs"], (i, j)


def test_int8_workspace_stream_and_stage_times():
    L, m, k, n = 2, 200, 300, 130
    print("[case] int8 workspace / stream / timing / finite check", flush=True)
    A, B = _operands(L, m, k, n, 70)
    Ag, Bg = _gpu(A), _gpu(B)
    want = _host(md.mdgemm_ex(Ag, Bg, flags=I8))
    need = md.mdgemm_workspace_bytes(m, n, k, L, flags=I8)
    ws = torch.full((need,), 0xAB, dtype=torch.uint8, device=DEV)  # stale contents must not matter
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        C = md.mdgemm_ex(Ag, Bg, flags=I8 | md.MDGEMM_TIME_STAGES, workspace=ws, stream=s)
    s.synchronize()
    assert np.array_equal(_host(C), want)
    times = md.mdgemm_stage_times()
    assert len(times) == 4 and all(t >= 0 for t in times)
    with pytest.raises(md.MdgemmError) as ei:  # one byte short
        md.mdgemm_ex(Ag, Bg, flags=I8, workspace=ws[: need - 1])
    assert ei.value.status == md.MDGEMM_EWORKSPACE
    A2 = A.copy()
    A2[1, 5, 7] = np.nan
    with pytest.raises(md.MdgemmError) as ei:
        md.mdgemm_ex(_gpu(A2), Bg, flags=I8 | md.MDGEMM_CHECK_FINITE)
    assert ei.value.status == md.MDGEMM_ENONFINITE
    # library workspace, twice (the cached algorithms are reused)
    for _ in range(2):
        C3 = torch.empty_like(C)
        o = md.make_opts(flags=I8)
        assert md.lib().mdgemm_ex(m, n, k, L, Ag.data_ptr(), Bg.data_ptr(), C3.data_ptr(), ctypes.byref(o)) == 0
        assert np.array_equal(_host(C3), want)


@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")  # the refused call leaves the graph empty
def test_int8_graph_capture():
    # With a caller workspace the int8 product (zeroing by kernel, no memsets,
    # no synchronization) is captured into a HIP graph, and every replay, with
    # eager work in between, equals the eager result; with the library's own
    # buffer it is refused under capture like the FP64 path.
    print("[case] int8 under graph capture", flush=True)
    L, m, k, n = 2, 64, 64, 64
    A, B = _operands(L, m, k, n, 80)
    Ag, Bg = _gpu(A), _gpu(B)
    want = _host(md.mdgemm_ex(Ag, Bg, flags=I8))
    assert np.array_equal(want, pipeline.full_reference(A, B, 15, 14, 7)["C"])
    C = torch.empty((L, m, n), dtype=torch.float64, device=DEV)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    g0 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g0, stream=s):
        o = md.make_opts(flags=I8, stream=s)
        st = md.lib().mdgemm_ex(m, n, k, L, Ag.data_ptr(), Bg.data_ptr(), C.data_ptr(), ctypes.byref(o))
    assert st == md.MDGEMM_EINVAL
    ws = torch.empty(md.mdgemm_workspace_bytes(m, n, k, L, flags=I8), dtype=torch.uint8, device=DEV)
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        md.mdgemm_ex(Ag, Bg, C, workspace=ws, flags=I8)  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        md.mdgemm_ex(Ag, Bg, C, workspace=ws, flags=I8)
    for r in range(4):
        C.fill_(7.0)
        md.mdgemm_ex(Ag, Bg, workspace=ws, flags=I8)  # eager work between replays
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(C.cpu().numpy(), want), r


def test_int8_zero_lines_k0_and_extreme_magnitudes():
    print("[case] int8 zero lines, k=0, extreme exponents, subnormal products", flush=True)
    A, B = _operands(2, 50, 30, 40, 90)
    A[:, 3, :] = 0.0
    B[:, :, 5] = 0.0
    A[:, 7, 4] = 0.0
    A[:, 10:15] *= 2.0**-600  # rows far below 1
    B[:, :, 20:24] *= 2.0**500  # columns far above 1
    A[:, 30:33] *= 2.0**-520  # with columns 30..32 of B below: products far below 2^-1022
    B[:, :, 30:33] *= 2.0**-520
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B), flags=I8))
    w, S, T = md.mdgemm_plan(50, 40, 30, 2, flags=I8)
    assert np.array_equal(C, pipeline.full_reference(A, B, S, T, w)["C"])
    assert np.array_equal(C, _fp64_same_digits(A, B, w, S, T, 0))
    assert (C[:, 3, :] == 0).all() and (C[:, :, 5] == 0).all()
    assert not np.signbit(C[:, 3, :]).any()
    Z = md.mdgemm_ex(torch.empty((2, 5, 0), dtype=torch.float64, device=DEV),
                     torch.empty((2, 0, 6), dtype=torch.float64, device=DEV),
                     C=torch.full((2, 5, 6), 3.0, dtype=torch.float64, device=DEV), flags=I8)
    z = _host(Z)
    assert (z == 0).all() and not np.signbit(z).any()


@pytest.mark.parametrize("m,k,n", [(1, 1, 1), (1, 700, 1), (300, 1, 17), (1, 64, 300), (17, 33, 1)])
def test_int8_degenerate_shapes(m, k, n):
    print(f"[case] int8 degenerate {m}x{k}x{n}", flush=True)
    A, B = _operands(2, m, k, n, m + 3 * k + 7 * n)
    w, S, T = md.mdgemm_plan(m, n, k, 2, flags=I8)
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B), flags=I8))
    assert np.array_equal(C, pipeline.full_reference(A, B, S, T, w)["C"])


@pytest.mark.parametrize("signs", ["same", "mixed"])
def test_int8_at_the_int32_limit(signs):
    # k = 8876 is the largest k with 15 pairs k 127^2 < 2^31 at w = 7 (checked
    # on the CPU).  Elements of value 1 - 2^-105 (the double-double (1, -2^-105))
    # have digits 63, 127, 127, ..., 127 on their grid, so the middle levels sum
    # products of nearly maximal digits over the full k: the int32 sums come
    # within a few percent of 2^31.
    m, k, n = 8, 8876, 8
    w, S, T = md.mdgemm_plan(m, n, k, 2, flags=I8)
    assert (w, S, T) == (7, 15, 14)
    print(f"[case] int8 at the int32 limit, {signs} signs", flush=True)
    A = np.zeros((2, m, k))
    B = np.zeros((2, k, n))
    A[0], A[1] = 1.0, -(2.0**-105)
    B[0], B[1] = 1.0, -(2.0**-105)
    if signs == "mixed":
        rng = np.random.default_rng(7)
        sa = rng.choice([-1.0, 1.0], size=(m, k))
        sb = rng.choice([-1.0, 1.0], size=(k, n))
        A *= sa[None]
        B *= sb[None]
    ref = pipeline.full_reference(A, B, S, T, w)
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B), flags=I8))
    assert np.array_equal(C, ref["C"])
    assert np.array_equal(C, _fp64_same_digits(A, B, w, S, T, 0))
    if signs == "same":
        # digits 63, 127, ..., 127; level 14 = k (2 63 127 + 13 127^2) = 0.93 2^31
        assert ref["DA"][:, 0, 0].tolist() == [63] + [127] * 14
        assert int(np.max(ref["G"])) == k * (2 * 63 * 127 + 13 * 127**2)
        assert int(np.max(ref["G"])) > 0.9 * 2**31


def _sweep_cases(count, seed):
    rng = random.Random(seed)
    cases = []
    for c in range(count):
        L = rng.choice([1, 2, 2, 3, 4, 8])
        m, k, n = rng.randint(1, 180), rng.randint(1, 300), rng.randint(1, 180)
        rb = rng.choice([0, 0, 0, 13, 40])
        if L == 8:
            rb = 0  # 60 digits already; range digits would pass 64
        cutoff = rng.choice([-1, -1, -2, "mid"])
        cases.append((c, L, m, k, n, rb, cutoff))
    return cases


@pytest.mark.parametrize("case", _sweep_cases(14, 2026))
def test_int8_random_sweep(case):
    c, L, m, k, n, rb, cutoff = case
    if cutoff == "mid":
        w0, S0, _ = md.mdgemm_plan(m, n, k, L, flags=I8, range_bits=rb)
        cutoff = max(0, S0 - 3)
    w, S, T = md.mdgemm_plan(m, n, k, L, flags=I8, cutoff=cutoff, range_bits=rb)
    assert (w, S, T) == exact.plan(L, k, int8=True, cutoff=cutoff, range_bits=rb)
    print(f"[case] int8 sweep {c}: L={L} {m}x{k}x{n} range={rb} w={w} S={S} T={T}", flush=True)
    A, B = _operands(L, m, k, n, 1000 + c, rb)
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B), flags=I8, cutoff=cutoff, range_bits=rb))
    assert np.array_equal(C, pipeline.full_reference(A, B, S, T, w)["C"])
    assert np.array_equal(C, _fp64_same_digits(A, B, w, S, T, rb))
