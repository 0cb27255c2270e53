"""The C-ABI library: it loads, exports every function of include/mdgemm.h, and
its host-side argument checks answer before any HIP call (no GPU needed)."""

import ctypes
import os
import re

import pytest

from oracle import exact
from paper_2607_06881_amd import mdgemm as md

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mdgemm.h")

# fake, non-overlapping device addresses: only the host-side checks read them
FA, FB, FC = 1 << 40, 2 << 40, 3 << 40


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(mdgemm\w*)\s*\(", text, flags=re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(md.LIB_PATH):
        import __graft_entry__

        __graft_entry__.build()
    return md.lib()


def test_header_declares_the_exported_set(lib):
    names = _declared_functions()
    assert names == sorted(md.EXPORTED)
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for st in range(0, -7, -1):
        s = md.status_string(st)
        assert s and s != "unknown status"
    assert md.status_string(-99) == "unknown status"


def test_opts_init_defaults(lib):
    o = md.mdgemm_opts()
    o.flags = 77
    lib.mdgemm_opts_init(ctypes.byref(o))
    assert (o.stream, o.workspace, o.workspace_bytes, o.slices_per_limb, o.cutoff, o.flags) == (None, None, 0, 0, -1,
                                                                                              0)


def _ex(lib, m, n, k, limbs, A=FA, B=FB, C=FC, **kw):
    o = md.mdgemm_opts()
    lib.mdgemm_opts_init(ctypes.byref(o))
    for key, v in kw.items():
        setattr(o, key, v)
    return lib.mdgemm_ex(m, n, k, limbs, A, B, C, ctypes.byref(o))


def test_invalid_arguments(lib):
    E = md.MDGEMM_EINVAL
    assert _ex(lib, -1, 4, 4, 2) == E
    assert _ex(lib, 4, 4, -3, 2) == E
    assert _ex(lib, 4, 4, 4, 0) == E
    assert _ex(lib, 4, 4, 4, md.MDGEMM_MAX_LIMBS + 1) == E
    assert _ex(lib, 4, 4, 4, 2, slices_per_limb=35) == E  # S = 70 > 68
    assert _ex(lib, 4, 4, 4, 16, slices_per_limb=5) == E  # S = 80 > 68
    assert _ex(lib, 4, 4, 4, 2, cutoff=15) == E  # > 2S - 2
    assert _ex(lib, 4, 4, 4, 2, cutoff=-3) == E
    assert _ex(lib, 4, 4, 4, 2, A=None) == E
    assert _ex(lib, 4, 4, 4, 2, C=None) == E
    # C overlapping A
    assert _ex(lib, 4, 4, 4, 2, C=FA + 8) == E
    assert lib.mdgemm_split(4, 4, 2, md.MDGEMM_MAX_SLICES + 1, 13, 0, FA, FB, FC, None) == E
    assert lib.mdgemm_split(4, 4, md.MDGEMM_MAX_LIMBS + 1, 8, 13, 0, FA, FB, FC, None) == E
    assert lib.mdgemm_split(4, 4, 2, 8, 13, 2, FA, FB, FC, None) == E
    assert lib.mdgemm_split(4, 4, 2, 8, 27, 0, FA, FB, FC, None) == E  # digits wider than 26 bits
    assert lib.mdgemm_split(4, 4, 2, 8, 0, 0, FA, FB, FC, None) == E
    assert lib.mdgemm_split(4, 4, 2, 35, 26, 0, FA, FB, FC, None) == E  # 35 x 26 > 908 digit bits
    assert lib.mdgemm_split_panel(4, 4, 2, 0, 13, 0, FA, FB, FC, None) == E
    assert lib.mdgemm_slice_gemm(4, 4, 4, 8, 13, 7, 0, FA + 8, FB, FC, None) == E  # panels must be 16-byte aligned
    assert lib.mdgemm_slice_gemm(4, 4, 4, 8, 13, 15, 0, FA, FB, FC, None) == E
    assert lib.mdgemm_slice_gemm(4, 4, 4, md.MDGEMM_MAX_SLICES + 1, 13, 7, 0, FA, FB, FC, None) == E
    assert lib.mdgemm_slice_gemm(4, 4, 4, 8, 27, 7, 0, FA, FB, FC, None) == E
    assert lib.mdgemm_accumulate(4, 4, md.MDGEMM_MAX_LEVELS + 1, 13, FA, FC, None) == E
    assert lib.mdgemm_accumulate(4, 4, 80, 26, FA, FC, None) == E  # 26 x 79 + 55 bits > 28 words
    assert lib.mdgemm_accum_renorm(4, 4, md.MDGEMM_MAX_LIMBS + 1, 8, 13, FA, FB, FB, FC, None) == E
    assert lib.mdgemm_accum_renorm(4, 4, 2, md.MDGEMM_MAX_LEVELS + 1, 13, FA, FB, FB, FC, None) == E
    assert lib.mdgemm_accum_renorm(4, 4, 2, 8, 0, FA, FB, FB, FC, None) == E
    assert _ex(lib, 4, 4, 4, 2, slice_bits=27) == E
    assert _ex(lib, 4, 4, 4, 2, slice_bits=-2) == E
    assert _ex(lib, 4, 4, 4, 2, slice_bits=md.MDGEMM_SLICE_BITS_AUTO, slices=6) == E
    assert _ex(lib, 4, 4, 4, 16, slice_bits=23, slices=40) == E  # 40 x 23 > 908
    assert lib.mdgemm_exponents(4, 4, 3, FA, FB, None) == E
    # m, n at most 2^27 (the level GEMM's 32-bit panel row offsets)
    assert _ex(lib, 2**27 + 1, 4, 4, 2, C=FC + (1 << 44)) == E
    assert _ex(lib, 4, 2**27 + 1, 4, 2, C=FC + (1 << 44)) == E
    assert md.mdgemm_workspace_bytes(2**27 + 1, 16, 16, 2) == 2**64 - 1


def test_empty_products_are_noops(lib):
    assert _ex(lib, 0, 5, 5, 2, A=None, B=None, C=None) == md.MDGEMM_OK
    assert _ex(lib, 5, 0, 5, 2, A=None, B=None, C=None) == md.MDGEMM_OK
    assert lib.mdgemm_split(0, 5, 2, 8, 13, 0, None, None, None, None) == md.MDGEMM_OK
    assert lib.mdgemm_slice_gemm(0, 5, 5, 8, 13, 7, 0, None, None, None, None) == md.MDGEMM_OK
    assert lib.mdgemm_exponents(0, 5, 0, None, None, None) == md.MDGEMM_OK


def _max_k(pairs):
    # largest k with pairs * k * 8191^2 < 2^53 (the exactness bound of the level sums)
    return (2**53 - 1) // (pairs * 8191**2)


@pytest.mark.parametrize("limbs,cutoff,pairs", [(2, -1, 8), (2, -2, 8), (4, -1, 16), (1, 0, 1), (3, 5, 6),
                                                (8, -1, 34), (16, -1, 66), (16, -2, 66)])
def test_exactness_bound(lib, limbs, cutoff, pairs):
    S = exact.default_slices(limbs)
    kmax = _max_k(pairs)
    assert _ex(lib, 4, 4, kmax + 1, limbs, cutoff=cutoff) == md.MDGEMM_EEXACT
    # at kmax the check passes and the call goes on to the workspace check
    assert _ex(lib, 4, 4, kmax, limbs, cutoff=cutoff, workspace=FC + (1 << 40),
               workspace_bytes=16) == md.MDGEMM_EWORKSPACE
    assert lib.mdgemm_slice_gemm(4, 4, kmax + 1, S, 13, cutoff if cutoff >= 0 else S - 1, 0, FA, FB, FC,
                                 None) == md.MDGEMM_EEXACT


def test_workspace_bytes_layout(lib):
    def expect(m, n, k, L, S, T):
        a = lambda x: (x + 255) // 256 * 256
        # 13-bit digits: FP32 panels with k rounded up to 32
        kp, mp, np_ = md.panel_k32(k), md.panel_mn(m), md.panel_mn(n)
        # pair schedule table (these shapes keep whole k): 3 words per level job, one per
        # pair, T + 2 chunk starts, an even word, one chunk (2 words) per level, 2 words
        # per digit of A and of B
        pairs = sum(len(exact.pairs_of_level(t, S)) for t in range(T + 1))
        words = 3 * (T + 1) + pairs + (T + 2)
        words += words % 2 + 2 * (T + 1) + 4 * S
        return (a(4 * m) + a(4 * n) + a(4) + a(4 * words) + a(4 * S * kp * mp) + a(4 * S * kp * np_) +
                a(8 * (T + 1) * m * n))

    assert md.mdgemm_workspace_bytes(100, 70, 33, 2) == expect(100, 70, 33, 2, 8, 7)
    assert md.mdgemm_workspace_bytes(100, 70, 33, 2, cutoff=-2) == expect(100, 70, 33, 2, 8, 14)
    assert md.mdgemm_workspace_bytes(64, 64, 64, 4, slices_per_limb=3, cutoff=5) == expect(64, 64, 64, 4, 12, 5)
    assert md.mdgemm_workspace_bytes(0, 64, 64, 2) == 0
    assert md.mdgemm_workspace_bytes(256, 8192, 128, 8) == expect(256, 8192, 128, 8, 34, 33)
    assert md.mdgemm_workspace_bytes(128, 8192, 64, 16) == expect(128, 8192, 64, 16, 66, 65)
    assert md.mdgemm_workspace_bytes(4, 4, 4, md.MDGEMM_MAX_LIMBS + 1) == 2**64 - 1


def test_workspace_too_small_is_reported_before_any_launch(lib):
    need = md.mdgemm_workspace_bytes(40, 30, 20, 3)
    assert _ex(lib, 40, 30, 20, 3, workspace=FC + (1 << 40), workspace_bytes=need - 1) == md.MDGEMM_EWORKSPACE


@pytest.mark.parametrize("flags", [0, md.MDGEMM_INT8])
def test_workspace_overlapping_an_operand_is_refused_before_any_launch(lib, flags):
    m, n, k, L = 40, 30, 20, 3
    need = md.mdgemm_workspace_bytes(m, n, k, L, flags=flags)
    abytes, bbytes, cbytes = 8 * L * m * k, 8 * L * k * n, 8 * L * m * n
    far = FC + (1 << 40)
    # each operand's first and last byte inside the workspace, and the workspace
    # starting inside each operand
    for ws in (FA - need + 1, FA + abytes - 1, FB - need + 8, FB + bbytes - 8, FC - need + 1, FC + cbytes - 1):
        assert _ex(lib, m, n, k, L, workspace=ws, workspace_bytes=need, flags=flags) == md.MDGEMM_EINVAL, hex(ws)
    # adjacent on both sides is fine: the call goes on to the HIP calls, which
    # without a device return MDGEMM_EHIP (never run with a device: the fake
    # addresses would then reach a kernel)
    import torch

    if torch.cuda.is_available():
        return
    for ws in (FA - need, FA + abytes):
        assert _ex(lib, m, n, k, L, workspace=ws, workspace_bytes=need, flags=flags) != md.MDGEMM_EINVAL
    assert _ex(lib, m, n, k, L, workspace=far, workspace_bytes=need, flags=flags) != md.MDGEMM_EINVAL


def test_workspace_layout_of_staged_and_fused_products(lib):
    # small outputs run the fused kernel, which leaves nothing in the workspace:
    # the layout is refused for them unless MDGEMM_STAGED selects the stages
    with pytest.raises(md.MdgemmError) as ei:
        md.mdgemm_workspace_layout(64, 64, 64, 2)
    assert ei.value.status == md.MDGEMM_EINVAL
    lay = md.mdgemm_workspace_layout(64, 64, 64, 2, flags=md.MDGEMM_STAGED)
    assert lay["total"] == md.mdgemm_workspace_bytes(64, 64, 64, 2) and lay["planes"] == 8
    # beyond 256 tiles of 16 x 16, or where the staged path's estimated time is lower
    # (64 x 64 x 4096: about 950 us fused), the stages run
    lay = md.mdgemm_workspace_layout(257, 256, 64, 2)
    assert lay["direct_levels"] == 1 and lay["panel_bytes"] == 4 and lay["planes"] == 8
    assert md.mdgemm_workspace_layout(64, 64, 4096, 2)["planes"] >= 8
    a = lambda x: (x + 255) // 256 * 256
    lay = md.mdgemm_workspace_layout(300, 270, 100, 3)
    assert lay["ea"] == 0 and lay["eb"] == a(4 * 300) and lay["kp"] == 128 and lay["mp"] == 384
    assert lay["np"] == 384 and lay["planes"] == 12 and lay["total"] == md.mdgemm_workspace_bytes(300, 270, 100, 3)


def _fused(m, n, k, L, **opts):
    try:
        md.mdgemm_workspace_layout(m, n, k, L, **opts)
    except md.MdgemmError as e:
        return e.status == md.MDGEMM_EINVAL
    return False


def test_fused_path_taken_where_its_estimated_time_is_lower(lib):
    # the fused kernel runs where its estimated time is below the staged path's;
    # each pair below was measured side by side on MI355X (fused / staged, us)
    auto = md.MDGEMM_SLICE_BITS_AUTO
    assert _fused(64, 64, 64, 2) and _fused(45, 60, 130, 4)   # 28.5 / 65.7, 104 / 208
    assert _fused(17, 33, 512, 2)                             # 123 / 173
    assert not _fused(17, 33, 1536, 2)                        # 342 / 192: k split 6 ways
    assert not _fused(17, 33, 1024, 1)                        # 124 / 103
    assert _fused(128, 128, 1024, 1)                          # 124 / 169: 128 x 128 tiles
    assert _fused(64, 960, 640, 2, slice_bits=auto)           # 135 / 175
    assert not _fused(64, 960, 1024, 2, slice_bits=auto)      # 207 / 158
    assert _fused(256, 256, 800, 2)                           # 198 / 335
    assert _fused(100, 100, 400, 3)                           # 180 / 660
    assert not _fused(17, 33, 1200, 3)                        # 504 / 309
    assert _fused(256, 256, 450, 4)                           # 326 / 998
    assert not _fused(45, 60, 1000, 4)                        # 639 / 334
    assert not _fused(17, 33, 512, 2, flags=md.MDGEMM_STAGED)


def test_taylor_refusals(lib):
    # sizes out of range have no workspace; null pointers and a short workspace
    # are refused before any device work
    big = 2**64 - 1
    assert lib.mdgemm_taylor_dd_workspace_bytes(0, 1, 0) == big
    assert lib.mdgemm_taylor_dd_workspace_bytes(4, 0, 0) == big
    assert lib.mdgemm_taylor_dd_workspace_bytes(4, 1, -1) == big
    assert lib.mdgemm_taylor_dd_workspace_bytes(40000, 1, 0) == big
    need = lib.mdgemm_taylor_dd_workspace_bytes(20, 3, 2)
    assert 0 < need < big and need > lib.mdgemm_taylor_dd_workspace_bytes(20, 3, 1)
    assert lib.mdgemm_taylor_dd(20, 3, 2, None, None, None, None, need, None) == md.MDGEMM_EINVAL
    fake = ctypes.c_void_p(1 << 40)
    assert lib.mdgemm_taylor_dd(20, 3, 2, fake, ctypes.c_void_p(2 << 40), ctypes.c_void_p(3 << 40),
                                ctypes.c_void_p(4 << 40), need - 1, None) == md.MDGEMM_EWORKSPACE
    # X on top of A, or the workspace on top of B: refused
    assert lib.mdgemm_taylor_dd(20, 3, 2, fake, ctypes.c_void_p(2 << 40), ctypes.c_void_p((1 << 40) + 64),
                                ctypes.c_void_p(4 << 40), need, None) == md.MDGEMM_EINVAL
    assert lib.mdgemm_taylor_dd(20, 3, 2, fake, ctypes.c_void_p(2 << 40), ctypes.c_void_p(3 << 40),
                                ctypes.c_void_p((2 << 40) - 64), need, None) == md.MDGEMM_EINVAL


def test_binding_refuses_cpu_tensors(lib):
    import torch

    A = torch.zeros(2, 4, 4, dtype=torch.float64)
    with pytest.raises(ValueError):
        md.mdgemm_ex(A, A)
    with pytest.raises(TypeError):
        md.mdgemm_ex(A.float(), A.float())


def test_plan_digit_width_and_count(lib):
    auto = md.MDGEMM_SLICE_BITS_AUTO
    # 13-bit digits: four per limb up to four limbs, ceil((53 L - 4) / 13) + 1 beyond,
    # or slices_per_limb, or an explicit count
    assert md.mdgemm_plan(64, 64, 64, 2) == (13, 8, 7)
    assert md.mdgemm_plan(64, 64, 64, 4) == (13, 16, 15)
    assert md.mdgemm_plan(64, 64, 64, 5) == (13, 22, 21)  # 261 bits: 21 digits + 1
    assert md.mdgemm_plan(64, 64, 64, 8) == (13, 34, 33)  # 420 bits: 33 digits + 1
    assert md.mdgemm_plan(64, 64, 64, 16) == (13, 66, 65)  # 844 bits: 65 digits + 1
    assert md.mdgemm_plan(64, 64, 64, 8, slices_per_limb=4) == (13, 32, 31)
    assert md.mdgemm_plan(64, 64, 64, 3, slices_per_limb=3, cutoff=-2) == (13, 9, 16)
    assert md.mdgemm_plan(64, 64, 64, 2, slices=9, cutoff=4) == (13, 9, 4)
    # explicit width: ceil(13 S13(L) / w) digits unless given
    assert md.mdgemm_plan(64, 64, 64, 2, slice_bits=19) == (19, 6, 5)
    assert md.mdgemm_plan(64, 64, 4, 4, slice_bits=21) == (21, 10, 9)
    assert md.mdgemm_plan(64, 64, 64, 2, slice_bits=17, slices=5, cutoff=-2) == (17, 5, 8)
    # the adaptive width at the workloads' k: closed forms worked by hand
    assert md.mdgemm_plan(4096, 4096, 4096, 2, slice_bits=auto) == (19, 6, 5)  # 21 pairs instead of 36
    assert md.mdgemm_plan(2048, 2048, 1024, 4, slice_bits=auto) == (19, 11, 10)  # 66 instead of 136
    assert md.mdgemm_plan(8192, 8192, 512, 3, slice_bits=auto) == (20, 8, 7)  # 36 instead of 78
    assert md.mdgemm_plan(128, 8192, 64, 16, slice_bits=auto) == (20, 43, 42)  # 946 instead of 2211
    for L in (1, 2, 3, 4, 8, 16):
        for k in (1, 7, 64, 512, 1000, 4096, 2**16, 2**20, 2**22):
            want = exact.adaptive_width(L, k)
            if want is None:
                with pytest.raises(md.MdgemmError):
                    md.mdgemm_plan(8, 8, k, L, slice_bits=auto)
            else:
                assert md.mdgemm_plan(8, 8, k, L, slice_bits=auto) == (*want, want[1] - 1), (L, k)


def test_exactness_bound_wide_digits(lib):
    # pairs * k * (2^w - 1)^2 < 2^53 with the width in the check
    w, S = 19, 6
    kmax = (2**53 - 1) // (S * (2**w - 1) ** 2)
    assert md.mdgemm_plan(4, 4, kmax, 2, slice_bits=w) == (w, S, S - 1)
    with pytest.raises(md.MdgemmError):
        md.mdgemm_plan(4, 4, kmax + 1, 2, slice_bits=w)
    assert lib.mdgemm_slice_gemm(4, 4, kmax + 1, S, w, S - 1, 0, FA, FB, FC, None) == md.MDGEMM_EEXACT
    assert md.mdgemm_workspace_bytes(4096, 4096, 4096, 2, slice_bits=md.MDGEMM_SLICE_BITS_AUTO) < \
        md.mdgemm_workspace_bytes(4096, 4096, 4096, 2)


def test_plan_matches_the_oracle_reading_of_the_options(lib):
    # The library's option resolution against the oracle's, written separately
    # from the same definitions (exact.plan), over a grid of option combinations.
    combos = 0
    for L in (1, 2, 3, 4, 8, 16):
        for k in (1, 64, 2048, 2**20):
            for slice_bits in (0, 13, 17, 22, md.MDGEMM_SLICE_BITS_AUTO):
                for slices in (0, 9):
                    for cutoff in (-1, -2, 5):
                        for range_bits in (0, 13, 60):
                            kw = dict(slice_bits=slice_bits, slices=slices, cutoff=cutoff, range_bits=range_bits)
                            try:
                                want = exact.plan(L, k, **kw)
                                err = None if want is not None else md.MDGEMM_EEXACT
                            except ValueError:
                                want, err = None, md.MDGEMM_EINVAL
                            if err is None:
                                assert md.mdgemm_plan(8, 8, k, L, **kw) == want, (L, k, kw)
                            else:
                                with pytest.raises(md.MdgemmError) as ei:
                                    md.mdgemm_plan(8, 8, k, L, **kw)
                                assert ei.value.status == err, (L, k, kw)
                            combos += 1
    assert combos == 6 * 4 * 5 * 2 * 3 * 3


def test_int8_plans(lib):
    I8 = md.MDGEMM_INT8
    # double-double at k = 4096: 7-bit digits, ceil(104 / 7) = 15, T = 14 (120 pairs);
    # 15 k 127^2 < 2^31 up to k = 8876, beyond that narrower digits
    assert md.mdgemm_plan(4096, 4096, 4096, 2, flags=I8) == (7, 15, 14)
    assert md.mdgemm_plan(64, 64, 8876, 2, flags=I8) == (7, 15, 14)
    assert md.mdgemm_plan(64, 64, 8877, 2, flags=I8) == (6, 18, 17)
    assert md.mdgemm_plan(64, 64, 65536, 2, flags=I8) == (5, 21, 20)
    assert md.mdgemm_plan(64, 64, 64, 8, flags=I8) == (7, 64, 63)  # ceil(442 / 7)
    assert md.mdgemm_plan(64, 64, 64, 2, flags=I8, slice_bits=4) == (4, 26, 25)
    assert md.mdgemm_plan(64, 64, 2048, 2, flags=I8, range_bits=60) == (7, 24, 32)
    E = md.MDGEMM_EINVAL
    for kw in (dict(slice_bits=8), dict(slice_bits=13), dict(slices=9), dict(flags=I8 | md.MDGEMM_KARATSUBA),
               dict(flags=I8 | md.MDGEMM_KARATSUBA_MIN_TERMS)):
        kw.setdefault("flags", I8)
        with pytest.raises(md.MdgemmError) as ei:
            md.mdgemm_plan(64, 64, 64, 2, **kw)
        assert ei.value.status == E, kw
    with pytest.raises(md.MdgemmError) as ei:  # hexa-double: ceil(858 / 7) = 123 digits > 64
        md.mdgemm_plan(64, 64, 64, 16, flags=I8)
    assert ei.value.status == E
    with pytest.raises(md.MdgemmError) as ei:  # even 1-bit digits overflow int32 sums
        md.mdgemm_plan(4, 4, 2**31, 1, flags=I8)
    assert ei.value.status == md.MDGEMM_EEXACT
    assert _ex(lib, 4, 4, 2**31, 1, flags=I8) == md.MDGEMM_EEXACT
    # workspace: EA, EB, flag, int8 digits of A and of B (rows of 128 zero bytes + S kp,
    # kp = k rounded up to 128, m and n rounded up to 256 rows), int32 levels, 256-byte aligned
    def al(x):
        return (x + 255) // 256 * 256
    m, n, k, S, T = 100, 70, 300, 15, 14
    kp, mp, np_ = 384, 256, 256
    ld = 128 + S * kp
    want = al(4 * m) + al(4 * n) + al(4) + al(mp * ld) + al(np_ * ld) + al(4 * (T + 1) * m * n)
    assert md.mdgemm_workspace_bytes(m, n, k, 2, flags=I8) == want


def test_int8_plans_match_the_oracle_reading(lib):
    combos = 0
    for L in (1, 2, 3, 4, 8, 16):
        for k in (1, 64, 4096, 9000, 2**20):
            for slice_bits in (0, 3, 7, md.MDGEMM_SLICE_BITS_AUTO):
                for cutoff in (-1, -2, 5):
                    for range_bits in (0, 60):
                        kw = dict(slice_bits=slice_bits, cutoff=cutoff, range_bits=range_bits)
                        try:
                            want = exact.plan(L, k, int8=True, **kw)
                            err = None if want is not None else md.MDGEMM_EEXACT
                        except ValueError:
                            want, err = None, md.MDGEMM_EINVAL
                        if err is None:
                            assert md.mdgemm_plan(8, 8, k, L, flags=md.MDGEMM_INT8, **kw) == want, (L, k, kw)
                        else:
                            with pytest.raises(md.MdgemmError) as ei:
                                md.mdgemm_plan(8, 8, k, L, flags=md.MDGEMM_INT8, **kw)
                            assert ei.value.status == err, (L, k, kw)
                        combos += 1
    assert combos == 6 * 5 * 4 * 3 * 2


def test_group_plans_match_the_oracle_reading(lib):
    # exponent classes / sign groups: the library's option resolution against
    # exact.plan's restatement, refusals included
    GE, GS = md.MDGEMM_GROUP_EXPONENT, md.MDGEMM_GROUP_SIGN
    assert md.mdgemm_plan(64, 64, 2048, 2, range_bits=60, flags=GE) == (13, 9, 9)  # 6 classes
    assert md.mdgemm_plan(64, 64, 2048, 2, flags=GS) == (13, 8, 7)
    combos = 0
    for L in (1, 2, 3, 4, 8):
        for k in (64, 2048):
            for flags in (GE, GS, GE | GS):
                for slice_bits in (0, 17, md.MDGEMM_SLICE_BITS_AUTO):
                    for cutoff in (-1, -2, 5):
                        for range_bits in (0, 13, 60):
                            kw = dict(slice_bits=slice_bits, cutoff=cutoff, range_bits=range_bits)
                            try:
                                want = exact.plan(L, k, group_exponent=bool(flags & GE), group_sign=bool(flags & GS),
                                                  **kw)
                                err = None if want is not None else md.MDGEMM_EEXACT
                            except ValueError:
                                want, err = None, md.MDGEMM_EINVAL
                            if err is None:
                                assert md.mdgemm_plan(8, 8, k, L, flags=flags, **kw) == want, (L, k, flags, kw)
                            else:
                                with pytest.raises(md.MdgemmError) as ei:
                                    md.mdgemm_plan(8, 8, k, L, flags=flags, **kw)
                                assert ei.value.status == err, (L, k, flags, kw)
                            combos += 1
    assert combos == 5 * 2 * 3 * 3 * 3 * 3
    for extra in (md.MDGEMM_INT8, md.MDGEMM_KARATSUBA):
        with pytest.raises(md.MdgemmError):
            md.mdgemm_plan(64, 64, 64, 2, flags=GS | extra)
    # the staged workspace: G S panels per operand and T + 1 + 2 (Ge - 1) level planes
    lay = md.mdgemm_workspace_layout(300, 270, 100, 2, range_bits=60, flags=GE | GS)
    assert lay["planes"] == 9 + 1 + 2 * 5 and lay["panel_bytes"] == 4
    assert (lay["db"] - lay["da"]) // (4 * lay["kp"] * lay["mp"]) == 12 * 9


def test_range_balancing_plans(lib):
    # D = ceil(range / w) more digits, default cutoff S0 - 1 + 2D
    assert md.mdgemm_plan(64, 64, 2048, 2, range_bits=60) == (13, 13, 17)
    assert md.mdgemm_plan(64, 64, 2048, 2, range_bits=13) == (13, 9, 9)
    assert md.mdgemm_plan(64, 64, 2048, 2, range_bits=1) == (13, 9, 9)
    assert md.mdgemm_plan(64, 64, 2048, 2, range_bits=60, slice_bits=md.MDGEMM_SLICE_BITS_AUTO) == (19, 10, 13)
    assert md.mdgemm_plan(64, 64, 2048, 2, range_bits=60, cutoff=-2) == (13, 13, 24)
    assert _ex(lib, 4, 4, 4, 2, range_bits=-1) == md.MDGEMM_EINVAL
    assert _ex(lib, 4, 4, 4, 16, range_bits=40) == md.MDGEMM_EINVAL  # 66 + 4 = 70 digits
    E = md.MDGEMM_EINVAL
    assert lib.mdgemm_line_spread(4, 4, 2, FA, FB, FC, None) == E
    assert lib.mdgemm_line_spread(4, 4, 0, FA, FB, FB, None) == E  # E and spread overlap
    assert lib.mdgemm_line_spread(0, 4, 0, None, None, None, None) == md.MDGEMM_OK


def _swz(r):
    # the int8 kernel's granule swizzle of LDS row r (level_gemm_i8.hip, swz)
    return ((r >> 1) & 1) | (((r & 1) ^ ((r >> 3) & 1)) << 1) | (r & 4)


def test_int8_kernel_lds_layout_model():
    """The int8 level kernel's LDS addressing, modelled on the CPU.

    Copies: lane L of copy instruction q of wave w lands at tile row
    32 w + 8 q + L / 8, physical granule L % 8, and fetches logical granule
    (L % 8) ^ swz(row).  Fragment reads: lane l of the wave at tile row
    R = base + 16 i + l % 16 wants logical granule 4 h + l / 16 and reads
    physical granule (4 h + l / 16) ^ swz(l % 16).  Checked: every logical
    granule of every row is written exactly once and read from where it was
    written; and a fragment read meets 16 distinct bank groups (64 banks of
    4 bytes) in each group of lanes that the LDS serves together
    (8a..8a+7 with 32+8a..32+8a+7, as the bank-conflict counter shows on
    gfx950; also 16 and 8 consecutive lanes).
    """
    where = {}
    for w in range(8):
        for q in range(4):
            for L in range(64):
                row = 32 * w + 8 * q + L // 8
                logical = (L % 8) ^ _swz(row)
                assert (row, logical) not in where
                where[(row, logical)] = L % 8
    assert len(where) == 256 * 8
    models = {
        "halves": ([list(range(i, i + 8)) + list(range(i + 32, i + 40)) for i in range(0, 32, 8)], 64),
        "consecutive 16": ([list(range(i, i + 16)) for i in range(0, 64, 16)], 64),
        "consecutive 8": ([list(range(i, i + 8)) for i in range(0, 64, 8)], 32),
    }
    # A: a wave reads 8 blocks of 16 rows from row 0 or 128; B: 4 blocks from 0, 64, 128 or 192
    for base, blocks in [(0, 8), (128, 8), (0, 4), (64, 4), (128, 4), (192, 4)]:
        for i in range(blocks):
            for h in range(2):
                addr = []
                for lane in range(64):
                    R = base + 16 * i + lane % 16
                    logical = 4 * h + lane // 16
                    phys = logical ^ _swz(lane % 16)
                    assert where[(R, logical)] == phys  # read where the copy wrote
                    addr.append(R * 128 + 16 * phys)
                for name, (groups, banks) in models.items():
                    for grp in groups:
                        hit = [(addr[l] // 4 + d) % banks for l in grp for d in range(4)]
                        assert len(set(hit)) == len(hit), (name, base, i, h)
