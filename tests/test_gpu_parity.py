"""GPU parity of every stage of the product against the CPU oracle.

Bit-exact: exponents, digits, level and pair products, the exact accumulated
sums and the final greedy rounding.  Tolerance: the final limbs against the
exact rational product, |C - C_exact| <= 4 k 2^-(53L-4) (|A||B|).  Sizes span
several 128 x 128 tiles and 16-deep k blocks with ragged tails.
"""

import ctypes
import math
import random

import numpy as np
import pytest
import torch

from oracle import coracle, exact, pipeline
from paper_2607_06881_amd import mdgemm as md
from paper_2607_06881_amd import workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _gpu(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _panel(D, axis):
    """Digit planes [S][rows][cols] -> level-GEMM panel (k-major, zero padded)."""
    S, rows, cols = D.shape
    if axis == 0:  # A: [S][kp(cols)][mp(rows)], transposed
        P = np.zeros((S, md.panel_k(cols), md.panel_mn(rows)))
        P[:, :cols, :rows] = D.transpose(0, 2, 1)
    else:  # B: [S][kp(rows)][np(cols)]
        P = np.zeros((S, md.panel_k(rows), md.panel_mn(cols)))
        P[:, :rows, :cols] = D
    return P


def _operands(L, m, k, n, seed, base="uniform", row_exp=0, col_exp=0, elem_exp=0):
    rng = np.random.default_rng(seed)
    A = workloads.make_operand(rng, L, m, k, base, row_exp=row_exp, elem_exp=elem_exp)
    B = workloads.make_operand(rng, L, k, n, base, col_exp=col_exp, elem_exp=elem_exp)
    return A, B


# --------------------------------------------------------------------------
# a1 exponents
# --------------------------------------------------------------------------

@pytest.mark.parametrize("rows,cols", [(1, 1), (7, 300), (300, 7), (129, 257), (1000, 64), (64, 5000)])
def test_exponents(rows, cols):
    print(f"[case] exponents {rows}x{cols}", flush=True)
    rng = np.random.default_rng(rows * 7 + cols)
    X = rng.standard_normal((rows, cols)) * np.ldexp(1.0, rng.integers(-900, 900, (rows, cols)))
    X[rng.random((rows, cols)) < 0.05] = 0.0
    X[0, :] = 0.0  # all-zero row
    if cols > 2:
        X[:, 2] = 0.0  # all-zero column
    X[-1, -1] = 7 * 2.0**-1074  # subnormal
    Xg = _gpu(X)
    for axis in (0, 1):
        got = _host(md.mdgemm_exponents(Xg, axis))
        want = coracle.exponents(X, axis)
        assert np.array_equal(got, want), axis


@pytest.mark.parametrize("rows,cols", [(1, 1), (7, 300), (300, 7), (129, 257), (64, 5000)])
def test_line_spread(rows, cols):
    print(f"[case] line spread {rows}x{cols}", flush=True)
    rng = np.random.default_rng(rows * 7 + cols)
    X = rng.standard_normal((rows, cols)) * np.ldexp(1.0, rng.integers(-80, 80, (rows, cols)))
    X[rng.random((rows, cols)) < 0.1] = 0.0
    if rows > 2:
        X[1, :] = 0.0          # an all-zero row
        X[2, :] = 0.0
        X[2, 0] = 5e-324       # a lone subnormal
    if cols > 2:
        X[:, 1] = 0.0          # an all-zero column
    for axis in (0, 1):
        E, spread = md.mdgemm_line_spread(_gpu(X), axis)
        assert np.array_equal(_host(E), coracle.exponents(X, axis))
        assert _host(spread).tolist() == exact.line_spread(X, axis).tolist()


# --------------------------------------------------------------------------
# a2 split
# --------------------------------------------------------------------------

@pytest.mark.parametrize("L,S,rows,cols,axis", [(1, 4, 33, 70, 0), (2, 8, 65, 129, 0), (2, 8, 130, 17, 1),
                                                 (3, 12, 40, 300, 1), (4, 16, 77, 91, 0), (2, 5, 20, 20, 1),
                                                 (4, 13, 31, 33, 1), (3, 16, 9, 9, 0),
                                                 (8, 32, 40, 70, 0), (8, 40, 17, 130, 1), (16, 64, 20, 33, 1),
                                                 (16, 64, 129, 18, 0), (16, 16, 9, 9, 0), (5, 20, 33, 17, 1)])
def test_split_random(L, S, rows, cols, axis):
    print(f"[case] split L={L} S={S} {rows}x{cols} axis={axis}", flush=True)
    rng = np.random.default_rng(L * 100 + S)
    X = workloads.make_operand(rng, L, rows, cols, "normal", elem_exp=12,
                               row_exp=20 if axis == 0 else 0, col_exp=20 if axis == 1 else 0)
    X[:, rng.random((rows, cols)) < 0.05] = 0.0
    E = coracle.exponents(X[0], axis)
    Xg = _gpu(X)
    Eg = md.mdgemm_exponents(Xg[0], axis)
    assert np.array_equal(_host(Eg), E)
    got = _host(md.mdgemm_split(Xg, Eg, S, axis))
    want = coracle.split(X, E, S, axis)
    assert np.array_equal(got, want)
    assert not np.signbit(got[got == 0]).any()  # zero digits are +0.0
    # the same digits as a level-GEMM panel, padding included
    pan = _host(md.mdgemm_split_panel(Xg, Eg, S, axis))
    assert np.array_equal(pan, _panel(want, axis))
    assert not np.signbit(pan[pan == 0]).any()


@pytest.mark.parametrize("L,S,bits,rows,cols,axis", [(2, 6, 19, 65, 129, 0), (4, 11, 19, 40, 300, 1),
                                                      (16, 42, 20, 20, 33, 1), (1, 2, 26, 33, 70, 0),
                                                      (3, 8, 20, 130, 17, 1), (8, 21, 20, 9, 129, 0),
                                                      (2, 5, 22, 129, 16, 0), (16, 64, 13, 5, 7, 1)])
def test_split_wide_digits(L, S, bits, rows, cols, axis):
    print(f"[case] split L={L} S={S} bits={bits} {rows}x{cols} axis={axis}", flush=True)
    rng = np.random.default_rng(L * 100 + S + bits)
    X = workloads.make_operand(rng, L, rows, cols, "normal", elem_exp=12,
                               row_exp=20 if axis == 0 else 0, col_exp=20 if axis == 1 else 0)
    X[:, rng.random((rows, cols)) < 0.05] = 0.0
    E = coracle.exponents(X[0], axis)
    Xg, Eg = _gpu(X), _gpu(E)
    want = coracle.split(X, E, S, axis, bits)
    got = _host(md.mdgemm_split(Xg, Eg, S, axis, bits=bits))
    assert np.array_equal(got, want)
    assert not np.signbit(got[got == 0]).any()
    pan = _host(md.mdgemm_split_panel(Xg, Eg, S, axis, bits=bits))
    assert np.array_equal(pan, _panel(want, axis))


def _adversarial_elements(L, count, seed):
    """Multiple doubles with opposite-signed limbs, half-ulp tails, gaps,
    exact zeros below nonzeros, powers of two and subnormal tails."""
    rng = random.Random(seed)
    out = []
    for _ in range(count):
        x0 = rng.choice([-1, 1]) * rng.choice([1.0, 0.5, 0.75, 1 - 2.0**-53, rng.uniform(0.5, 1)]) \
            * 2.0 ** rng.randint(-30, 30)
        limbs = [x0]
        for _ in range(1, L):
            prev = limbs[-1]
            if prev == 0.0:
                limbs.append(0.0)
                continue
            h = math.ulp(prev) / 2
            kind = rng.random()
            if kind < 0.2:
                y = rng.choice([-1, 1]) * h
            elif kind < 0.35:
                y = 0.0
            elif kind < 0.5:
                y = rng.choice([-1, 1]) * h * 2.0 ** -rng.randint(1, 60)
            else:
                y = rng.uniform(-1, 1) * h
            limbs.append(y)
        out.append(limbs)
    return out


@pytest.mark.parametrize("L", [2, 3, 4, 8, 16])
def test_split_adversarial(L):
    print(f"[case] split adversarial L={L}", flush=True)
    els = _adversarial_elements(L, 64 * 33, 900 + L)
    X = np.array(els).T.reshape(L, 64, 33).copy()
    assert all(exact.is_nonoverlapping(X[:, r, c]) for r in range(64) for c in range(33))
    for axis in (0, 1):
        E = coracle.exponents(X[0], axis)
        for S in (4 * L, 4 * L - 1, 3):
            got = _host(md.mdgemm_split(_gpu(X), _gpu(E), S, axis))
            want = coracle.split(X, E, S, axis)
            assert np.array_equal(got, want), (axis, S)
            pan = _host(md.mdgemm_split_panel(_gpu(X), _gpu(E), S, axis))
            assert np.array_equal(pan, _panel(want, axis)), (axis, S)


def test_split_golden_cases():
    print("[case] split golden", flush=True)
    fbits = "1001000110100110011001001110110100100011010011001100"
    x = int(fbits, 2) * 2.0**-52
    X = np.array([x]).reshape(1, 1, 1)
    got = _host(md.mdgemm_split(_gpu(X), _gpu(np.array([0], np.int32)), 4, 0)).ravel()
    assert got.tolist() == [0x1234, 0x1993, 0x1691, 0x14CC]
    # opposite-sign limbs (the borrow of section 3)
    X = np.array([1.0, -(2.0**-60)]).reshape(2, 1, 1)
    got = _host(md.mdgemm_split(_gpu(X), _gpu(np.array([1], np.int32)), 8, 0)).ravel()
    assert got.tolist() == [4095, 8191, 8191, 8191, 8176, 0, 0, 0]


# --------------------------------------------------------------------------
# a3 level and pair GEMMs
# --------------------------------------------------------------------------

@pytest.mark.parametrize("S,T,m,k,n", [(8, 7, 65, 37, 129), (8, 14, 130, 50, 131), (4, 3, 1, 1, 1),
                                       (12, 11, 200, 33, 70), (16, 15, 64, 16, 64), (16, 30, 33, 20, 17),
                                       (3, 2, 257, 129, 300), (8, 7, 16, 1, 16),
                                       # tile grids with partial tile-row groups and uneven XCD chunks
                                       (8, 7, 1100, 40, 900), (4, 3, 3000, 17, 130), (2, 2, 130, 33, 2900),
                                       # octo / hexa doubles: 32 and 64 digits, up to 127 levels
                                       (32, 31, 130, 20, 140), (64, 63, 70, 17, 129), (64, 126, 20, 5, 30),
                                       (40, 32, 33, 45, 257)])
def test_levels(S, T, m, k, n):
    print(f"[case] levels S={S} T={T} {m}x{k}x{n}", flush=True)
    rng = np.random.default_rng(S * 1000 + m)
    DA = rng.integers(-8191, 8192, (S, m, k)).astype(np.float64)
    DB = rng.integers(-8191, 8192, (S, k, n)).astype(np.float64)
    DA[:, rng.random((m, k)) < 0.1] = 0.0
    got = _host(md.mdgemm_slice_gemm(_gpu(_panel(DA, 0)), _gpu(_panel(DB, 1)), m, n, k, T))
    want = coracle.levels(DA, DB, T)
    assert np.array_equal(got, want.astype(np.float64))


@pytest.mark.parametrize("S,T,bits,m,k,n", [(6, 5, 19, 130, 40, 129), (2, 0, 26, 65, 1, 70), (5, 4, 22, 33, 64, 257),
                                            (11, 10, 19, 40, 100, 45), (42, 41, 20, 20, 9, 130), (8, 14, 20, 17, 64, 17)])
def test_levels_wide_digits(S, T, bits, m, k, n):
    # digits up to 2^w - 1 at the largest k the exactness condition allows nearby
    print(f"[case] levels S={S} T={T} bits={bits} {m}x{k}x{n}", flush=True)
    assert min(S, T + 1) * k * (2**bits - 1) ** 2 < 2**53
    rng = np.random.default_rng(S * 1000 + bits)
    top = 2**bits
    DA = rng.integers(-top + 1, top, (S, m, k)).astype(np.float64)
    DB = rng.integers(-top + 1, top, (S, k, n)).astype(np.float64)
    DA[:, 0, :] = top - 1  # largest digits
    DB[:, :, 0] = -(top - 1)
    got = _host(md.mdgemm_slice_gemm(_gpu(_panel(DA, 0)), _gpu(_panel(DB, 1)), m, n, k, T, bits=bits))
    want = coracle.levels(DA, DB, T)
    assert np.array_equal(got, want.astype(np.float64))


@pytest.mark.parametrize("S,T", [(8, 14), (8, 7), (4, 2), (32, 31), (24, 46)])
def test_pair_products(S, T):
    print(f"[case] pairs S={S} T={T}", flush=True)
    rng = np.random.default_rng(S + T)
    m, k, n = 70, 45, 140
    DA = rng.integers(-8191, 8192, (S, m, k)).astype(np.float64)
    DB = rng.integers(-8191, 8192, (S, k, n)).astype(np.float64)
    out = torch.full((S, S, m, n), -1.0, dtype=torch.float64, device=DEV)
    got = _host(md.mdgemm_slice_gemm(_gpu(_panel(DA, 0)), _gpu(_panel(DB, 1)), m, n, k, T, per_pair=True, out=out))
    want = coracle.levels(DA, DB, T, per_pair=True)
    for p in range(S):
        for q in range(S):
            if p + q <= T:
                assert np.array_equal(got[p, q], want[p, q].astype(np.float64)), (p, q)
            else:
                assert (got[p, q] == -1.0).all(), (p, q)  # untouched


def test_levels_near_exactness_limit():
    # All digits 8191: G_t = pairs_t k 8191^2 in closed form, up to 2^51.
    print("[case] levels near 2^53", flush=True)
    S, T, m, n, k = 16, 15, 128, 128, 2**21
    DA = torch.full((S, k, m), 8191.0, dtype=torch.float64, device=DEV)  # panels: k-major, already whole tiles
    DB = torch.full((S, k, n), -8191.0, dtype=torch.float64, device=DEV)
    got = _host(md.mdgemm_slice_gemm(DA, DB, m, n, k, T))
    for t in range(T + 1):
        want = -float(len(exact.pairs_of_level(t, S)) * k * 8191**2)
        assert (got[t] == want).all(), t
    assert abs(got[15, 0, 0]) > 2**50
    del DA, DB
    torch.cuda.empty_cache()


# --------------------------------------------------------------------------
# a4 accumulation and a5 rounding
# --------------------------------------------------------------------------

def _words_to_int(words):
    v = 0
    for w in range(len(words)):
        v |= (int(words[w]) & ((1 << 64) - 1)) << (64 * w)
    if v >> (64 * len(words) - 1):
        v -= 1 << (64 * len(words))
    return v


@pytest.mark.parametrize("levels", [1, 2, 5, 8, 12, 15, 16, 31, 32, 63, 64, 100, 127])
def test_accumulate_exact(levels):
    print(f"[case] accumulate levels={levels}", flush=True)
    rng = np.random.default_rng(levels)
    m, n = 9, 300
    G = rng.integers(-(2**53) + 1, 2**53, (levels, m, n)).astype(np.float64)
    G[:, 0, :] = 2.0**53 - 1  # largest allowed magnitudes
    G[:, 1, :] = -(2.0**53 - 1)
    G[:, 2, :] = 0.0
    G[:, 3, ::2] = rng.integers(-5, 5, (levels, (n + 1) // 2))
    Z = _host(md.mdgemm_accumulate(_gpu(G)))
    T = levels - 1
    for i in range(m):
        for j in range(0, n, 7):
            want = sum(int(G[t, i, j]) << (13 * (T - t)) for t in range(levels))
            assert _words_to_int(Z[:, i, j]) == want, (i, j)


@pytest.mark.parametrize("levels,bits", [(6, 19), (3, 26), (83, 20), (100, 14), (11, 19), (1, 22)])
def test_accumulate_wide_digits(levels, bits):
    print(f"[case] accumulate levels={levels} bits={bits}", flush=True)
    rng = np.random.default_rng(levels + 1000 * bits)
    m, n = 7, 200
    G = rng.integers(-(2**53) + 1, 2**53, (levels, m, n)).astype(np.float64)
    G[:, 0, :] = 2.0**53 - 1
    G[:, 1, :] = -(2.0**53 - 1)
    G[:, 2, :] = 0.0
    Z = _host(md.mdgemm_accumulate(_gpu(G), bits=bits))
    T = levels - 1
    for i in range(m):
        for j in range(0, n, 7):
            want = sum(int(G[t, i, j]) << (bits * (T - t)) for t in range(levels))
            assert _words_to_int(Z[:, i, j]) == want, (i, j)


def _cases_for_rounding(levels, m, n, seed):
    rng = np.random.default_rng(seed)
    G = np.zeros((levels, m, n))
    kind = rng.integers(0, 6, (m, n))
    for i in range(m):
        for j in range(n):
            c = kind[i, j]
            if c == 0:  # generic
                G[:, i, j] = rng.integers(-(2**52), 2**52, levels)
            elif c == 1:  # sparse, small
                G[:, i, j] = rng.integers(-3, 4, levels) * (rng.random(levels) < 0.3)
            elif c == 2:  # ties: value = odd * 2^s + exactly half an ulp
                G[:, i, j] = 0
                G[0, i, j] = 2**52 + 1
                if levels > 4:
                    G[4, i, j] = 2**51  # 2^51 2^-52 = 1/2 unit of the 53-bit lead
            elif c == 3 and levels >= 2:  # cancellation across levels
                g = int(rng.integers(1, 2**40))
                G[:, i, j] = 0
                G[0, i, j] = g
                G[1, i, j] = -g * 8192 + int(rng.integers(-5, 5))
            elif c == 4:  # only the last level
                G[:, i, j] = 0
                G[-1, i, j] = rng.integers(-(2**52), 2**52)
            else:  # alternating signs of maximal size
                G[:, i, j] = (2**53 - 1) * np.where(np.arange(levels) % 2 == 0, 1, -1)
    return G


@pytest.mark.parametrize("L,levels", [(1, 4), (2, 8), (2, 15), (3, 12), (4, 16), (4, 31), (2, 1), (8, 32), (8, 63),
                                      (16, 64), (16, 127), (5, 40)])
def test_accum_renorm_greedy_rounding(L, levels):
    print(f"[case] accum_renorm L={L} levels={levels}", flush=True)
    m, n = 13, 71
    G = _cases_for_rounding(levels, m, n, 10 * L + levels)
    rng = np.random.default_rng(levels)
    EA = rng.integers(-40, 40, m).astype(np.int32)
    EB = rng.integers(-40, 40, n).astype(np.int32)
    C = _host(md.mdgemm_accum_renorm(_gpu(G), _gpu(EA), _gpu(EB), L))
    for i in range(m):
        for j in range(n):
            z = exact.accumulate([int(g) for g in G[:, i, j]], int(EA[i]), int(EB[j]))
            want = exact.round_to_limbs(z, L)
            assert C[:, i, j].tolist() == want, (i, j, G[:, i, j])
            assert not any(v == 0 and math.copysign(1, v) < 0 for v in C[:, i, j])


@pytest.mark.parametrize("L,levels,bits", [(2, 6, 19), (4, 11, 19), (16, 42, 20), (3, 8, 20), (1, 2, 26), (8, 21, 20)])
def test_accum_renorm_wide_digits(L, levels, bits):
    print(f"[case] accum_renorm L={L} levels={levels} bits={bits}", flush=True)
    m, n = 13, 71
    G = _cases_for_rounding(levels, m, n, 10 * L + levels + bits)
    rng = np.random.default_rng(levels + bits)
    EA = rng.integers(-40, 40, m).astype(np.int32)
    EB = rng.integers(-40, 40, n).astype(np.int32)
    C = _host(md.mdgemm_accum_renorm(_gpu(G), _gpu(EA), _gpu(EB), L, bits=bits))
    for i in range(m):
        for j in range(n):
            z = exact.accumulate([int(g) for g in G[:, i, j]], int(EA[i]), int(EB[j]), bits)
            assert C[:, i, j].tolist() == exact.round_to_limbs(z, L), (i, j)
            assert not any(v == 0 and math.copysign(1, v) < 0 for v in C[:, i, j])


# --------------------------------------------------------------------------
# end to end
# --------------------------------------------------------------------------

@pytest.mark.parametrize("L,m,k,n,cutoff,seed", [(2, 64, 64, 64, -2, 0), (2, 130, 47, 129, -1, 1),
                                                 (1, 65, 33, 17, -2, 2), (3, 40, 100, 70, -1, 3),
                                                 (4, 33, 20, 45, -1, 4), (4, 17, 64, 9, -2, 5),
                                                 (2, 1, 1, 1, -1, 6), (3, 129, 16, 1, -2, 7),
                                                 (8, 70, 33, 129, -1, 8), (16, 20, 17, 130, -1, 9),
                                                 (8, 9, 40, 5, -2, 10), (16, 129, 3, 2, -2, 11)])
def test_mdgemm_end_to_end(L, m, k, n, cutoff, seed):
    print(f"[case] mdgemm L={L} {m}x{k}x{n} cutoff={cutoff}", flush=True)
    A, B = _operands(L, m, k, n, seed, base="normal" if seed % 2 else "uniform", row_exp=15, col_exp=15)
    S = exact.default_slices(L)
    T = S - 1 if cutoff == -1 else 2 * S - 2
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B), cutoff=cutoff))
    ref = pipeline.full_reference(A, B, S, T)
    assert np.array_equal(C, ref["C"])
    pick = random.Random(seed)
    for _ in range(20):
        i, j = pick.randrange(m), pick.randrange(n)
        assert exact.is_nonoverlapping(C[:, i, j])


def test_mdgemm_plain_entry_point_and_tolerance():
    print("[case] mdgemm plain c0", flush=True)
    A, B = workloads.make_workload("c0")
    C = _host(md.mdgemm(_gpu(A), _gpu(B)))  # default: T = S - 1, default stream, library workspace
    ref = pipeline.full_reference(A, B, 8, 7)
    assert np.array_equal(C, ref["C"])
    worst = 0.0
    for i in range(0, 64, 9):
        for j in range(0, 64, 7):
            want, mag = exact.exact_product(A, B, i, j)
            ratio = abs(exact.value(C[:, i, j]) - want) / exact.tolerance(64, 2, mag)
            worst = max(worst, float(ratio))
    assert worst <= 1.0, worst
    md.mdgemm_release()


def test_mdgemm_zero_lines_and_k0():
    print("[case] mdgemm zero rows/cols and k=0", flush=True)
    A, B = _operands(2, 50, 30, 40, 11)
    A[:, 3, :] = 0.0
    B[:, :, 5] = 0.0
    A[:, 7, 4] = 0.0
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B)))
    ref = pipeline.full_reference(A, B, 8, 7)
    assert np.array_equal(C, ref["C"])
    assert (C[:, 3, :] == 0).all() and (C[:, :, 5] == 0).all()
    assert not np.signbit(C[:, 3, :]).any()
    # k = 0: C = +0.0
    Z = md.mdgemm_ex(torch.empty((2, 5, 0), dtype=torch.float64, device=DEV),
                     torch.empty((2, 0, 6), dtype=torch.float64, device=DEV),
                     C=torch.full((2, 5, 6), 3.0, dtype=torch.float64, device=DEV))
    z = _host(Z)
    assert (z == 0).all() and not np.signbit(z).any()


def test_mdgemm_tiny_and_huge_magnitudes():
    print("[case] mdgemm extreme exponents", flush=True)
    A, B = _operands(2, 20, 24, 18, 12)
    A[:, :5] *= 2.0**-600  # rows far below 1
    B[:, :, :4] *= 2.0**500  # columns far above 1
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B)))
    ref = pipeline.full_reference(A, B, 8, 7)
    assert np.array_equal(C, ref["C"])


def test_mdgemm_caller_workspace_and_stream():
    print("[case] mdgemm caller workspace, side stream, stage timing", flush=True)
    A, B = _operands(3, 100, 64, 90, 13, base="normal")
    need = md.mdgemm_workspace_bytes(100, 90, 64, 3)
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    s = torch.cuda.Stream()
    Ag, Bg = _gpu(A), _gpu(B)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        C = md.mdgemm_ex(Ag, Bg, workspace=ws, flags=md.MDGEMM_TIME_STAGES)
    s.synchronize()
    times = md.mdgemm_stage_times()
    assert len(times) == 4 and all(t >= 0 for t in times)
    ref = pipeline.full_reference(A, B, 12, 11)
    assert np.array_equal(C.cpu().numpy(), ref["C"])
    with pytest.raises(md.MdgemmError) as ei:
        md.mdgemm_ex(Ag, Bg, workspace=ws[: need - 1])
    assert ei.value.status == md.MDGEMM_EWORKSPACE


def test_mdgemm_check_finite():
    print("[case] mdgemm nonfinite check", flush=True)
    A, B = _operands(2, 8, 8, 8, 14)
    A[1, 2, 3] = np.inf
    with pytest.raises(md.MdgemmError) as ei:
        md.mdgemm_ex(_gpu(A), _gpu(B), flags=md.MDGEMM_CHECK_FINITE)
    assert ei.value.status == md.MDGEMM_ENONFINITE
    A[1, 2, 3] = 0.0
    C = md.mdgemm_ex(_gpu(A), _gpu(B), flags=md.MDGEMM_CHECK_FINITE | md.MDGEMM_SYNC)
    assert np.array_equal(C.cpu().numpy(), pipeline.full_reference(A, B, 8, 7)["C"])


def test_mdgemm_library_workspace_grows():
    print("[case] mdgemm library workspace: small then larger product", flush=True)
    md.mdgemm_release()
    for (m, k, n, seed) in [(20, 16, 12, 21), (150, 70, 140, 22), (40, 33, 30, 23)]:
        A, B = _operands(2, m, k, n, seed)
        C = _host(md.mdgemm(_gpu(A), _gpu(B)))
        assert np.array_equal(C, pipeline.full_reference(A, B, 8, 7)["C"]), (m, k, n)
    md.mdgemm_release()


def _library_ex(A, B, C, stream, flags=md.MDGEMM_STAGED):
    """mdgemm_ex through the C ABI with the library-owned workspace on `stream`
    (the staged kernels: the fused small-product kernel uses no workspace)."""
    o = md.make_opts(stream=stream, flags=flags)
    o.workspace, o.workspace_bytes = None, 0
    L, m, k = A.shape
    n = B.shape[2]
    return md.lib().mdgemm_ex(m, n, k, L, A.data_ptr(), B.data_ptr(), C.data_ptr(), ctypes.byref(o))


def test_mdgemm_library_workspace_across_streams():
    # Products on two streams at once share the library buffer; they are ordered
    # on the GPU, so each one still computes its own product.
    print("[case] library workspace shared by two streams", flush=True)
    md.mdgemm_release()
    cases = [_operands(2, 130, 100, 140, 40 + i, base="normal", row_exp=4, col_exp=4) for i in range(4)]
    dev = [(_gpu(A), _gpu(B)) for A, B in cases]
    outs = [torch.full((2, 130, 140), 3.0, dtype=torch.float64, device=DEV) for _ in cases]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for i, ((Ag, Bg), C) in enumerate(zip(dev, outs)):
        assert _library_ex(Ag, Bg, C, streams[i % 2]) == md.MDGEMM_OK
    torch.cuda.synchronize()
    for (A, B), C in zip(cases, outs):
        assert np.array_equal(C.cpu().numpy(), pipeline.full_reference(A, B, 8, 7)["C"])
    md.mdgemm_release()


@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")  # the refused call leaves the graph empty
def test_mdgemm_library_workspace_refuses_capture():
    print("[case] capture with the library workspace is refused", flush=True)
    A, B = _operands(2, 40, 30, 50, 45)
    Ag, Bg = _gpu(A), _gpu(B)
    C = torch.empty((2, 40, 50), dtype=torch.float64, device=DEV)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        st = _library_ex(Ag, Bg, C, s)
    assert st == md.MDGEMM_EINVAL
    # outside capture the same call works
    assert _library_ex(Ag, Bg, C, s) == md.MDGEMM_OK
    torch.cuda.synchronize()
    assert np.array_equal(C.cpu().numpy(), pipeline.full_reference(A, B, 8, 7)["C"])


def test_mdgemm_graph_capture_replays():
    # The product uses no memsets, no events (without MDGEMM_TIME_STAGES) and no
    # synchronization (without CHECK_FINITE / SYNC), so it can be captured into a
    # HIP graph; every replay must equal the eager result.
    print("[case] mdgemm captured in a HIP graph", flush=True)
    A, B = _operands(3, 130, 48, 140, 24, base="normal", row_exp=5, col_exp=5)
    Ag, Bg = _gpu(A), _gpu(B)
    ws = torch.empty(md.mdgemm_workspace_bytes(130, 140, 48, 3), dtype=torch.uint8, device=DEV)
    eager = md.mdgemm_ex(Ag, Bg, workspace=ws)
    torch.cuda.synchronize()
    want = eager.cpu().numpy()
    assert np.array_equal(want, pipeline.full_reference(A, B, 12, 11)["C"])
    C = torch.empty_like(eager)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        md.mdgemm_ex(Ag, Bg, C, workspace=ws)  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        md.mdgemm_ex(Ag, Bg, C, workspace=ws)
    for r in range(4):
        C.fill_(7.0)
        md.mdgemm_ex(Ag, Bg, workspace=ws)  # eager work between replays
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(C.cpu().numpy(), want), r


@pytest.mark.parametrize("L,m,k,n,seed", [(2, 130, 64, 129, 20), (4, 33, 64, 45, 21), (3, 40, 100, 70, 22),
                                          (16, 20, 17, 130, 23), (8, 9, 40, 5, 24), (1, 65, 200, 17, 25),
                                          (2, 1, 1, 1, 26)])
def test_mdgemm_adaptive_width_end_to_end(L, m, k, n, seed):
    auto = md.MDGEMM_SLICE_BITS_AUTO
    w, S, T = md.mdgemm_plan(m, n, k, L, slice_bits=auto)
    assert (w, S) == exact.adaptive_width(L, k) and T == S - 1
    print(f"[case] mdgemm auto width L={L} {m}x{k}x{n}: w={w} S={S}", flush=True)
    A, B = _operands(L, m, k, n, seed, base="normal", row_exp=15, col_exp=15)
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B), slice_bits=auto))
    ref = pipeline.full_reference(A, B, S, T, w)
    assert np.array_equal(C, ref["C"])
    for i in range(0, m, max(1, m // 3)):
        for j in range(0, n, max(1, n // 3)):
            want, mag = exact.exact_product(A, B, i, j)
            err = abs(exact.value(C[:, i, j]) - want)
            assert err <= exact.tolerance(k, L, mag), (i, j)


@pytest.mark.parametrize("L,bits,slices,cutoff", [(2, 17, 0, -2), (3, 22, 8, -1), (2, 20, 6, 3), (4, 13, 12, -1)])
def test_mdgemm_explicit_width_end_to_end(L, bits, slices, cutoff):
    m, k, n = 70, 20, 65
    w, S, T = md.mdgemm_plan(m, n, k, L, slice_bits=bits, slices=slices, cutoff=cutoff)
    print(f"[case] mdgemm width {w} S={S} T={T} L={L}", flush=True)
    A, B = _operands(L, m, k, n, 30 + bits, base="normal", row_exp=5, col_exp=5)
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B), slice_bits=bits, slices=slices, cutoff=cutoff))
    assert np.array_equal(C, pipeline.full_reference(A, B, S, T, w)["C"])


@pytest.mark.parametrize("L,m,k,n,range_bits,auto", [(2, 70, 48, 65, 60, False), (2, 33, 100, 129, 60, True),
                                                     (3, 20, 40, 17, 30, False), (4, 17, 33, 9, 26, True),
                                                     (8, 9, 20, 8, 40, False)])
def test_mdgemm_range_balancing_end_to_end(L, m, k, n, range_bits, auto):
    opts = {"range_bits": range_bits}
    if auto:
        opts["slice_bits"] = md.MDGEMM_SLICE_BITS_AUTO
    w, S, T = md.mdgemm_plan(m, n, k, L, **opts)
    assert (w, S, T) == exact.plan(L, k, **opts)
    print(f"[case] mdgemm range {range_bits} L={L} {m}x{k}x{n}: w={w} S={S} T={T}", flush=True)
    wl = workloads.WORKLOADS["c7"]
    rng = np.random.default_rng(L + k + range_bits)
    A = workloads.make_operand(rng, L, m, k, "normal")
    B = workloads.make_operand(rng, L, k, n, "normal")
    e = rng.integers(0, range_bits + 1, k)  # the wide-range recipe of workload c7
    A *= np.ldexp(1.0, -e)[None, None, :]
    B *= np.ldexp(1.0, e - range_bits)[None, :, None]
    assert wl.inner_exp == 60
    C = _host(md.mdgemm_ex(_gpu(A), _gpu(B), **opts))
    ref = pipeline.full_reference(A, B, S, T, w)
    assert np.array_equal(C, ref["C"])
    for i in range(0, m, max(1, m // 3)):
        for j in range(0, n, max(1, n // 3)):
            want, mag = exact.exact_product(A, B, i, j)
            err = abs(exact.value(C[:, i, j]) - want)
            bound = exact.tolerance(k, L, mag)
            assert err <= bound, (i, j, float(err / bound))
