"""Pins of the CPU oracle against what the paper and mathematics fix.

None of these checks retypes the oracle's own formula: each compares it with a
value the paper prints, a closed form, an independent formulation (the
materialized rewritten product, schoolbook digit extraction, exact rational
arithmetic) or an invariant.  Section numbers refer to Chen and Verschelde,
"Multiple Double Arithmetic on NVIDIA Tensor Cores".
"""

import math
import os
import random
from fractions import Fraction

import numpy as np
import pytest

from checks import nonoverlap_all
from oracle import coracle, exact, pipeline
from paper_2607_06881_amd import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return [ln.rstrip("\n") for ln in fh if ln.strip() and not ln.startswith("#")]


# --------------------------------------------------------------------------
# section 2: the worked 52-bit -> 4 x 13-bit split
# --------------------------------------------------------------------------

def _worked_example():
    fields, quarters = {}, {}
    for ln in _golden_lines("worked_split.txt"):
        key, rest = [s.strip() for s in ln.split(":", 1)]
        if key.startswith("f"):
            fields[key] = int(rest.replace(" ", ""), 2)
        else:
            parts = rest.split()
            bits = "".join(parts[:4])  # leading bit and 12 more significand bits
            quarters[key] = (int(bits, 2), int(parts[-1]))
    return fields, quarters


def test_worked_example_fields_partition_f():
    fields, _ = _worked_example()
    f = fields["f"]
    assert f.bit_length() == 52
    parts = [fields[f"f{s}"] for s in range(4)]
    assert sum(parts) == f
    for a in range(4):
        for b in range(a + 1, 4):
            assert parts[a] & parts[b] == 0


@pytest.mark.parametrize("impl", ["python", "c"])
def test_worked_example_split(impl):
    fields, quarters = _worked_example()
    x = fields["f"] * 2.0**-52  # the double whose 52 fraction bits are f, exponent 0
    E = 0
    assert exact.frexp_exp(x) == E
    if impl == "python":
        digits, R = exact.split_element([x], E, 4)
        assert R == 0
    else:
        X = np.array([x]).reshape(1, 1, 1)
        assert coracle.exponents(X[0], 0)[0] == E
        digits = [int(d) for d in coracle.split(X, np.array([E]), 4, 0).ravel()]
    for s in range(4):
        # digit s is the field f_s moved down to an integer
        assert digits[s] << (13 * (3 - s)) == fields[f"f{s}"]
        # and equals the printed quarter, whose exponent is 0, -13, -26, -39
        q_bits, q_exp = quarters[f"x{s}"]
        assert digits[s] == q_bits
        assert exact.frexp_exp(digits[s] * 2.0 ** (-13 * (s + 1))) == q_exp


def test_truncation_not_rounding_matches_worked_example():
    # Reading: the parts are truncated bit fields.  Rounding the first part to
    # nearest would change f0 because the 14th bit of f is 1.
    fields, _ = _worked_example()
    f = fields["f"]
    assert (f >> (52 - 14)) & 1 == 1
    rounded_f0 = (f + (1 << (38 - 1))) >> 39
    assert rounded_f0 != fields["f0"] >> 39


# --------------------------------------------------------------------------
# sections 2-3: borrow / opposite-sign limbs, invariants, brute force
# --------------------------------------------------------------------------

def _parse_borrow():
    cases = []
    for ln in _golden_lines("borrow_split.txt"):
        limbs, E, S, digits = [s.strip() for s in ln.split("|")]
        cases.append(([float.fromhex(t) for t in limbs.split()], int(E), int(S), [int(t) for t in digits.split()]))
    return cases


@pytest.mark.parametrize("case", _parse_borrow())
def test_borrow_vectors(case):
    limbs, E, S, want = case
    d, R = exact.split_element(limbs, E, S)
    assert d == want and R == 0
    X = np.array(limbs).reshape(len(limbs), 1, 1)
    dc = coracle.split(X, np.array([E]), S, 0).ravel().astype(np.int64).tolist()
    assert dc == want


def _schoolbook_digits(limbs, E, S, base=8192):
    """Base-2^13 (or `base`) digits by repeated multiplication (an independent algorithm)."""
    v = sum(Fraction(x) for x in limbs)
    sign = 1 if v >= 0 else -1
    r = abs(v) / Fraction(2) ** E
    out = []
    for _ in range(S):
        r *= base
        d = math.floor(r)
        out.append(sign * d if d else 0)
        r -= d
    return out


def _random_md(rng, L, spread=60):
    """A random normalized multiple double with random gaps between limbs."""
    x0 = rng.choice([-1, 1]) * rng.uniform(0.5, 1.0) * 2.0 ** rng.randint(-spread, spread)
    limbs = [x0]
    for _ in range(1, L):
        prev = limbs[-1]
        if prev == 0.0 or rng.random() < 0.1:
            limbs.append(0.0)
            continue
        half_ulp = math.ulp(prev) / 2
        kind = rng.random()
        if kind < 0.15:
            y = rng.choice([-1, 1]) * half_ulp  # extreme allowed magnitude
        elif kind < 0.3:
            y = rng.choice([-1, 1]) * half_ulp * 2.0 ** -rng.randint(1, 30)  # gap
        else:
            y = rng.uniform(-1, 1) * half_ulp
        limbs.append(y)
    return limbs


@pytest.mark.parametrize("L", [1, 2, 3, 4, 8, 16])
def test_split_invariants_and_brute_force(L):
    rng = random.Random(1234 + L)
    for trial in range(300 if L <= 4 else 80):
        limbs = _random_md(rng, L)
        assert exact.is_nonoverlapping(limbs)
        e0 = exact.frexp_exp(limbs[0])
        E = e0 + rng.choice([0, 0, 0, 1, 3, 13, 40])
        S = rng.choice([1, 2, 3, 4, 4 * L, min(4 * L + 3, 64)])
        d, R = exact.split_element(limbs, E, S)
        v = exact.value(limbs)
        u = exact.grid_unit(E, S - 1)
        # slices plus residual give back the value exactly
        assert sum(di * exact.grid_unit(E, s) for s, di in enumerate(d)) + R == v
        assert abs(R) < u and R * v >= 0
        assert all(0 <= abs(di) <= 8191 and di * v >= 0 for di in d)
        assert d == _schoolbook_digits(limbs, E, S)
        X = np.array(limbs).reshape(L, 1, 1)
        dc = coracle.split(X, np.array([E]), S, 0).ravel().astype(np.int64).tolist()
        assert dc == d, (limbs, E, S)


@pytest.mark.parametrize("L", [1, 2, 4, 8, 16])
def test_split_wide_digits(L):
    # The adaptive width cuts the same value into fewer, wider fields: the same
    # invariants, and the digits of repeated multiplication by 2^w.
    rng = random.Random(777 + L)
    for trial in range(150 if L <= 4 else 40):
        limbs = _random_md(rng, L)
        E = exact.frexp_exp(limbs[0]) + rng.choice([0, 0, 1, 5])
        bits = rng.randint(14, 26)
        S = rng.randint(1, min(64, 844 // bits))
        d, R = exact.split_element(limbs, E, S, bits)
        v = exact.value(limbs)
        assert sum(di * exact.grid_unit(E, s, bits) for s, di in enumerate(d)) + R == v
        assert abs(R) < exact.grid_unit(E, S - 1, bits) and R * v >= 0
        assert all(abs(di) < 2**bits and di * v >= 0 for di in d)
        assert d == _schoolbook_digits(limbs, E, S, 2**bits), (limbs, E, S, bits)
        X = np.array(limbs).reshape(L, 1, 1)
        assert coracle.split(X, np.array([E]), S, 0, bits).ravel().astype(np.int64).tolist() == d


def test_split_full_coverage_has_zero_residual():
    # With enough slices to reach the lowest set bit, the split is exact (R == 0).
    rng = random.Random(7)
    for _ in range(200):
        L = rng.randint(1, 4)
        limbs = _random_md(rng, L, spread=5)
        E = exact.frexp_exp(limbs[0])
        lows = [exact.frexp_exp(x) - 53 for x in limbs if x != 0.0]
        S_full = math.ceil((E - min(lows)) / 13)
        _, R = exact.split_element(limbs, E, S_full)
        assert R == 0


def test_split_subnormal_and_zero():
    tiny = [5 * 2.0**-1074, 0.0]
    E = exact.frexp_exp(tiny[0])
    assert E == -1071
    d, R = exact.split_element(tiny, E, 1)
    assert d == [5 << 10] and R == 0
    X = np.array(tiny).reshape(2, 1, 1)
    assert coracle.split(X, np.array([E]), 1, 0).ravel().tolist() == [5 << 10]
    assert exact.split_element([0.0, 0.0], 0, 3) == ([0, 0, 0], 0)
    with pytest.raises(ValueError):
        exact.split_element([1.0], 0, 4)  # |x| = 2^E is not below the grid top


def test_exponents_against_numpy_frexp():
    rng = np.random.default_rng(5)
    X = rng.standard_normal((37, 53)) * np.ldexp(1.0, rng.integers(-300, 300, (37, 53)))
    X[3, :] = 0.0
    X[:, 7] = 0.0
    X[5, 9] = 3 * 2.0**-1074  # subnormal
    for axis in (0, 1):
        Ec = coracle.exponents(X, axis)
        _, ex = np.frexp(X)
        masked = np.where(X != 0, ex, np.iinfo(np.int32).min)
        want = masked.max(axis=1 - axis)
        want = np.where(want == np.iinfo(np.int32).min, 0, want)
        assert np.array_equal(Ec, want)
        assert np.array_equal(Ec, exact.line_exponents(X, axis))
    # every element lies below 2^E of its row
    Er = coracle.exponents(X, 0)
    assert np.all(np.abs(X) < np.ldexp(1.0, Er[:, None]))


# --------------------------------------------------------------------------
# section 2: equation (3), the rewritten product and the bound (NBound)
# --------------------------------------------------------------------------

def test_eq3_level_structure():
    for ln in _golden_lines("eq3_levels.txt"):
        t, pairs = ln.split(":")
        want = sorted(tuple(int(v) for v in p.split(",")) for p in pairs.split())
        assert sorted(exact.pairs_of_level(int(t), 4)) == want


def test_rewritten_product_matches_levels():
    # The double-double rewrite: Abar = [A_0 ... A_7] and Bbar block upper
    # triangular Toeplitz with B_0 on the diagonal; block column l of Abar Bbar is
    # the level-l product, and the 36 blocks on or above the diagonal are the pairs.
    rng = np.random.default_rng(11)
    S, m, k, n = 8, 5, 6, 4
    DA = rng.integers(-8191, 8192, (S, m, k))
    DB = rng.integers(-8191, 8192, (S, k, n))
    Abar = np.concatenate([DA[p] for p in range(S)], axis=1)  # m x S k
    Bbar = np.zeros((S * k, S * n), dtype=np.int64)
    for r in range(S):
        for c in range(r, S):
            Bbar[r * k:(r + 1) * k, c * n:(c + 1) * n] = DB[c - r]
    Cbar = Abar.astype(object) @ Bbar.astype(object)
    T = S - 1
    assert sum(len(exact.pairs_of_level(t, S)) for t in range(T + 1)) == 36
    G = coracle.levels(DA.astype(np.float64), DB.astype(np.float64), T)
    Gpy = exact.level_products(DA, DB, T)
    for l in range(S):
        blk = np.array(Cbar[:, l * n:(l + 1) * n], dtype=np.int64)
        assert np.array_equal(blk, G[l])
        assert np.array_equal(blk, np.array(Gpy[l], dtype=np.int64))


def test_nbound_value():
    # N (2^0 + ... + 2^25) <= 2^52 gives N <= 67,108,865 (section 2).
    B = sum(2**i for i in range(26))
    assert B == 2**26 - 1
    assert 2**52 // B == 67108865
    assert 67108865 * B <= 2**52 < 67108866 * B


def test_levels_against_float_matmul_and_per_pair():
    rng = np.random.default_rng(3)
    S, T, m, k, n = 6, 7, 9, 33, 7
    DA = rng.integers(-8191, 8192, (S, m, k)).astype(np.float64)
    DB = rng.integers(-8191, 8192, (S, k, n)).astype(np.float64)
    G = coracle.levels(DA, DB, T)
    P = coracle.levels(DA, DB, T, per_pair=True)
    for t in range(T + 1):
        acc = np.zeros((m, n))
        for p, q in exact.pairs_of_level(t, S):
            prod = DA[p] @ DB[q]  # float64 BLAS: exact, every partial sum < 2^53
            assert np.array_equal(P[p, q], prod.astype(np.int64))
            acc += prod
        assert np.array_equal(G[t], acc.astype(np.int64))


@pytest.mark.parametrize("S,T,m,k,n", [(8, 7, 37, 64, 29), (12, 11, 16, 32, 40), (5, 8, 3, 1, 2), (4, 0, 6, 9, 5)])
def test_levels_rewritten_matches_int64_and_python_ints(S, T, m, k, n):
    # The rewritten-product form of the levels (one float64 matrix product per
    # level) against the int64 loops of the C oracle on maximal digits of both
    # signs, and against Python ints on a small corner.
    rng = np.random.default_rng(S * 100 + T)
    DA = rng.choice([-8191.0, 8191.0, -1.0, 0.0, 4096.0], size=(S, m, k))
    DB = rng.choice([-8191.0, 8191.0, 7.0, 0.0, -4095.0], size=(S, k, n))
    G = pipeline.levels_rewritten(DA, DB, T)
    assert G.shape == (T + 1, m, n)
    assert np.array_equal(G.astype(np.int64), coracle.levels(DA, DB, T))
    small = exact.level_products(DA[:, :3, :], DB[:, :, :2], T)
    for t in range(T + 1):
        assert G[t, :3, :2].astype(np.int64).tolist() == small[t]
    # dropping one pair of the last level changes it (the check is not vacuous)
    if T < S:
        assert not np.array_equal(G[T] - DA[0] @ DB[T], G[T])


@pytest.mark.parametrize("bits", [13, 19, 24])
def test_all_pairs_identity_with_truncated_operands(bits):
    # With every pair kept (T = 2S - 2), the weighted levels are exactly the
    # product of the truncated operands: sum_t G_t 2^(EA+EB-2w-wt) = sum_k tr(a) tr(b).
    for seed in range(3):
        rng = np.random.default_rng(seed)
        L, m, k, n = 2, 4, 5, 3
        A = workloads.make_operand(rng, L, m, k, row_exp=9)
        B = workloads.make_operand(rng, L, k, n, col_exp=9)
        S = int(rng.integers(2, 9))
        T = 2 * S - 2
        ref = pipeline.full_reference(A, B, S, T, bits)
        for i in range(m):
            for j in range(n):
                z = exact.accumulate([int(ref["G"][t, i, j]) for t in range(T + 1)],
                                     int(ref["EA"][i]), int(ref["EB"][j]), bits)
                want = Fraction(0)
                for kk in range(k):
                    da, ra = exact.split_element(A[:, i, kk], int(ref["EA"][i]), S, bits)
                    db, rb = exact.split_element(B[:, kk, j], int(ref["EB"][j]), S, bits)
                    want += (exact.value(A[:, i, kk]) - ra) * (exact.value(B[:, kk, j]) - rb)
                assert z == want


# --------------------------------------------------------------------------
# greedy rounding into L limbs
# --------------------------------------------------------------------------

def test_round_to_limbs_hand_cases():
    u = Fraction(2) ** -52  # ulp(1)
    # exactly representable
    assert exact.round_to_limbs(Fraction(3, 4), 2) == [0.75, 0.0]
    # a half-ulp tail stays in the second limb (tie at the first limb goes to even 1.0)
    assert exact.round_to_limbs(1 + u / 2, 2) == [1.0, 2.0**-53]
    # 1 + 3/2 ulp: tie between 1+u and 1+2u, even is 1 + 2u; remainder -u/2
    assert exact.round_to_limbs(1 + 3 * u / 2, 2) == [1.0 + 2.0**-51, -(2.0**-53)]
    # a tail below half an ulp rounds down
    z = 1 + u / 2 - Fraction(1, 2**200)
    c = exact.round_to_limbs(z, 3)
    assert c[0] == 1.0 and c[1] == 2.0**-53 and c[2] == -(2.0**-200)
    assert exact.round_to_limbs(Fraction(0), 3) == [0.0, 0.0, 0.0]


def test_round_to_limbs_properties():
    rng = random.Random(99)
    for _ in range(500):
        L = rng.randint(1, 4)
        z = Fraction(rng.randint(-2**300, 2**300), 2 ** rng.randint(0, 400))
        c = exact.round_to_limbs(z, L)
        assert exact.is_nonoverlapping(c)
        err = abs(z - sum(Fraction(x) for x in c))
        if c[-1] != 0.0:
            assert err <= Fraction(math.ulp(c[-1])) / 2
        else:
            assert err == 0


def test_default_digit_count_closed_forms():
    # four 13-bit quarters per limb up to quad doubles (52 L >= 53 L - 4 bits);
    # beyond, the 53 L - 4 bits of the tolerance in whole digits plus one
    assert [exact.default_slices(L) for L in (1, 2, 3, 4)] == [4, 8, 12, 16]
    assert [52 * L >= 53 * L - 4 for L in (1, 2, 3, 4, 5)] == [True, True, True, True, False]
    assert exact.default_slices(5) == 22 and exact.default_slices(8) == 34 and exact.default_slices(16) == 66
    for L in range(5, 17):
        S = exact.default_slices(L)
        assert 13 * (S - 2) < 53 * L - 4 <= 13 * (S - 1)


@pytest.mark.parametrize("L,k", [(5, 128), (8, 128), (16, 64)])
def test_default_digit_count_meets_the_tolerance_beyond_four_limbs(L, k):
    # The sliced chain with the default digit count meets 4 k 2^-(53L-4) (|A||B|)
    # on N(0,1) octo/hexa-double data (the shapes' k of the od/hd workloads),
    # while four digits per limb miss it for octo and hexa doubles.
    rng = np.random.default_rng(L)
    A = workloads.make_operand(rng, L, 6, k, "normal")
    B = workloads.make_operand(rng, L, k, 5, "normal")
    worst = {}
    for S in (4 * L, exact.default_slices(L)):
        C = pipeline.full_reference(A, B, S, S - 1)["C"]
        r = 0.0
        for i in range(6):
            for j in range(5):
                want, mag = exact.exact_product(A, B, i, j)
                r = max(r, float(abs(exact.value(C[:, i, j]) - want) / exact.tolerance(k, L, mag)))
        worst[S] = r
    assert worst[exact.default_slices(L)] < 1e-3
    if L >= 8:
        assert worst[4 * L] > 1.0


@pytest.mark.parametrize("x0", [1.0, 1.5, -0.75, 3.0 * 2.0**-600, -(2.0**900) * 1.125, 2.0**-1000 * 1.25])
def test_nonoverlap_checkers_accept_the_boundary_and_reject_overlap(x0):
    """Both nonoverlap checkers (the oracle's per element and the tests' whole-array
    one) take section 1's nonoverlapping in the half-ulp sense.  The boundary
    |x1| = ulp(x0)/2 is accepted; one ulp of x1 beyond it, |x1| = ulp(x0)/2 +
    ulp(x1), is rejected, which a checker loosened to a whole ulp would accept;
    a nonzero limb after a zero limb is rejected, which a checker without the
    zero rule would accept."""
    h = 0.5 * math.ulp(x0)
    over = h + math.ulp(h)
    assert Fraction(over) - Fraction(h) == Fraction(math.ulp(h)) and over < math.ulp(x0)
    accepted = [[x0, h], [x0, -h], [x0, h, 0.5 * math.ulp(h)], [x0, 0.0, 0.0], [0.0, 0.0, 0.0]]
    rejected = [[x0, over], [x0, -over], [x0, h, 0.5 * math.ulp(h) + math.ulp(0.5 * math.ulp(h))],
                [0.0, h], [x0, 0.0, 2.0**-1074], [0.0, 0.0, -x0]]
    for limbs in accepted:
        assert exact.is_nonoverlapping(limbs), limbs
        assert nonoverlap_all(np.array(limbs)[:, None]), limbs
    for limbs in rejected:
        assert not exact.is_nonoverlapping(limbs), limbs
        assert not nonoverlap_all(np.array(limbs)[:, None]), limbs
    # the array checker rejects a whole array when one element overlaps
    many = np.array([[x0, h]] * 5 + [[x0, over]] + [[x0, -h]] * 3).T.reshape(2, 3, 3)
    assert not nonoverlap_all(many)
    assert nonoverlap_all(np.array([[x0, h]] * 9).T.reshape(2, 3, 3))


# --------------------------------------------------------------------------
# error-free transformations and classic arithmetic (section 1, section 4)
# --------------------------------------------------------------------------

def _rand_doubles(rng, n):
    out = []
    for _ in range(n):
        kind = rng.random()
        if kind < 0.1:
            out.append(rng.choice([0.0, -0.0, 1.0, -1.0, 2.0**-1074, -(2.0**-1022)]))
        else:
            out.append(rng.uniform(-1, 1) * 2.0 ** rng.randint(-200, 200))
    return np.array(out)


def test_eft_exactness():
    rng = random.Random(5)
    a, b = _rand_doubles(rng, 2000), _rand_doubles(rng, 2000)
    s, e = coracle.two_sum(a, b)
    for x, y, sx, ex in zip(a, b, s, e):
        assert Fraction(sx) + Fraction(ex) == Fraction(x) + Fraction(y)
        assert sx == x + y
    p, e = coracle.two_prod(a, b)
    checked = 0
    for x, y, px, ex in zip(a, b, p, e):
        exact_xy = Fraction(x) * Fraction(y)
        if exact_xy != 0 and abs(exact_xy) < Fraction(2) ** (-1022 + 53):
            continue  # the error term of an underflowing product is not representable
        assert Fraction(px) + Fraction(ex) == exact_xy
        checked += 1
    assert checked > 1500
    # FastTwoSum is exact when |a| >= |b|
    big = np.where(np.abs(a) >= np.abs(b), a, b)
    small = np.where(np.abs(a) >= np.abs(b), b, a)
    s, e = coracle.fast_two_sum(big, small)
    for x, y, sx, ex in zip(big, small, s, e):
        assert Fraction(sx) + Fraction(ex) == Fraction(x) + Fraction(y)


def _rand_md_array(rng, L, n):
    return np.array([_random_md(rng, L, spread=20) for _ in range(n)]).T.copy()


@pytest.mark.parametrize("L", [1, 2, 3, 4, 8, 16])
def test_md_fma_relative_error(L):
    rng = random.Random(40 + L)
    n = 400 if L <= 4 else 60
    acc, a, b = _rand_md_array(rng, L, n), _rand_md_array(rng, L, n), _rand_md_array(rng, L, n)
    out = coracle.md_fma(acc, a, b)
    worst = 0.0
    for e in range(n):
        va, vb, vc = exact.value(a[:, e]), exact.value(b[:, e]), exact.value(acc[:, e])
        want = vc + va * vb
        got = exact.value(out[:, e])
        scale = abs(vc) + abs(va * vb)
        if scale:
            worst = max(worst, float(abs(got - want) / scale))
    # one rounding to L limbs plus dropped products of order 2^-53(L+1)
    assert worst <= 8 * 2.0 ** (-52 * L), worst


def test_dd_add_mul_relative_error():
    rng = random.Random(77)
    n = 1000
    a, b = _rand_md_array(rng, 2, n), _rand_md_array(rng, 2, n)
    s, p = coracle.dd_add(a, b), coracle.dd_mul(a, b)
    ws = wp = 0.0
    for e in range(n):
        va, vb = exact.value(a[:, e]), exact.value(b[:, e])
        if va + vb != 0:
            ws = max(ws, float(abs(exact.value(s[:, e]) - (va + vb)) / (abs(va) + abs(vb))))
        if va * vb != 0:
            wp = max(wp, float(abs(exact.value(p[:, e]) - va * vb) / abs(va * vb)))
    assert ws <= 4 * 2.0**-106 and wp <= 8 * 2.0**-106, (ws, wp)


@pytest.mark.parametrize("L,variant", [(1, 1), (2, 0), (2, 1), (3, 1), (4, 1), (8, 1), (16, 1)])
def test_classic_gemm_within_bound(L, variant):
    rng = np.random.default_rng(20 + L)
    m, k, n = 5, 7, 4
    A = workloads.make_operand(rng, L, m, k, row_exp=6)
    B = workloads.make_operand(rng, L, k, n, col_exp=6)
    C, _ = coracle.classic_gemm(A, B, variant=variant)
    for i in range(m):
        for j in range(n):
            want, mag = exact.exact_product(A, B, i, j)
            assert abs(exact.value(C[:, i, j]) - want) <= exact.tolerance(k, L, mag)


def test_classic_gemm_row_range_and_threads():
    rng = np.random.default_rng(8)
    A = workloads.make_operand(rng, 2, 6, 9)
    B = workloads.make_operand(rng, 2, 9, 5)
    full, used = coracle.classic_gemm(A, B, nthreads=2)
    part, _ = coracle.classic_gemm(A, B, rows=(2, 4), nthreads=2)
    assert used >= 1
    assert np.array_equal(part[:, 2:4], full[:, 2:4]) and not part[:, :2].any()


# --------------------------------------------------------------------------
# the sliced chain against the exact product (the componentwise tolerance)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("L,S,T", [(1, 4, 3), (2, 8, 14), (2, 8, 7), (3, 12, 11), (4, 16, 15)])
def test_sliced_chain_within_tolerance(L, S, T):
    # The bound 4 k 2^-(53L-4) (|A||B|) leaves room for the bits an element loses
    # below its line's shared exponent; k = 64 (the smallest workload) keeps it
    # meaningful.  At k = 9 a quad-double row with N(0,1) entries exceeds it:
    # an inherent limit of one shared exponent per row / column.
    rng = np.random.default_rng(100 + L + T)
    m, k, n = 3, 64, 3
    A = workloads.make_operand(rng, L, m, k, base="normal", row_exp=10)
    B = workloads.make_operand(rng, L, k, n, base="normal", col_exp=10)
    ref = pipeline.full_reference(A, B, S, T)
    for i in range(m):
        for j in range(n):
            got = ref["C"][:, i, j]
            assert exact.is_nonoverlapping(got)
            want, mag = exact.exact_product(A, B, i, j)
            assert abs(exact.value(got) - want) <= exact.tolerance(k, L, mag)


@pytest.mark.parametrize("L,S,T,k", [(2, 8, 7, 64), (4, 16, 15, 40), (3, 12, 20, 9), (8, 32, 31, 24),
                                     (16, 64, 63, 9), (8, 40, 32, 12)])
def test_sliced_chain_within_method_bound(L, S, T, k):
    # The truncation and dropped-pair bound of the sliced product (exact.method_bound)
    # holds for every digit count and cutoff, including octo and hexa doubles with
    # four digits per limb, where the 53 L-bit tolerance cannot.
    rng = np.random.default_rng(300 + L + S + T)
    m, n = 2, 3
    A = workloads.make_operand(rng, L, m, k, base="normal", row_exp=10)
    B = workloads.make_operand(rng, L, k, n, base="normal", col_exp=10)
    ref = pipeline.full_reference(A, B, S, T)
    EA, EB = coracle.exponents(A[0], 0), coracle.exponents(B[0], 1)
    for i in range(m):
        for j in range(n):
            got = ref["C"][:, i, j]
            assert exact.is_nonoverlapping(got)
            want, mag = exact.exact_product(A, B, i, j)
            bound = exact.method_bound(A, B, i, j, S, T, int(EA[i]), int(EB[j]))
            err = abs(exact.value(got) - want)
            assert err <= bound, (i, j, float(err / bound))
            # not vacuous: far below the magnitude, at the scale of 2^-13S per unit of the grid
            assert bound < mag * Fraction(2) ** (-13 * min(S, T + 1) + 30)


@pytest.mark.parametrize("L,k", [(1, 64), (2, 64), (3, 100), (4, 64), (2, 4096)])
def test_adaptive_width_chain_within_tolerance(L, k):
    # Fewer, wider digits at the adaptive width keep at least the digit bits of
    # four 13-bit digits per limb, so the stated tolerance still holds.
    w, S = exact.adaptive_width(L, k)
    assert w * S >= 52 * L and S * k * (2**w - 1) ** 2 < 2**53
    T = S - 1
    rng = np.random.default_rng(400 + L + k)
    m, n = 2, 2
    A = workloads.make_operand(rng, L, m, k, base="normal", row_exp=10)
    B = workloads.make_operand(rng, L, k, n, base="normal", col_exp=10)
    ref = pipeline.full_reference(A, B, S, T, w)
    for i in range(m):
        for j in range(n):
            got = ref["C"][:, i, j]
            assert exact.is_nonoverlapping(got)
            want, mag = exact.exact_product(A, B, i, j)
            err = abs(exact.value(got) - want)
            assert err <= exact.tolerance(k, L, mag), (i, j)
            assert err <= exact.method_bound(A, B, i, j, S, T, int(ref["EA"][i]), int(ref["EB"][j]), w)


def test_adaptive_width_closed_forms():
    # worked by hand from S k (2^w - 1)^2 < 2^53 and S = ceil(52 L / w)
    assert exact.adaptive_width(2, 4096) == (19, 6)   # 21 pairs instead of 36
    assert exact.adaptive_width(4, 1024) == (19, 11)  # 66 instead of 136
    assert exact.adaptive_width(3, 512) == (20, 8)    # 36 instead of 78
    assert exact.adaptive_width(2, 64) == (22, 5)     # 15 instead of 36
    assert exact.adaptive_width(2, 2**26) is None     # 8 k 8191^2 >= 2^53: no width stays exact
    assert exact.adaptive_width(2, 2**22) == (14, 8)  # 8 k (2^14 - 1)^2 < 2^53 <= 7 k (2^15 - 1)^2;
    # at equal pair counts the wider digit is taken


def test_wrong_level_weight_for_wide_digits_is_caught():
    # Planted: 19-bit digits accumulated with the 13-bit weights.
    L, k = 2, 64
    rng = np.random.default_rng(9)
    A = workloads.make_operand(rng, L, 1, k, base="normal")
    B = workloads.make_operand(rng, L, k, 1, base="normal")
    ref = pipeline.full_reference(A, B, 6, 5, 19)
    G = [int(ref["G"][t, 0, 0]) for t in range(6)]
    bad = exact.accumulate(G, int(ref["EA"][0]), int(ref["EB"][0]), 13)
    want, mag = exact.exact_product(A, B, 0, 0)
    assert abs(bad - want) > exact.tolerance(k, L, mag)


def test_line_spread_against_numpy_frexp():
    rng = np.random.default_rng(12)
    X = rng.standard_normal((9, 40)) * np.ldexp(1.0, rng.integers(-50, 50, (9, 40)))
    X[2, :] = 0.0
    X[3, :] = 0.0
    X[3, 5] = 5e-324  # a lone subnormal: its line spans nothing
    X[4, ::3] = 0.0
    for axis in (0, 1):
        lines = X if axis == 0 else X.T
        want = []
        for line in lines:
            nz = line[line != 0]
            _, e = np.frexp(nz)
            want.append(int(e.max() - e.min()) if nz.size else 0)
        assert exact.line_spread(X, axis).tolist() == want


def test_range_balancing_restores_the_tolerance():
    # Rows of A and columns of B spanning 60 bits with balanced products
    # (workload c7's recipe, small): with one grid per line and four digits per
    # limb the small elements lose their bits and the tolerance fails; with 60 bits
    # of range balancing the chain is back within it.
    w = workloads.WORKLOADS["c7"]
    A, B = workloads.make_workload(w, m=3, n=3, k=48, seed=3)
    assert max(exact.line_spread(A[0], 0)) >= 40 and max(exact.line_spread(B[0], 1)) >= 40
    L, k = 2, 48
    plain = pipeline.full_reference(A, B, 8, 7)
    wb, Sb, Tb = exact.plan(L, k, range_bits=60)
    balanced = pipeline.full_reference(A, B, Sb, Tb, wb)
    worst_plain = worst_bal = 0.0
    for i in range(3):
        for j in range(3):
            want, mag = exact.exact_product(A, B, i, j)
            tol = exact.tolerance(k, L, mag)
            worst_plain = max(worst_plain, float(abs(exact.value(plain["C"][:, i, j]) - want) / tol))
            worst_bal = max(worst_bal, float(abs(exact.value(balanced["C"][:, i, j]) - want) / tol))
    assert worst_plain > 1e6  # the shared grid alone misses the tolerance by far
    assert worst_bal <= 1.0
    # the adaptive width with the same balancing stays within it too
    wa, Sa, Ta = exact.plan(L, k, range_bits=60, slice_bits=-1)
    adaptive = pipeline.full_reference(A, B, Sa, Ta, wa)
    for i in range(3):
        for j in range(3):
            want, mag = exact.exact_product(A, B, i, j)
            assert abs(exact.value(adaptive["C"][:, i, j]) - want) <= exact.tolerance(k, L, mag)


# --------------------------------------------------------------------------
# grouped products (section 3: by sign and by exponent class)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("L,m,k,n,seed", [(2, 7, 40, 6, 1), (3, 5, 17, 9, 2), (1, 4, 64, 4, 3)])
def test_sign_groups_sum_to_the_ungrouped_levels(L, m, k, n, seed):
    # A = A+ + A-, B = B+ + B-: the digits of the sign groups add up to the
    # digits of the whole operand, so the four group products give the levels
    # of the ungrouped product exactly (the int64 loops of the C oracle)
    rng = np.random.default_rng(seed)
    A = workloads.make_operand(rng, L, m, k, "normal", row_exp=6)
    B = workloads.make_operand(rng, L, k, n, "normal", col_exp=6)
    S = 4 * L
    EA, EB = pipeline.exponents(A, B)
    DA = pipeline.group_digits(A, EA, S, 0, 1, True)
    DB = pipeline.group_digits(B, EB, S, 1, 1, True)
    assert DA.shape == (2, S, m, k)
    assert np.array_equal(DA[0] + DA[1], coracle.split(A, EA.astype(np.int32), S, 0))
    assert not (DA[0] < 0).any() and not (DA[1] > 0).any()
    G = pipeline.group_levels(DA, DB, S - 1, 1)
    want = coracle.levels(coracle.split(A, EA.astype(np.int32), S, 0), coracle.split(B, EB.astype(np.int32), S, 1),
                          S - 1)
    assert np.array_equal(G.astype(np.int64), want)


@pytest.mark.parametrize("L,S", [(1, 6), (2, 10)])
def test_exponent_classes_are_exact_when_the_digits_cover_every_element(L, S):
    # Elements spread over 39 bits below their line's exponent, 4 classes of 13
    # bits: on its class grid every element has its leading bit within one digit
    # of the top, so S digits of 13 bits hold it exactly (53 L bits + 13), and
    # with every pair kept the grouped product is the exact product, rounded
    # greedily.  A class offset one digit off changes the value.
    rng = np.random.default_rng(L)
    m, k, n = 4, 12, 3
    A = workloads.make_operand(rng, L, m, k, "uniform")
    B = workloads.make_operand(rng, L, k, n, "uniform")
    A *= np.ldexp(1.0, -rng.integers(0, 40, (m, k)))[None]
    B *= np.ldexp(1.0, -rng.integers(0, 40, (k, n)))[None]
    classes, T = 4, 2 * S - 2
    C = pipeline.full_reference_groups(A, B, S, T, classes, False)
    EA, EB = pipeline.exponents(A, B)
    grp = pipeline.element_groups(A[0], EA, 0, classes, False)
    assert set(np.unique(grp)) >= {0, 1, 2}  # several classes in use
    for i in range(m):
        for j in range(n):
            want, _ = exact.exact_product(A, B, i, j)
            assert C[:, i, j].tolist() == exact.round_to_limbs(want, L), (i, j)
    # planted mistake: the levels of every group pair one level too low
    DA = pipeline.group_digits(A, EA, S, 0, classes, False)
    DB = pipeline.group_digits(B, EB, S, 1, classes, False)
    good = pipeline.group_levels(DA, DB, T, classes)
    bad = np.zeros_like(good)
    for g in range(classes):
        for h in range(classes):
            for t in range(T + 1):
                for p, q in exact.pairs_of_level(t, S):
                    bad[min(t + g + h + 1, bad.shape[0] - 1)] += DA[g][p] @ DB[h][q]
    z_good = exact.accumulate([int(good[t, 0, 0]) for t in range(good.shape[0])], int(EA[0]), int(EB[0]))
    z_bad = exact.accumulate([int(bad[t, 0, 0]) for t in range(bad.shape[0])], int(EA[0]), int(EB[0]))
    assert z_good == exact.exact_product(A, B, 0, 0)[0] and z_bad != z_good


def test_exponent_classes_restore_the_tolerance():
    # workload c7's recipe, small: the shared grid misses the tolerance by far,
    # exponent classes over the 60 bits meet it (as range balancing does)
    w = workloads.WORKLOADS["c7"]
    A, B = workloads.make_workload(w, m=3, n=3, k=48, seed=3)
    L, k = 2, 48
    wg, Sg, Tg = exact.plan(L, k, range_bits=60, group_exponent=True)
    assert (wg, Sg, Tg) == (13, 9, 9)
    classes = 1 + -(-60 // 13)
    C = pipeline.full_reference_groups(A, B, Sg, Tg, classes, False)
    Cs = pipeline.full_reference_groups(A, B, Sg, Tg, classes, True)  # with sign groups too: the same limbs
    assert np.array_equal(C, Cs)
    for i in range(3):
        for j in range(3):
            want, mag = exact.exact_product(A, B, i, j)
            assert abs(exact.value(C[:, i, j]) - want) <= exact.tolerance(k, L, mag)
    ref = pipeline.reference_entries_groups(A, B, Sg, Tg, classes, False, [(0, 0), (2, 1)])
    assert ref[(0, 0)]["limbs"] == C[:, 0, 0].tolist() and ref[(2, 1)]["limbs"] == C[:, 2, 1].tolist()


# --------------------------------------------------------------------------
# the downstream application: Householder QR in double-double
# --------------------------------------------------------------------------

def test_qr_oracle_closed_form():
    # x = (3, 4): ||x|| = 5, v_1 = -sigma / (x_1 + mu) = -16 / 8 = -2, so the stored
    # vector is 4 / -2 = -2 and tau = 2 v_1^2 / (sigma + v_1^2) = 8 / 20 = 0.4
    A = np.zeros((2, 2, 1))
    A[0, :, 0] = [3.0, 4.0]
    QR, tau = coracle.qr_dd(A)
    assert QR[:, 0, 0].tolist() == [5.0, 0.0] and QR[:, 1, 0].tolist() == [-2.0, 0.0]
    assert abs(exact.value(tau[:, 0]) - Fraction(2, 5)) < Fraction(1, 2**105)  # 0.4 to double-double precision


def _exact_q(QR, tau):
    """Thin Q as Fractions from the stored vectors and tau (reflections applied to I)."""
    _, m, n = QR.shape
    Q = [[Fraction(int(r == c)) for c in range(n)] for r in range(m)]
    for j in range(n - 1, -1, -1):
        t = exact.value(tau[:, j])
        v = [Fraction(0)] * j + [Fraction(1)] + [exact.value(QR[:, r, j]) for r in range(j + 1, m)]
        for c in range(n):
            w = sum(v[r] * Q[r][c] for r in range(j, m))
            for r in range(j, m):
                Q[r][c] -= t * w * v[r]
    return Q


def test_qr_oracle_exact_residual_and_orthogonality():
    # the oracle's factorization checked in exact rational arithmetic (no
    # double-double on the checking side): A - Q R and Q^T Q - I at the level of
    # double-double rounding, and the oracle's own check agrees with it
    rng = np.random.default_rng(4)
    A = workloads.make_operand(rng, 2, 6, 4, "normal")
    QR, tau = coracle.qr_dd(A)
    Q = _exact_q(QR, tau)
    m, n = 6, 4
    amax = max(abs(exact.value(A[:, r, c])) for r in range(m) for c in range(n))
    res = max(abs(exact.value(A[:, r, c]) - sum(Q[r][l] * exact.value(QR[:, l, c]) for l in range(c + 1)))
              for r in range(m) for c in range(n)) / amax
    orth = max(abs(sum(Q[r][i] * Q[r][c] for r in range(m)) - int(i == c)) for i in range(n) for c in range(n))
    assert res < Fraction(1, 2**100) and orth < Fraction(1, 2**100)
    r2, o2, _ = coracle.qr_dd_check(A, QR, tau)
    assert r2 < 2.0**-100 and o2 < 2.0**-100
    assert all(QR[0, j, j] >= 0.0 for j in range(n))
    # a wrong tau (one part in 2^60) is visible to both checks
    bad = tau.copy()
    bad[1, 1] += bad[0, 1] * 2.0**-60
    Qb = _exact_q(QR, bad)
    orth_b = max(abs(sum(Qb[r][i] * Qb[r][c] for r in range(m)) - int(i == c)) for i in range(n) for c in range(n))
    assert orth_b > Fraction(1, 2**70)
    assert coracle.qr_dd_check(A, QR, bad)[1] > 2.0**-70


def test_qr_oracle_agrees_with_float64_qr():
    # R of the double-double factorization rounded to doubles against LAPACK's
    # float64 QR (numpy), rows' signs normalized to a nonnegative diagonal
    rng = np.random.default_rng(5)
    A = workloads.make_operand(rng, 2, 50, 30, "normal")
    QR, _ = coracle.qr_dd(A)
    R = np.triu(QR[0])[:30]
    Rn = np.linalg.qr(A[0] + A[1])[1]
    Rn *= np.sign(np.diag(Rn))[:, None]
    assert np.abs(R - Rn).max() <= 1e-12 * np.abs(Rn).max()


def test_method_bound_catches_a_dropped_kept_pair():
    # Planted in the oracle's chain: leave out pair (0, T) of the last kept level.
    L, S, T, k = 8, 32, 31, 16
    rng = np.random.default_rng(5)
    A = workloads.make_operand(rng, L, 1, k, base="normal")
    B = workloads.make_operand(rng, L, k, 1, base="normal")
    EA, EB = coracle.exponents(A[0], 0), coracle.exponents(B[0], 1)
    DA, DB = coracle.split(A, EA, S, 0), coracle.split(B, EB, S, 1)
    per = coracle.levels(DA, DB, T, per_pair=True)
    levels = [int(sum(per[p, t - p, 0, 0] for p, q in exact.pairs_of_level(t, S) if not (t == T and p == 0)))
              for t in range(T + 1)]
    bad = exact.round_to_limbs(exact.accumulate(levels, int(EA[0]), int(EB[0])), L)
    want, _ = exact.exact_product(A, B, 0, 0)
    bound = exact.method_bound(A, B, 0, 0, S, T, int(EA[0]), int(EB[0]))
    assert abs(exact.value(bad) - want) > bound


def test_reference_entries_agree_with_full_reference():
    A, B = workloads.make_workload("c0", m=12, n=10, k=16)
    S, T = 8, 14
    full = pipeline.full_reference(A, B, S, T)
    entries = [(0, 0), (3, 7), (11, 9), (5, 2)]
    samp = pipeline.reference_entries(A, B, S, T, entries)
    for (i, j), r in samp.items():
        assert r["limbs"] == full["C"][:, i, j].tolist()
        assert r["levels"] == full["G"][:, i, j].tolist()


# --------------------------------------------------------------------------
# planted mistakes: the pins above must notice them
# --------------------------------------------------------------------------

def test_pins_detect_planted_mistakes():
    fields, quarters = _worked_example()
    x = fields["f"] * 2.0**-52
    # (a) an off-by-one grid exponent breaks the worked example
    d_wrong, _ = exact.split_element([x], 1, 4)
    assert d_wrong[0] != fields["f0"] >> 39
    # (b) a dropped pair breaks the rewritten-product comparison
    rng = np.random.default_rng(1)
    DA = rng.integers(-50, 50, (4, 3, 3))
    DB = rng.integers(-50, 50, (4, 3, 3))
    good = exact.level_products(DA, DB, 3)
    bad3 = sum(np.array(DA[p]) @ np.array(DB[q]) for p, q in exact.pairs_of_level(3, 4)[:-1])
    assert not np.array_equal(np.array(good[3]), bad3)
    # (c) a wrong level weight breaks the truncated-operand identity
    A = workloads.make_operand(np.random.default_rng(2), 2, 2, 3)
    B = workloads.make_operand(np.random.default_rng(3), 2, 3, 2)
    ref = pipeline.full_reference(A, B, 8, 14)
    G = [int(g) for g in ref["G"][:, 0, 0]]
    z = exact.accumulate(G, int(ref["EA"][0]), int(ref["EB"][0]))
    z_bad = exact.accumulate([0] + G[:-1], int(ref["EA"][0]), int(ref["EB"][0]))
    assert z != z_bad
