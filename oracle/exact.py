"""Exact reference arithmetic for the multiple-double product -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module.  It shares no code with the GPU path.

Every function here is the plain mathematical definition written out with
Python integers and ``fractions.Fraction`` (all finite doubles are dyadic
rationals, so every step is exact); it is slow and meant for small inputs or
sampled entries.  Citations refer to Chen and Verschelde, "Multiple Double
Arithmetic on NVIDIA Tensor Cores":

* section 1, definition of a multiple double: an unevaluated sum of
  nonoverlapping doubles -> ``value``;
* section 2, the 52-bit fraction cut into four 13-bit quarters with exponents
  0, -13, -26, -39 (worked example) and the balanced grid -> ``split_element``;
* section 3, balancing: one exponent grid per group of numbers (here one per row
  of A and one per column of B) -> ``line_exponents``;
* section 2, equations (1)-(3) and the rewritten product: level t collects the
  slice pairs with p + q = t -> ``pairs_of_level`` and ``level_products``;
* section 2, steps 4-5 of the overview: the parts of the product are extracted
  and added into a multiple double -> ``accumulate`` and ``round_to_limbs``.

The rounding of the exact sum into L limbs is greedy round-to-nearest-even:
c_0 = RN(Z), c_l = RN(Z - c_0 - ... - c_{l-1}).  CPython's ``float(Fraction)``
is correctly rounded (an integer true division), so RN is that conversion.
"""

from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

SLICE_BITS = 13
DIGIT_MAX = (1 << SLICE_BITS) - 1  # 8191


# --------------------------------------------------------------------------
# values and exponents
# --------------------------------------------------------------------------

def value(limbs) -> Fraction:
    """Exact value of a multiple double: the sum of its limbs (section 1)."""
    return sum((Fraction(float(x)) for x in limbs), Fraction(0))


def frexp_exp(x: float) -> int:
    """Exponent e with x = f 2^e, 1/2 <= |f| < 1 (x != 0)."""
    return math.frexp(float(x))[1]


def line_exponents(X0: np.ndarray, axis: int) -> np.ndarray:
    """Shared grid exponent of every row (axis 0) or column (axis 1) of the
    leading-limb plane: the largest frexp exponent of a nonzero entry, and 0 for
    an all-zero line (section 3: a zero needs no balancing)."""
    X0 = np.asarray(X0, dtype=np.float64)
    lines = X0 if axis == 0 else X0.T
    out = np.zeros(lines.shape[0], dtype=np.int64)
    for r in range(lines.shape[0]):
        nz = [frexp_exp(x) for x in lines[r] if x != 0.0]
        out[r] = max(nz) if nz else 0
    return out


# --------------------------------------------------------------------------
# the exact splitter
# --------------------------------------------------------------------------

def grid_unit(E: int, s: int, bits: int = SLICE_BITS) -> Fraction:
    """Unit of slice s on the grid of exponent E: 2^(E - w (s + 1)), w = bits
    (13 in section 2)."""
    return Fraction(2) ** int(E - bits * (s + 1))


def split_element(limbs, E: int, S: int, bits: int = SLICE_BITS):
    """Digits and residual of one multiple double on the grid of exponent E.

    Following the worked example of section 2, the magnitude of the exact value
    is cut into consecutive 13-bit fields below 2^E, truncating (the fields are
    plain bit fields of the value); every digit carries the sign of the value
    (sign-magnitude, the same-signed parts that the sign grouping and the 2^-52
    transfer of section 3 aim at).  With bits = w the fields are w bits wide
    (the adaptive slice width; w = 13 is section 2's cut).  Returns (digits, R) with
    value = sum_s digits[s] 2^(E - w(s+1)) + R, |R| < 2^(E - w S), R * value >= 0.
    Raises ValueError when |value| >= 2^E (the element is not on this grid).
    """
    E, S, bits = int(E), int(S), int(bits)
    v = value(limbs)
    if v == 0:
        return [0] * S, Fraction(0)
    sign = 1 if v > 0 else -1
    u = grid_unit(E, S - 1, bits)
    D = math.floor(abs(v) / u)
    if D >> (bits * S):
        raise ValueError("|value| >= 2^E: element is not on the grid")
    mask = (1 << bits) - 1
    digits = [sign * ((D >> (bits * (S - 1 - s))) & mask) for s in range(S)]
    R = v - sum((d * grid_unit(E, s, bits) for s, d in enumerate(digits)), Fraction(0))
    return digits, R


def split(X: np.ndarray, E: np.ndarray, S: int, axis: int, bits: int = SLICE_BITS) -> np.ndarray:
    """Digits [S][rows][cols] (int64) of an operand X [L][rows][cols]."""
    X = np.asarray(X, dtype=np.float64)
    L, rows, cols = X.shape
    D = np.zeros((S, rows, cols), dtype=np.int64)
    for r in range(rows):
        for c in range(cols):
            e = int(E[r] if axis == 0 else E[c])
            d, _ = split_element(X[:, r, c], e, S, bits)
            D[:, r, c] = d
    return D


# --------------------------------------------------------------------------
# slice pairs, levels, accumulation and rounding
# --------------------------------------------------------------------------

def pairs_of_level(t: int, S: int):
    """Slice pairs (p, q) with p + q = t, 0 <= p, q < S, in increasing p."""
    return [(p, t - p) for p in range(S) if 0 <= t - p < S]


def level_products(DA: np.ndarray, DB: np.ndarray, T: int) -> list:
    """G_t = sum over p + q = t of DA_p DB_q for t = 0..T, as Python-int matrices.

    Products of integers are exact; Python ints cannot overflow."""
    S, m, k = DA.shape
    n = DB.shape[2]
    A = [[[int(x) for x in row] for row in DA[p]] for p in range(S)]
    B = [[[int(x) for x in row] for row in DB[q]] for q in range(S)]
    G = []
    for t in range(T + 1):
        g = [[0] * n for _ in range(m)]
        for p, q in pairs_of_level(t, S):
            for i in range(m):
                ai = A[p][i]
                for j in range(n):
                    g[i][j] += sum(ai[kk] * B[q][kk][j] for kk in range(k))
        G.append(g)
    return G


def accumulate(levels, EA: int, EB: int, bits: int = SLICE_BITS) -> Fraction:
    """Z = sum_t G_t 2^(-13 t), times the grid scale 2^(EA + EB - 26).

    Slice p of A has unit 2^(EA - 13(p+1)) and slice q of B has unit
    2^(EB - 13(q+1)); their product has unit 2^(EA + EB - 26 - 13(p+q)), so level
    t = p + q carries weight 2^(EA + EB - 26 - 13 t).  With w-bit digits
    (bits = w) the weights are 2^(EA + EB - 2w - w t)."""
    z = Fraction(0)
    for t, g in enumerate(levels):
        z += Fraction(int(g)) * Fraction(2) ** int(EA + EB - 2 * bits - bits * t)
    return z


def round_to_limbs(z: Fraction, L: int):
    """Greedy round-to-nearest-even of an exact value into L doubles."""
    out = []
    r = z
    for _ in range(L):
        c = float(r) if r != 0 else 0.0
        out.append(c)
        r -= Fraction(c)
    return out


def exact_product(A: np.ndarray, B: np.ndarray, i: int, j: int):
    """(C_exact[i][j], (|A||B|)[i][j]) of the exact multiple-double operands."""
    k = A.shape[2]
    c = Fraction(0)
    mag = Fraction(0)
    for kk in range(k):
        a = value(A[:, i, kk])
        b = value(B[:, kk, j])
        c += a * b
        mag += abs(a) * abs(b)
    return c, mag


def tolerance(k: int, L: int, mag: Fraction) -> Fraction:
    """Componentwise bound 4 k 2^-(53 L - 4) (|A||B|)_ij on |C - C_exact|."""
    return 4 * k * Fraction(2) ** (-(53 * L - 4)) * mag


def method_bound(A: np.ndarray, B: np.ndarray, i: int, j: int, S: int, T: int, EA: int, EB: int,
                 bits: int = SLICE_BITS) -> Fraction:
    """Bound on |C[i][j] - C_exact[i][j]| of the sliced product with S digits per
    element and the pairs p + q <= T, from the parts of section 2:

    * truncation: a = alpha + r_a with |r_a| < 2^(EA - 13 S) and |alpha| <= |a|
      (the digits are the truncated quarters), likewise b, so
      |a b - alpha beta| <= |a| 2^(EB - 13 S) + |b| 2^(EA - 13 S) + 2^(EA + EB - 26 S);
    * dropped pairs: a product of digits is below 2^26 and the pair (p, q) weighs
      2^(EA + EB - 13 (p + q + 2)), so level t > T adds at most
      pairs_t 2^26 2^(EA + EB - 13 (t + 2)) per term of the inner product;
    * the final rounding into L limbs, greedy round to nearest: at most
      2^(-53 L) (1 + 2^-53) |Z| with |Z| <= |C_exact| + the two terms above.

    With S = 4 L this is about 2^(5 - 13 S) k 2^(EA + EB) relative, which for
    L >= 5 is looser than 4 k 2^-(53 L - 4) (|A||B|): four 13-bit digits carry 52
    of the 53 bits of every limb.  With w-bit digits (bits = w) every 13 above is w
    and a product of digits is below 2^(2w)."""
    w = int(bits)
    k = A.shape[2]
    two = Fraction(2)
    L = A.shape[0]
    trunc = Fraction(0)
    mag = Fraction(0)
    for kk in range(k):
        a, b = abs(value(A[:, i, kk])), abs(value(B[:, kk, j]))
        mag += a * b
        trunc += a * two ** (EB - w * S) + b * two ** (EA - w * S) + two ** (EA + EB - 2 * w * S)
    dropped = Fraction(0)
    for t in range(T + 1, 2 * S - 1):
        dropped += len(pairs_of_level(t, S)) * two ** (2 * w + EA + EB - w * (t + 2))
    dropped *= k
    return trunc + dropped + 2 * two ** (-53 * L) * (mag + trunc + dropped)


MAX_SLICES = 68  # digits per element
MAX_DIGIT_BITS = 908  # digits times width


def default_slices(L: int) -> int:
    """The default number of 13-bit digits of an L-limb element.  Up to four limbs
    the paper's four quarters per limb (section 2), 52 L bits, at least the 53 L - 4
    bits that the tolerance 4 k 2^-(53 L - 4) (|A||B|) asks for.  From five limbs
    on, four quarters per limb give fewer bits than that; the count is then the
    smallest number of 13-bit digits holding 53 L - 4 bits, plus one more for the
    levels that the cutoff T = S - 1 leaves out."""
    if L <= 4:
        return 4 * L
    return math.ceil((53 * L - 4) / 13) + 1


def adaptive_width(L: int, k: int, max_digit_bits: int = MAX_DIGIT_BITS):
    """(w, S) of the adaptive slice width: among w = 13..26 with S = ceil(13 S13 / w)
    digits (S13 = default_slices(L): the bits of the default 13-bit digits) such
    that every level with T <= S - 1 stays exact, S k (2^w - 1)^2 < 2^53 (the bound
    (NBound) of section 2 with w-bit digits), the fewest pairs S (S + 1) / 2, the
    wider digit on a tie; S <= 68 and S w <= max_digit_bits.  None when no width
    qualifies."""
    best = None
    bits = 13 * default_slices(L)
    for w in range(13, 27):
        S = -(-bits // w)
        if S > MAX_SLICES or S * w > max_digit_bits or S * k * (2**w - 1) ** 2 >= 2**53:
            continue
        key = (S * (S + 1) // 2, -w)
        if best is None or key < best[0]:
            best = (key, w, S)
    return None if best is None else (best[1], best[2])


def line_spread(X0: np.ndarray, axis: int) -> np.ndarray:
    """Exponent range of every row (axis 0) or column (axis 1) of a leading-limb
    plane: the line's grid exponent minus the smallest frexp exponent of a nonzero
    entry (section 3: the exponents a group of numbers spans); 0 for a zero line."""
    X0 = np.asarray(X0, dtype=np.float64)
    lines = X0 if axis == 0 else X0.T
    out = np.zeros(lines.shape[0], dtype=np.int64)
    for i, line in enumerate(lines):
        exps = [frexp_exp(float(x)) for x in line if x != 0.0]
        if exps:
            out[i] = max(exps) - min(exps)
    return out


def _pair_count(S: int, T: int) -> int:
    return sum(len(pairs_of_level(t, S)) for t in range(T + 1))


def _max_pairs(S: int, T: int) -> int:
    return max(len(pairs_of_level(t, S)) for t in range(T + 1))


def plan(L: int, k: int, *, slice_bits: int = 0, slices: int = 0, slices_per_limb: int = 0, cutoff: int = -1,
         range_bits: int = 0, int8: bool = False, group_exponent: bool = False, group_sign: bool = False):
    """(w, S, T) of the product's digit width, digit count and cutoff, or None when
    the levels cannot stay exact.  Written from the options' definitions:

    * w = 13 (slice_bits 0 or 13): S0 = slices, or slices_per_limb L, or
      (slices_per_limb 0) default_slices(L);
      w explicit: S0 = slices or ceil(13 default_slices(L) / w);
      automatic (slice_bits -1): the width of 13..26 with the fewest pairs of the
      resulting (S, T) among those whose levels stay exact, the wider on a tie;
    * range balancing: D = ceil(range_bits / w) more digits, S = S0 + D, default
      cutoff T = S0 - 1 + 2 D (a product of two elements D digits below their
      lines' grids keeps its S0 leading levels); cutoff -2 keeps every pair;
    * exactness: max pairs of a kept level times k (2^w - 1)^2 below 2^53;
    * int8 (level sums in int32 on the int8 matrix cores): digits of at most 7
      bits; slice_bits 0 or -1 take the widest w = 7, 6, ..., 1 whose (S, T) is
      valid and whose level sums stay below 2^31 (the same bound with 2^31 in
      place of 2^53), slice_bits 1..7 that width, S0 = slices or
      ceil(13 default_slices(L) / w), at most 64 digits;
    * exponent classes (group_exponent, section 3): range_bits sets
      1 + ceil(range_bits / w) classes instead of extra digits, one more digit
      per element (S = S0 + 1 when there is more than one class), default cutoff
      S0 + 1 per class pair; the levels reach T + 2 (classes - 1); sign groups
      (group_sign) change no count; grouped products take up to 4 limbs and no
      automatic width.
    Raises ValueError for invalid options (S > 68, S w > 908, ...)."""
    bits = 13 * default_slices(L)
    if ((group_exponent and range_bits > 0) or group_sign) and slice_bits == -1:
        raise ValueError("groups with the automatic width")

    def finish(w, S0):
        if group_exponent:
            # exponent classes (section 3): range_bits sets 1 + ceil(range_bits / w)
            # classes; one more digit per element (it lies up to one digit below
            # its class grid) when there is more than one class
            D = 1 if range_bits > 0 else 0
            classes = 1 + -(-range_bits // w)
        else:
            D = -(-range_bits // w)
            classes = 1
        S = S0 + D
        if S < 1 or S > (64 if int8 else MAX_SLICES) or S * w > MAX_DIGIT_BITS:
            raise ValueError("digit count")
        T = S0 - 1 + 2 * D if cutoff == -1 else (2 * S - 2 if cutoff == -2 else cutoff)
        if not 0 <= T <= 2 * S - 2:
            raise ValueError("cutoff")
        if w * (T + 2 * (classes - 1)) + 55 > 64 * 28:  # the exact level sum fits 28 words
            raise ValueError("levels")
        if (group_exponent and classes > 1) or group_sign:
            # grouped products: up to 4 limbs, the split's integer in 6 words, 4096 panels
            if int8 or slice_bits == -1 or L > 4 or -(-(w * S + 52) // 64) > 6 or \
                    (2 if group_sign else 1) * classes * S > 4096:
                raise ValueError("groups")
        return w, S, T

    def exact_ok(w, S, T):
        return _max_pairs(S, T) * k * (2**w - 1) ** 2 < 2**53

    if int8:
        def exact32(w, S, T):
            return _max_pairs(S, T) * k * (2**w - 1) ** 2 < 2**31

        if slice_bits in (0, -1):
            if slices:
                raise ValueError("slices with the automatic width")
            sized = False
            for w in range(7, 0, -1):
                try:
                    cand = finish(w, -(-bits // w))
                except ValueError:
                    continue
                sized = True
                if exact32(*cand):
                    return cand
            if not sized:
                raise ValueError("digit count")
            return None
        if not 1 <= slice_bits <= 7:
            raise ValueError("width")
        cand = finish(slice_bits, slices or -(-bits // slice_bits))
        return cand if exact32(*cand) else None

    if slice_bits == -1:
        if slices:
            raise ValueError("slices with the automatic width")
        best = None
        for w in range(13, 27):
            try:
                cand = finish(w, -(-bits // w))
            except ValueError:
                continue
            if not exact_ok(*cand):
                continue
            key = (_pair_count(cand[1], cand[2]), -w)
            if best is None or key < best[0]:
                best = (key, cand)
        return None if best is None else best[1]
    w = 13 if slice_bits in (0, 13) else slice_bits
    if not 1 <= w <= 26:
        raise ValueError("width")
    if w == 13:
        S0 = slices or (slices_per_limb * L if slices_per_limb else default_slices(L))
    else:
        S0 = slices or -(-bits // w)
    cand = finish(w, S0)
    return cand if exact_ok(*cand) else None


def is_nonoverlapping(limbs) -> bool:
    """|x_{l+1}| <= ulp(x_l)/2 and a zero limb is followed only by zeros."""
    for a, b in zip(limbs[:-1], limbs[1:]):
        a, b = float(a), float(b)
        if a == 0.0:
            if b != 0.0:
                return False
            continue
        if abs(b) > 0.5 * math.ulp(a):
            return False
    return True
