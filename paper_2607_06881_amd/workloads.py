"""Seeded synthetic multiple-double operands.

This module only draws inputs.  It holds none of the product's arithmetic (no
splitting, no slice products, no accumulation); both the HIP path and the CPU
oracle consume the arrays it returns, so it must not import either of them.

The paper states only that random numbers were generated (section 4, bottom-up
method), so the five workloads below are synthetic stand-ins with the shapes of
its experiments: double-double and quad-double products of size 1024 to 4096
(Table 1) and the 1024 x 512 by 512 x 8192 rewritten double-double product of
the top-down method (section 4, Table 2).

Layout: an operand with L limbs and shape rows x cols is a float64 array
``[L][rows][cols]`` (limb-major, row-major planes, contiguous).  Limb 0 is the
most significant; every element is a *normalized* multiple double: for each
limb l, ``|x[l+1]| <= ulp(x[l]) / 2`` and ``x[l] == 0`` implies ``x[l+1] == 0``
(section 1, the definition of a multiple double as a sum of nonoverlapping
doubles, read with the usual half-ulp strength).

Draw order per operand: base values of limb 0, then the factors of the lower
limbs, then the power-of-two scales; operand A is drawn before operand B from
one ``numpy.random.default_rng(seed)`` (PCG64) stream.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "Workload",
    "WORKLOADS",
    "make_operand",
    "make_workload",
    "is_normalized",
    "pair_count",
]


@dataclass(frozen=True)
class Workload:
    """One synthetic product C[m x n] = A[m x k] . B[k x n] with L limbs.

    ``slices`` is the number S of 13-bit slices per operand element and
    ``cutoff`` the largest slice-index sum T = p + q kept in the product.
    """

    name: str
    limbs: int
    m: int
    n: int
    k: int
    slices: int
    cutoff: int
    seed: int
    base: str  # "uniform": limb 0 ~ U[-1, 1]; "normal": limb 0 ~ N(0, 1)
    row_exp: int = 0  # A rows scaled by 2^e, e ~ U{-row_exp..row_exp}
    col_exp: int = 0  # B columns scaled by 2^e, e ~ U{-col_exp..col_exp}
    elem_exp: int = 0  # every element scaled by 2^e, e ~ U{-elem_exp..elem_exp}
    # column k of A scaled by 2^-e_k and row k of B by 2^(e_k - inner_exp), e_k ~ U{0..inner_exp}:
    # every product a_ik b_kj has the same scale while each line of A and B spans inner_exp bits
    inner_exp: int = 0
    range_bits: int = 0  # the product's range balancing (extra digits for inner_exp bits of range)
    description: str = field(default="", compare=False)

    def options(self, adaptive: bool = False) -> dict:
        """Keyword options of mdgemm_ex for this workload's digits and cutoff, or
        for the adaptive width (with the same range balancing)."""
        if adaptive:
            opts = {"slice_bits": -1}
            if self.range_bits:
                opts["range_bits"] = self.range_bits
            return opts
        if self.range_bits:
            return {"range_bits": self.range_bits}
        return {"slices": self.slices, "cutoff": self.cutoff}

    @property
    def pairs(self) -> int:
        return pair_count(self.slices, self.cutoff)

    def slice_flops(self) -> float:
        """Flops of the slice products: 2 m n k for every kept pair."""
        return 2.0 * self.m * self.n * self.k * self.pairs

    def md_flops(self) -> float:
        """Flops of the multiple-double product counted as one operation per multiply-add."""
        return 2.0 * self.m * self.n * self.k


def pair_count(slices: int, cutoff: int) -> int:
    """Number of slice pairs (p, q), 0 <= p, q < slices, with p + q <= cutoff."""
    return sum(1 for p in range(slices) for q in range(slices) if p + q <= cutoff)


WORKLOADS = {
    "c0": Workload(
        "c0", 2, 64, 64, 64, 8, 14, 0, "uniform",
        description="double-double 64^3, hi ~ U[-1,1], lo = hi 2^-53 u, all slice pairs"),
    "c1": Workload(
        "c1", 2, 1024, 1024, 1024, 8, 14, 1, "uniform", row_exp=20, col_exp=20,
        description="double-double 1024^3, row/column scales 2^e, e ~ U{-20..20}, all slice pairs"),
    "c2": Workload(
        "c2", 2, 4096, 4096, 4096, 8, 7, 2, "uniform", elem_exp=8,
        description="double-double 4096^3, element scales 2^e, e ~ U{-8..8}, pairs p+q <= 7"),
    "c3": Workload(
        "c3", 4, 2048, 2048, 1024, 16, 15, 3, "normal",
        description="quad-double 2048x2048x1024, limb 0 ~ N(0,1), pairs p+q <= 15"),
    "c4": Workload(
        "c4", 3, 8192, 8192, 512, 12, 11, 4, "normal", row_exp=30, col_exp=30,
        description="triple-double 8192x8192x512, N(0,1) times row/column scales 2^e, e ~ U{-30..30}, pairs p+q <= 11"),
    # More limbs: the octo- and hexa-double shapes of the top-down method (section 4,
    # the table of dimensions adapted for dd, qd, od and hd), A 256 x 128 (od) and
    # 128 x 64 (hd), B with the 8192 columns of the rewritten second operand;
    # the default digit count for more than four limbs (the 53 L - 4 bits of the
    # tolerance in whole 13-bit digits plus one guard digit: 34 and 66).
    "c5": Workload(
        "c5", 8, 256, 8192, 128, 34, 33, 5, "normal",
        description="octo-double 256x8192x128, limb 0 ~ N(0,1), 34 digits, pairs p+q <= 33"),
    "c6": Workload(
        "c6", 16, 128, 8192, 64, 66, 65, 6, "normal",
        description="hexa-double 128x8192x64, limb 0 ~ N(0,1), 66 digits, pairs p+q <= 65"),
    # A wide range inside every line (section 3, balancing): the inner dimension is
    # scaled oppositely in A and B, so each row of A and column of B spans 60
    # bits while every term a_ik b_kj has the same size; one shared grid per line
    # loses the small elements' bits unless the lines get range balancing.
    "c7": Workload(
        "c7", 2, 2048, 2048, 2048, 13, 17, 7, "normal", inner_exp=60, range_bits=60,
        description="double-double 2048^3, A column k x 2^-e_k, B row k x 2^(e_k-60), e_k ~ U{0..60}; "
                    "range balancing over 60 bits: 13 digits, pairs p+q <= 17"),
}


def _two_sum(a: np.ndarray, b: np.ndarray):
    """Knuth's two-sum on arrays: s = fl(a + b) and e with s + e == a + b exactly."""
    s = a + b
    bb = s - a
    e = (a - (s - bb)) + (b - bb)
    return s, e


def is_normalized(x: np.ndarray) -> np.ndarray:
    """Elementwise check of the nonoverlap condition on a limb-major array ``[L, ...]``."""
    ok = np.isfinite(x).all(axis=0)
    for l in range(x.shape[0] - 1):
        hi, lo = x[l], x[l + 1]
        half_ulp = 0.5 * np.spacing(np.abs(hi))
        ok &= np.where(hi == 0, lo == 0, np.abs(lo) <= half_ulp)
    return ok


def _normalize(x: np.ndarray) -> np.ndarray:
    """Make the limbs nonoverlapping without changing any element's exact value.

    Sweeps of Knuth two-sums over neighbouring limbs (each sweep is exact) are
    repeated until every element passes ``is_normalized``.
    """
    x = x.copy()
    L = x.shape[0]
    for _ in range(4 * L + 4):
        for l in range(L - 1):
            x[l], x[l + 1] = _two_sum(x[l], x[l + 1])
        for l in range(L - 2, -1, -1):
            x[l], x[l + 1] = _two_sum(x[l], x[l + 1])
        # a zero leading limb with a nonzero tail is moved down by the sweeps above
        if is_normalized(x).all():
            return x
    raise RuntimeError("input normalization did not converge")


def make_operand(rng: np.random.Generator, limbs: int, rows: int, cols: int, base: str = "uniform",
                 row_exp: int = 0, col_exp: int = 0, elem_exp: int = 0) -> np.ndarray:
    """Draw one normalized operand ``[limbs, rows, cols]``.

    Limb 0 is U[-1, 1] (``base="uniform"``) or N(0, 1) (``base="normal"``);
    limb l > 0 is limb l-1 times 2^-53 u_l with u_l ~ U[-1, 1]; the limbs are
    then normalized.  Power-of-two scales (exact) are applied last.
    """
    shape = (rows, cols)
    x = np.empty((limbs,) + shape, dtype=np.float64)
    if base == "uniform":
        x[0] = rng.uniform(-1.0, 1.0, size=shape)
    elif base == "normal":
        x[0] = rng.standard_normal(size=shape)
    else:
        raise ValueError(base)
    for l in range(1, limbs):
        x[l] = x[l - 1] * 2.0**-53 * rng.uniform(-1.0, 1.0, size=shape)
    if limbs > 1:
        x = _normalize(x)
    scale = np.zeros(shape, dtype=np.int64)
    if row_exp:
        scale += rng.integers(-row_exp, row_exp + 1, size=(rows, 1))
    if col_exp:
        scale += rng.integers(-col_exp, col_exp + 1, size=(1, cols))
    if elem_exp:
        scale += rng.integers(-elem_exp, elem_exp + 1, size=shape)
    if row_exp or col_exp or elem_exp:
        x = np.ldexp(x, scale[None].astype(np.int32))
    return np.ascontiguousarray(x)


def make_workload(w: Workload | str, m: int | None = None, n: int | None = None, k: int | None = None,
                  seed: int | None = None):
    """Return ``(A, B)`` for a workload, optionally at a different size or seed.

    A gets the row scales and B the column scales; element scales apply to both.
    """
    if isinstance(w, str):
        w = WORKLOADS[w]
    m = w.m if m is None else m
    n = w.n if n is None else n
    k = w.k if k is None else k
    rng = np.random.default_rng(w.seed if seed is None else seed)
    A = make_operand(rng, w.limbs, m, k, w.base, row_exp=w.row_exp, elem_exp=w.elem_exp)
    B = make_operand(rng, w.limbs, k, n, w.base, col_exp=w.col_exp, elem_exp=w.elem_exp)
    if w.inner_exp:
        e = rng.integers(0, w.inner_exp + 1, k)
        A *= np.ldexp(1.0, -e)[None, None, :]  # powers of two: the limbs stay normalized
        B *= np.ldexp(1.0, e - w.inner_exp)[None, :, None]
    return A, B
