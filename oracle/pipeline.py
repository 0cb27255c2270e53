"""The method's steps chained on the CPU -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use this module; it shares no code with the GPU path.

The steps follow the overview of section 2 of Chen and Verschelde, "Multiple
Double Arithmetic on NVIDIA Tensor Cores", in its order:

1. split every multiple double into 13-bit parts (on the balanced grid of its
   row of A or column of B, section 3)            -> ``coracle.split``;
2.-3. multiply the parts pairwise, level t = p + q collecting the pairs of
   equation (3) / the rewritten product             -> int64 dot products;
4.-5. extract the parts of the product and add them into a multiple double
   (exactly, then rounded greedily to L limbs)      -> ``exact.accumulate`` and
   ``exact.round_to_limbs``.

``reference_entries`` evaluates this chain for chosen output entries only, so
that large products can be checked on samples.
"""

from __future__ import annotations

import numpy as np

from . import coracle, exact


def exponents(A: np.ndarray, B: np.ndarray):
    """(EA per row of A, EB per column of B) from the leading limbs."""
    return coracle.exponents(A[0], 0).astype(np.int64), coracle.exponents(B[0], 1).astype(np.int64)


def row_digits(A: np.ndarray, EA: np.ndarray, rows, S: int, bits: int = 13) -> dict:
    """Digits [S][k] (int64) of the chosen rows of A."""
    out = {}
    for i in rows:
        X = np.ascontiguousarray(A[:, i:i + 1, :])
        out[i] = coracle.split(X, np.array([EA[i]], dtype=np.int32), S, 0, bits)[:, 0, :].astype(np.int64)
    return out


def col_digits(B: np.ndarray, EB: np.ndarray, cols, S: int, bits: int = 13) -> dict:
    """Digits [S][k] (int64) of the chosen columns of B."""
    out = {}
    for j in cols:
        X = np.ascontiguousarray(B[:, :, j:j + 1])
        out[j] = coracle.split(X, np.array([EB[j]], dtype=np.int32), S, 1, bits)[:, :, 0].astype(np.int64)
    return out


def levels_of_entry(da: np.ndarray, db: np.ndarray, T: int) -> list:
    """G_t for one output entry from the digit row da [S][k] and column db [S][k].

    int64 dot products are exact: every partial sum is below 2^53 under the
    exactness condition pairs * k * (2^w - 1)^2 < 2^53 (w = 13: the analogue of
    the bound N (2^26 - 1) <= 2^52 of section 2)."""
    S = da.shape[0]
    G = []
    for t in range(T + 1):
        g = 0
        for p, q in exact.pairs_of_level(t, S):
            g += int(np.dot(da[p], db[q]))
        G.append(g)
    return G


def levels_rewritten(DA: np.ndarray, DB: np.ndarray, T: int) -> np.ndarray:
    """Level products G [T+1][m][n] (float64, integer valued) of whole digit
    planes DA [S][m][k], DB [S][k][n], one float64 matrix product per level.

    Level t is block column t of the rewritten product of section 2 (the
    stacked parts of A times the block-Toeplitz parts of B):
    G_t = [DA_p0 .. DA_p1] . [DB_(t-p0); ..; DB_(t-p1)] over the pairs p + q = t.
    Every product of two digits and every partial sum is an integer below 2^53
    under the exactness condition pairs * k * (2^w - 1)^2 < 2^53, so the matrix
    product (a library routine, any summation order) is exact."""
    S, m, k = DA.shape
    n = DB.shape[2]
    G = np.empty((T + 1, m, n), dtype=np.float64)
    for t in range(T + 1):
        ps = [p for p, _ in exact.pairs_of_level(t, S)]
        if not ps:
            G[t] = 0.0
            continue
        abar = np.concatenate([DA[p] for p in ps], axis=1)  # m x (pairs k)
        bbar = np.concatenate([DB[t - p] for p in ps], axis=0)  # (pairs k) x n
        np.matmul(abar, bbar, out=G[t])
    return G


def reference_entries(A: np.ndarray, B: np.ndarray, S: int, T: int, entries, bits: int = 13):
    """For each (i, j): dict with exponents, level products, exact Z and the
    greedy L-limb rounding of Z (the product's expected limbs)."""
    L = A.shape[0]
    EA, EB = exponents(A, B)
    rows = sorted({i for i, _ in entries})
    cols = sorted({j for _, j in entries})
    dA = row_digits(A, EA, rows, S, bits)
    dB = col_digits(B, EB, cols, S, bits)
    out = {}
    for i, j in entries:
        G = levels_of_entry(dA[i], dB[j], T)
        z = exact.accumulate(G, int(EA[i]), int(EB[j]), bits)
        out[(i, j)] = {
            "EA": int(EA[i]),
            "EB": int(EB[j]),
            "levels": G,
            "Z": z,
            "limbs": exact.round_to_limbs(z, L),
        }
    return out


def full_reference(A: np.ndarray, B: np.ndarray, S: int, T: int, bits: int = 13):
    """Whole-matrix chain for small products: exponents, digits, int64 levels
    and the rounded limbs C [L][m][n]."""
    L, m, k = A.shape
    n = B.shape[2]
    EA, EB = exponents(A, B)
    DA = coracle.split(A, EA.astype(np.int32), S, 0, bits)
    DB = coracle.split(B, EB.astype(np.int32), S, 1, bits)
    G = coracle.levels(DA, DB, T)
    C = np.zeros((L, m, n), dtype=np.float64)
    for i in range(m):
        for j in range(n):
            z = exact.accumulate([int(G[t, i, j]) for t in range(T + 1)], int(EA[i]), int(EB[j]), bits)
            C[:, i, j] = exact.round_to_limbs(z, L)
    return {"EA": EA, "EB": EB, "DA": DA, "DB": DB, "G": G, "C": C}
