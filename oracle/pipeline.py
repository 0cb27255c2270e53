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


# --------------------------------------------------------------------------
# Grouped products (section 3: numbers grouped by sign, A = A+ + A-, and by the
# exponent of their leading part, A = A_0 + A_1 + ...; every group of A is
# multiplied with every group of B)
# --------------------------------------------------------------------------

def element_groups(X0: np.ndarray, E: np.ndarray, axis: int, classes: int, sign: bool, bits: int = 13) -> np.ndarray:
    """Group of every element of a leading-limb plane [rows][cols]: exponent class
    c = min(classes - 1, floor((E - e) / bits)) with e the frexp exponent of the
    element (0 for a zero element) and E its line's grid exponent, plus
    `classes` for a negative element when grouping by sign."""
    X0 = np.asarray(X0, dtype=np.float64)
    Eb = (E[:, None] if axis == 0 else E[None, :]).astype(np.int64)
    e = np.frexp(X0)[1].astype(np.int64)
    c = np.minimum(classes - 1, (Eb - e) // bits)
    c = np.where(X0 == 0.0, 0, c)
    if sign:
        c = c + np.where(X0 < 0.0, classes, 0)
    return c


def group_digits(X: np.ndarray, E: np.ndarray, S: int, axis: int, classes: int, sign: bool,
                 bits: int = 13) -> np.ndarray:
    """Digits [G][S][rows][cols] of the groups of X [L][rows][cols]: group g holds
    the digits of its own elements (zeros elsewhere), taken on the grid of its
    exponent class, E - (g mod classes) bits."""
    grp = element_groups(X[0], E, axis, classes, sign, bits)
    G = classes * (2 if sign else 1)
    out = np.zeros((G, S) + X.shape[1:], dtype=np.float64)
    for g in range(G):
        mask = grp == g
        if not mask.any():
            continue
        Xg = np.where(mask[None], X, 0.0)
        Eg = (np.asarray(E, dtype=np.int64) - (g % classes) * bits).astype(np.int32)
        out[g] = coracle.split(Xg, Eg, S, axis, bits)
    return out


def group_levels(DA: np.ndarray, DB: np.ndarray, T: int, classes: int) -> np.ndarray:
    """Levels of a grouped product: group pair (g, h) contributes DA[g][p] . DB[h][q]
    for p + q <= T at level p + q + (g mod classes) + (h mod classes); levels
    0 .. T + 2 (classes - 1), float64 matrix products (exact: integers < 2^53)."""
    G, S, m, k = DA.shape
    n = DB.shape[3]
    Tg = T + 2 * (classes - 1)
    out = np.zeros((Tg + 1, m, n), dtype=np.float64)
    for g in range(G):
        for h in range(G):
            o = g % classes + h % classes
            if not DA[g].any() or not DB[h].any():
                continue
            for t in range(T + 1):
                for p, q in exact.pairs_of_level(t, S):
                    out[t + o] += DA[g][p] @ DB[h][q]
    return out


def full_reference_groups(A: np.ndarray, B: np.ndarray, S: int, T: int, classes: int, sign: bool,
                          bits: int = 13) -> np.ndarray:
    """C [L][m][n] of the grouped product: group digits, levels, exact sum and
    greedy rounding (the sum uses the level weights of the shared line grids)."""
    L, m, k = A.shape
    n = B.shape[2]
    EA, EB = exponents(A, B)
    DA = group_digits(A, EA, S, 0, classes, sign, bits)
    DB = group_digits(B, EB, S, 1, classes, sign, bits)
    G = group_levels(DA, DB, T, classes)
    C = np.zeros((L, m, n), dtype=np.float64)
    for i in range(m):
        for j in range(n):
            z = exact.accumulate([int(G[t, i, j]) for t in range(G.shape[0])], int(EA[i]), int(EB[j]), bits)
            C[:, i, j] = exact.round_to_limbs(z, L)
    return C


def reference_entries_groups(A: np.ndarray, B: np.ndarray, S: int, T: int, classes: int, sign: bool, entries,
                             bits: int = 13) -> dict:
    """The grouped chain for chosen output entries: {(i, j): {"levels", "limbs"}}."""
    L = A.shape[0]
    EA, EB = exponents(A, B)
    G = classes * (2 if sign else 1)
    rows = sorted({i for i, _ in entries})
    cols = sorted({j for _, j in entries})
    dA = {i: group_digits(np.ascontiguousarray(A[:, i:i + 1, :]), EA[i:i + 1], S, 0, classes, sign, bits)[:, :, 0, :]
          for i in rows}
    dB = {j: group_digits(np.ascontiguousarray(B[:, :, j:j + 1]), EB[j:j + 1], S, 1, classes, sign, bits)[:, :, :, 0]
          for j in cols}
    out = {}
    Tg = T + 2 * (classes - 1)
    for i, j in entries:
        lv = [0] * (Tg + 1)
        a = dA[i].astype(np.int64)
        b = dB[j].astype(np.int64)
        for g in range(G):
            for h in range(G):
                o = g % classes + h % classes
                for t in range(T + 1):
                    for p, q in exact.pairs_of_level(t, S):
                        lv[t + o] += int(np.dot(a[g][p], b[h][q]))
        z = exact.accumulate(lv, int(EA[i]), int(EB[j]), bits)
        out[(i, j)] = {"levels": lv, "limbs": exact.round_to_limbs(z, L)}
    return out
