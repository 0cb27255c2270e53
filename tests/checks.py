"""Checks of results shared by several test files (no GPU code, no oracle
arithmetic): the nonoverlap invariant of multiple doubles over whole arrays."""

import numpy as np


def nonoverlap_all(C) -> bool:
    """Every element of C [L][...] is nonoverlapping in the half-ulp sense of
    section 1: |x_{l+1}| <= ulp(x_l)/2, and a zero limb is followed only by zeros."""
    C = np.asarray(C, dtype=np.float64)
    ok = np.ones(C.shape[1:], dtype=bool)
    for l in range(C.shape[0] - 1):
        hi, lo = C[l], C[l + 1]
        ok &= np.where(hi == 0, lo == 0, np.abs(lo) <= 0.5 * np.spacing(np.abs(hi)))
    return bool(ok.all())
