"""A seeded sweep of small products through mdgemm_ex, every limb of every
output compared bit for bit with the oracle's chain (grid exponents, exact
digits, int64 levels, exact sum, greedy rounding: pipeline.full_reference).

Each case draws, from its own seed, the limb count (1 to 4), the output shape
(1 to 90 rows and columns), k (from 1 to 700, around the fused kernel's LDS
chunk and the staged path's k-split thresholds), the digit width (13 bits, the
adaptive width), the cutoff (the default, all pairs, or one in between), the
path (fused where it qualifies, or the stages) and the operands' spread of
row and column magnitudes, with zero rows and columns and limbs of opposite
sign mixed in.
"""

import numpy as np
import pytest
import torch

from checks import nonoverlap_all
from oracle import pipeline
from paper_2607_06881_amd import mdgemm as md
from paper_2607_06881_amd import workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
K_CHOICES = [1, 3, 4, 16, 63, 64, 65, 129, 200, 256, 383, 384, 385, 512, 700]


def _draw(case):
    rng = np.random.default_rng(7000 + case)
    L = int(rng.integers(1, 5))
    m, n = int(rng.integers(1, 91)), int(rng.integers(1, 91))
    k = int(rng.choice(K_CHOICES))
    opts = {}
    if rng.random() < 0.4:
        opts["slice_bits"] = md.MDGEMM_SLICE_BITS_AUTO
    w, S, T = md.mdgemm_plan(m, n, k, L, **opts)
    pick = rng.random()
    if pick < 0.3:
        opts["cutoff"] = md.MDGEMM_CUTOFF_ALL
    elif pick < 0.5:
        opts["cutoff"] = int(rng.integers(0, 2 * S - 1))
    if rng.random() < 0.5:
        opts["flags"] = md.MDGEMM_STAGED
    A = workloads.make_operand(rng, L, m, k, "normal", row_exp=int(rng.integers(0, 30)),
                               col_exp=int(rng.integers(0, 30)))
    B = workloads.make_operand(rng, L, k, n, "normal", row_exp=int(rng.integers(0, 30)),
                               col_exp=int(rng.integers(0, 30)))
    if m > 2 and rng.random() < 0.5:
        A[:, int(rng.integers(m)), :] = 0.0
    if n > 2 and rng.random() < 0.5:
        B[:, :, int(rng.integers(n))] = 0.0
    if L > 1 and m > 1:
        r = int(rng.integers(m))
        A[1, r, :] = -np.abs(A[1, r, :]) * np.sign(A[0, r, :])  # second limbs against the first
    return L, m, n, k, opts, A, B


@pytest.mark.parametrize("case", range(32))
def test_random_products_against_the_oracle(case):
    L, m, n, k, opts, A, B = _draw(case)
    w, S, T = md.mdgemm_plan(m, n, k, L, **opts)
    print(f"[case] sweep {case}: L={L} {m}x{k}x{n} w={w} S={S} T={T} opts={opts}", flush=True)
    C = md.mdgemm_ex(torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV), **opts)
    torch.cuda.synchronize()
    got = C.cpu().numpy()
    want = pipeline.full_reference(A, B, S, T, bits=w)["C"]
    bad = np.argwhere((got != want).any(axis=0))
    assert len(bad) == 0, f"{len(bad)} entries differ, first {bad[:4].tolist()}"
    assert nonoverlap_all(got)
