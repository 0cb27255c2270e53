"""GPU parity of the grouped products (section 3's balancing: by sign,
A = A+ + A-, and by exponent class, A = A_0 + A_1 + ...).

The digits of every group, the levels (every group pair at its level offset),
the exact sum and the greedy rounding must equal the oracle's grouped chain bit
for bit; sign groups alone must give the ungrouped product bit for bit (the
groups' digits add up to the operand's).  The wide-range workload c7 is run at
full size with exponent classes over its 60 bits: sampled entries bit-exact and
within the stated tolerance, where one grid per line misses it.
"""

import numpy as np
import pytest
import torch

from oracle import coracle, exact, pipeline
from paper_2607_06881_amd import mdgemm as md
from paper_2607_06881_amd import workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
GE, GS = md.MDGEMM_GROUP_EXPONENT, md.MDGEMM_GROUP_SIGN


def _wide(L, m, k, n, range_bits, seed):
    # workload c7's recipe: column kk of A scaled 2^-e_kk, row kk of B 2^(e_kk - range)
    rng = np.random.default_rng(seed)
    A = workloads.make_operand(rng, L, m, k, "normal")
    B = workloads.make_operand(rng, L, k, n, "normal")
    e = rng.integers(0, range_bits + 1, k)
    A *= np.ldexp(1.0, -e)[None, None, :]
    B *= np.ldexp(1.0, e - range_bits)[None, :, None]
    return A, B


@pytest.mark.parametrize("L,m,k,n,range_bits,flags,cutoff", [
    (2, 70, 48, 65, 60, GE, -1), (2, 33, 100, 129, 30, GE | GS, -1), (3, 20, 40, 17, 26, GE, -2),
    (4, 17, 33, 9, 13, GE | GS, -1), (1, 130, 64, 140, 40, GE, 5), (2, 129, 70, 131, 0, GS, -1),
    (3, 40, 100, 70, 0, GS, -2)])
def test_grouped_product_against_the_oracle(L, m, k, n, range_bits, flags, cutoff):
    w, S, T = md.mdgemm_plan(m, n, k, L, range_bits=range_bits, flags=flags, cutoff=cutoff)
    classes = 1 + -(-range_bits // w) if flags & GE else 1
    print(f"[case] grouped L={L} {m}x{k}x{n} range={range_bits} flags={flags}: S={S} T={T} classes={classes}",
          flush=True)
    assert (w, S, T) == exact.plan(L, k, range_bits=range_bits, cutoff=cutoff, group_exponent=bool(flags & GE),
                                   group_sign=bool(flags & GS))
    A, B = _wide(L, m, k, n, range_bits, L * 100 + k)
    Ag, Bg = torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV)
    C = md.mdgemm_ex(Ag, Bg, range_bits=range_bits, flags=flags, cutoff=cutoff).cpu().numpy()
    want = pipeline.full_reference_groups(A, B, S, T, classes, bool(flags & GS))
    assert np.array_equal(C, want)
    if flags == GS:  # sign groups alone: the ungrouped product
        plain = md.mdgemm_ex(Ag, Bg, cutoff=cutoff, flags=md.MDGEMM_STAGED).cpu().numpy()
        assert np.array_equal(C, plain)


def test_grouped_levels_from_the_workspace():
    # the level planes the grouped product leaves in its workspace equal the
    # oracle's grouped levels (every group pair at its offset) over the whole matrix
    L, m, k, n, rb = 2, 150, 90, 140, 40
    flags = GE | GS
    w, S, T = md.mdgemm_plan(m, n, k, L, range_bits=rb, flags=flags)
    classes = 1 + -(-rb // w)
    print(f"[case] grouped levels from the workspace: S={S} T={T} classes={classes}", flush=True)
    A, B = _wide(L, m, k, n, rb, 11)
    Ag, Bg = torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV)
    ws = torch.empty(md.mdgemm_workspace_bytes(m, n, k, L, range_bits=rb, flags=flags), dtype=torch.uint8,
                     device=DEV)
    md.mdgemm_ex(Ag, Bg, workspace=ws, range_bits=rb, flags=flags)
    torch.cuda.synchronize()
    parts = md.workspace_parts(ws, m, n, k, L, range_bits=rb, flags=flags)
    assert parts["G"].shape[0] == T + 1 + 2 * (classes - 1)
    EA, EB = pipeline.exponents(A, B)
    DA = pipeline.group_digits(A, EA, S, 0, classes, True)
    DB = pipeline.group_digits(B, EB, S, 1, classes, True)
    G = pipeline.group_levels(DA, DB, T, classes)
    assert np.array_equal(parts["G"].cpu().numpy(), G)
    # the digit panels: group g's digits in panels g S .. g S + S - 1 (A transposed)
    pa = parts["DA"].cpu().numpy()
    assert np.array_equal(pa[:, :k, :m], DA.reshape(-1, m, k).transpose(0, 2, 1))


def test_workload_c7_exponent_classes_full_size():
    w = workloads.WORKLOADS["c7"]
    opts = {"range_bits": w.range_bits, "flags": GE}
    bits, S, T = md.mdgemm_plan(w.m, w.n, w.k, w.limbs, **opts)
    classes = 1 + -(-w.range_bits // bits)
    print(f"[case] workload c7 with exponent classes: S={S} T={T} classes={classes}", flush=True)
    A_h, B_h = workloads.make_workload(w)
    A, B = torch.from_numpy(A_h).to(DEV), torch.from_numpy(B_h).to(DEV)
    ws = torch.empty(md.mdgemm_workspace_bytes(w.m, w.n, w.k, w.limbs, **opts), dtype=torch.uint8, device=DEV)
    C = md.mdgemm_ex(A, B, workspace=ws, **opts).cpu().numpy()
    del ws
    torch.cuda.empty_cache()
    EA, EB = coracle.exponents(A_h[0], 0), coracle.exponents(B_h[0], 1)
    rng = np.random.default_rng(77)
    entries = sorted({(int(rng.integers(w.m)), int(rng.integers(w.n))) for _ in range(14)}
                     | {(int(np.argmin(EA)), int(np.argmax(EB))), (0, 0)})
    ref = pipeline.reference_entries_groups(A_h, B_h, S, T, classes, False, entries)
    worst = 0.0
    for (i, j) in entries:
        assert C[:, i, j].tolist() == ref[(i, j)]["limbs"], (i, j)
        want, mag = exact.exact_product(A_h, B_h, i, j)
        r = float(abs(exact.value(C[:, i, j]) - want) / exact.tolerance(w.k, w.limbs, mag))
        assert r <= 1.0, (i, j, r)
        worst = max(worst, r)
    print(f"[result] c7 exponent classes: {len(entries)} entries bit-exact, max err/tolerance {worst:.3e}", flush=True)
