"""GPU parity of the level GEMM's 64-row tiles (slice_gemm32_kernel<64>), the
tiles that products with at most 64 output rows take on FP32 digit panels,
such as the V^T X products of the blocked QR.

The staged path is forced (MDGEMM_STAGED) so that the fused small-product
kernel does not take the smaller of these shapes.  Without a k split the level
planes the product leaves in its workspace are compared over the whole matrix
with the oracle's levels of the oracle's digits.  With a k split (the QR's
64 x 4096 x 4032 at the adaptive digit width among them) the limbs are compared
bit for bit with the same product with one more row of A (128-row tiles,
checked against the oracle elsewhere) and with the oracle at sampled entries.
"""

import numpy as np
import pytest
import torch

from checks import nonoverlap_all
from oracle import coracle, pipeline
from paper_2607_06881_amd import mdgemm as md
from paper_2607_06881_amd import workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _operands(L, m, k, n, seed):
    rng = np.random.default_rng(seed)
    A = workloads.make_operand(rng, L, m + 1, k, "normal", row_exp=4, col_exp=4)
    B = workloads.make_operand(rng, L, k, n, "normal", row_exp=4, col_exp=4)
    A[:, 0, 3:9] = 0.0  # zeros inside a row
    return A, B


@pytest.mark.parametrize("m,k,n,L", [(64, 250, 1000, 2), (1, 200, 700, 2), (37, 255, 1300, 3), (64, 16, 129, 1),
                                     (17, 100, 4000, 2)])
def test_skinny_levels_against_the_oracle(m, k, n, L):
    print(f"[case] 64-row tiles, levels: {m}x{k}x{n} L={L}", flush=True)
    A1, B = _operands(L, m, k, n, m * 7 + n)
    A = np.ascontiguousarray(A1[:, :m])
    opts = {"flags": md.MDGEMM_STAGED}
    w, S, T = md.mdgemm_plan(m, n, k, L, **opts)
    info = md.mdgemm_schedule_info(m, n, k, S, T)
    assert info["panels_f32"] == 1 and info["ksplit"] == 1
    ws = torch.empty(md.mdgemm_workspace_bytes(m, n, k, L, **opts), dtype=torch.uint8, device=DEV)
    C = md.mdgemm_ex(torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV), workspace=ws, **opts)
    torch.cuda.synchronize()
    parts = md.workspace_parts(ws, m, n, k, L, **opts)
    assert parts["layout"]["panel_bytes"] == 4 and parts["layout"]["direct_levels"] == 1
    EA, EB = coracle.exponents(A[0], 0), coracle.exponents(B[0], 1)
    DA, DB = coracle.split(A, EA, S, 0), coracle.split(B, EB, S, 1)
    G = parts["G"][: T + 1].cpu().numpy()
    assert np.array_equal(G, pipeline.levels_rewritten(DA, DB, T))
    C_h = C.cpu().numpy()
    assert nonoverlap_all(C_h)
    entries = [(0, 0), (m - 1, n - 1), (m // 2, n // 3), (0, n - 1)]
    for (i, j), r in pipeline.reference_entries(A, B, S, T, entries).items():
        assert C_h[:, i, j].tolist() == r["limbs"], (i, j)


@pytest.mark.parametrize("m,k,n,L,auto", [(64, 4096, 4032, 2, True), (40, 3000, 2100, 2, False),
                                          (64, 1000, 130, 3, False), (5, 2000, 300, 2, True)])
def test_skinny_with_k_split_equals_128_row_tiles(m, k, n, L, auto):
    print(f"[case] 64-row tiles, k split: {m}x{k}x{n} L={L} auto={auto}", flush=True)
    A1, B = _operands(L, m, k, n, m + k + n)
    A = np.ascontiguousarray(A1[:, :m])
    opts = {"flags": md.MDGEMM_STAGED}
    if auto:
        opts["slice_bits"] = md.MDGEMM_SLICE_BITS_AUTO
    w, S, T = md.mdgemm_plan(m, n, k, L, **opts)
    info = md.mdgemm_schedule_info(m, n, k, S, T, bits=w)
    assert info["panels_f32"] == 1 and info["ksplit"] > 1
    Bg = torch.from_numpy(B).to(DEV)
    C = md.mdgemm_ex(torch.from_numpy(A).to(DEV), Bg, **opts)
    C1 = md.mdgemm_ex(torch.from_numpy(A1).to(DEV), Bg, **opts)  # m + 1 rows: 128-row tiles
    torch.cuda.synchronize()
    assert md.mdgemm_plan(m + 1, n, k, L, **opts) == (w, S, T)
    assert torch.equal(C, C1[:, :m])
    C_h = C.cpu().numpy()
    assert nonoverlap_all(C_h)
    entries = [(0, 0), (m - 1, n - 1), (m // 2, n // 2), (m - 1, 0)]
    for (i, j), r in pipeline.reference_entries(A, B, S, T, entries, bits=w).items():
        assert C_h[:, i, j].tolist() == r["limbs"], (i, j)
