"""GPU parity of the LDS-tiled split (split_tile_kernel), the split that panels of
at least 2048 tiles of 64 lines x 16 k values take for up to four limbs.

Every panel is compared with the oracle's digits (coracle.split, an exact
splitter of its own) over the whole panel, padding included, at shapes whose
line count and k are not multiples of the tile: through the stage entry
mdgemm_split_panel (FP64 panels, any width) and through mdgemm_ex (FP32 panels,
read back from the workspace).  The cases cover one to four limbs, both
operands, 13-, 19-, 24- and 26-bit digits, the 128-bit and 256-bit floors and
the general floor (digit windows above 256 bits), grid exponents above the
lines' maxima, and zero lines, zeros, subnormals and opposite-sign limbs.
"""

import numpy as np
import pytest
import torch

from oracle import coracle
from paper_2607_06881_amd import mdgemm as md
from paper_2607_06881_amd import workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _operand(L, rows, cols, seed):
    rng = np.random.default_rng(seed)
    X = workloads.make_operand(rng, L, rows, cols, "normal", row_exp=6, col_exp=6)
    X[:, 5, :] = 0.0                       # a zero row
    X[:, :, 7] = 0.0                       # a zero column
    X[:, 11, 3:40] *= 2.0**-1040           # subnormal leading limbs (lower limbs flush to zero)
    X[1:, 11, 3:40] = 0.0
    if L > 1:                              # limbs of opposite sign
        X[1, 20:30, :] = -np.abs(X[1, 20:30, :]) * np.sign(X[0, 20:30, :])
    return X


def _panel_from_oracle(D, axis, kp, cp):
    """Oracle digits [S][rows][cols] in the panel layout [S][kp][cp] with zero padding."""
    S, rows, cols = D.shape
    P = np.zeros((S, kp, cp))
    if axis == 0:      # A: lines are rows, k runs along columns
        P[:, :cols, :rows] = D.transpose(0, 2, 1)
    else:              # B: lines are columns, k runs along rows
        P[:, :rows, :cols] = D
    return P


def _wide(lines, k):
    return (md.panel_mn(lines) // 64) * (md.panel_k(k) // 16) >= 2048


@pytest.mark.parametrize("L,axis,bits,S,eshift", [
    (1, 0, 13, 4, 0), (2, 0, 13, 8, 0), (2, 1, 13, 8, 0), (3, 1, 13, 12, 0), (4, 0, 13, 16, 0),
    (2, 0, 19, 6, 0), (3, 1, 24, 7, 0), (2, 1, 26, 4, 0), (4, 1, 13, 22, 0), (2, 0, 13, 8, 5)])
def test_split_tile_stage_entry_against_the_oracle(L, axis, bits, S, eshift):
    rows, cols = (1000, 2100) if axis == 0 else (2100, 1000)
    lines, k = (rows, cols) if axis == 0 else (cols, rows)
    assert _wide(lines, k)
    print(f"[case] split tile stage entry L={L} axis={axis} w={bits} S={S} window={bits * S} +E={eshift}",
          flush=True)
    X = _operand(L, rows, cols, 100 * L + 10 * axis + bits)
    E = coracle.exponents(X[0], axis) + eshift
    Dg = md.mdgemm_split_panel(torch.from_numpy(X).to(DEV), torch.from_numpy(E).to(DEV), S, axis, bits=bits)
    torch.cuda.synchronize()
    want = _panel_from_oracle(coracle.split(X, E, S, axis, bits=bits), axis, md.panel_k(k), md.panel_mn(lines))
    got = Dg.cpu().numpy()
    assert got.shape == want.shape
    assert np.array_equal(got, want)
    assert not np.signbit(got[got == 0.0]).any()  # zero digits are +0.0


@pytest.mark.parametrize("L,bits", [(2, 13), (3, 13), (1, 13), (2, 19)])
def test_split_tile_fp32_panels_of_mdgemm_ex(L, bits):
    m, k, n = 1000, 2100, 1000
    opts = {} if bits == 13 else {"slice_bits": bits}
    w, S, T = md.mdgemm_plan(m, n, k, L, **opts)
    lay = md.mdgemm_workspace_layout(m, n, k, L, **opts)
    assert lay["panel_bytes"] == 4 and (lay["mp"] // 64) * (lay["kp"] // 16) >= 2048
    print(f"[case] split tile FP32 panels L={L} w={w} S={S} T={T}", flush=True)
    A = _operand(L, m, k, 7 + L)
    B = _operand(L, k, n, 9 + L)
    ws = torch.empty(md.mdgemm_workspace_bytes(m, n, k, L, **opts), dtype=torch.uint8, device=DEV)
    md.mdgemm_ex(torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV), workspace=ws, **opts)
    torch.cuda.synchronize()
    parts = md.workspace_parts(ws, m, n, k, L, **opts)
    EA, EB = coracle.exponents(A[0], 0), coracle.exponents(B[0], 1)
    assert np.array_equal(parts["EA"].cpu().numpy(), EA) and np.array_equal(parts["EB"].cpu().numpy(), EB)
    kp, mp, np_ = lay["kp"], lay["mp"], lay["np"]
    wantA = _panel_from_oracle(coracle.split(A, EA, S, 0, bits=w), 0, kp, mp)
    wantB = _panel_from_oracle(coracle.split(B, EB, S, 1, bits=w), 1, kp, np_)
    assert np.array_equal(parts["DA"][:S].cpu().numpy().astype(np.float64), wantA)
    assert np.array_equal(parts["DB"][:S].cpu().numpy().astype(np.float64), wantB)


@pytest.mark.parametrize("k", [2100, 64])
def test_staged_path_with_operands_off_16_byte_alignment(k):
    # the same product through views of A and B that start 8 bytes into their
    # buffers (the exponent pass then reads A's rows with 8-byte loads): the
    # exponents equal the oracle's and C equals the aligned product's bit for bit
    m, n, L = 1000, 1000, 2
    print(f"[case] staged product on operands 8 bytes off alignment, k={k}", flush=True)
    A = _operand(L, m, k, 31)
    B = _operand(L, k, n, 32)
    Ag, Bg = torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV)
    bufA = torch.empty(A.size + 1, dtype=torch.float64, device=DEV)
    bufB = torch.empty(B.size + 1, dtype=torch.float64, device=DEV)
    Au, Bu = bufA[1:].view(L, m, k), bufB[1:].view(L, k, n)
    Au.copy_(Ag)
    Bu.copy_(Bg)
    assert Au.data_ptr() % 16 == 8 and Bu.data_ptr() % 16 == 8
    ws = torch.empty(md.mdgemm_workspace_bytes(m, n, k, L), dtype=torch.uint8, device=DEV)
    C = md.mdgemm_ex(Au, Bu, workspace=ws, flags=md.MDGEMM_STAGED)
    torch.cuda.synchronize()
    parts = md.workspace_parts(ws, m, n, k, L, flags=md.MDGEMM_STAGED)
    assert np.array_equal(parts["EA"].cpu().numpy(), coracle.exponents(A[0], 0))
    assert np.array_equal(parts["EB"].cpu().numpy(), coracle.exponents(B[0], 1))
    C0 = md.mdgemm_ex(Ag, Bg, flags=md.MDGEMM_STAGED)
    torch.cuda.synchronize()
    assert torch.equal(C, C0)
