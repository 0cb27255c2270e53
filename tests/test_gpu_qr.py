"""GPU checks of the blocked Householder QR in double-double (mdgemm_qr_dd),
the downstream application whose trailing updates run on mdgemm.  Every panel
takes the multi-workgroup path (one launch per column; workgroups of 8, 16 or
32 rows by the panel's height), up to 70000 rows (2188 workgroups per launch).

The GPU factorization is checked in double-double arithmetic by the CPU
oracle: the residual max |A - Q R| / max |A| and the orthogonality
max |Q^T Q - I| of the Q formed from the returned vectors and tau must be at
the level of double-double rounding (the oracle's own unblocked factorization
reaches ~1e-31); R must agree with the oracle's R to the precision the
problem's conditioning allows; the diagonal of R is nonnegative and every
returned double-double is normalized.
"""

import numpy as np
import pytest
import torch

from checks import nonoverlap_all
from oracle import coracle
from paper_2607_06881_amd import mdgemm as md
from paper_2607_06881_amd import workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


@pytest.mark.parametrize("m,n,nb,seed", [(256, 128, 32, 1), (300, 173, 32, 2), (64, 64, 16, 3), (129, 1, 8, 4),
                                         (100, 37, 7, 5), (520, 96, 32, 6), (1100, 300, 32, 7), (700, 700, 32, 8),
                                         (1000, 61, 13, 9), (700, 700, 64, 10), (1100, 300, 64, 11), (300, 173, 48, 12),
                                         (129, 1, 64, 13), (520, 96, 40, 14), (70000, 40, 32, 15)])
def test_qr_dd_against_the_oracle(m, n, nb, seed):
    print(f"[case] qr dd {m}x{n} nb={nb}", flush=True)
    rng = np.random.default_rng(seed)
    A = workloads.make_operand(rng, 2, m, n, "normal")
    Ag = torch.from_numpy(A).to(DEV)
    QRg, taug = md.mdgemm_qr_dd(Ag.clone(), nb=nb)
    torch.cuda.synchronize()
    QR, tau = QRg.cpu().numpy(), taug.cpu().numpy()
    assert np.isfinite(QR).all() and np.isfinite(tau).all()
    for name, X in (("QR", QR), ("tau", tau)):
        hi, lo = X[0], X[1]
        bad = np.argwhere(~np.where(hi == 0, lo == 0, np.abs(lo) <= 0.5 * np.spacing(np.abs(hi))))
        if len(bad):
            print(f"[diag] {name}: {len(bad)} overlapping entries, first:",
                  [(tuple(int(x) for x in b), float(hi[tuple(b)]), float(lo[tuple(b)])) for b in bad[:6]], flush=True)
    assert nonoverlap_all(QR) and nonoverlap_all(tau)
    assert (np.diag(QR[0][:n]) >= 0.0).all()
    res, orth, _ = coracle.qr_dd_check(A, QR, tau)
    print(f"[result] qr {m}x{n}: residual {res:.2e}, orthogonality {orth:.2e}", flush=True)
    assert res < 1e-28 and orth < 1e-28
    QRo, tauo = coracle.qr_dd(A)
    ro, oo, _ = coracle.qr_dd_check(A, QRo, tauo)
    assert ro < 1e-29 and oo < 1e-29
    R = np.triu(QR[0] + QR[1])[:n]
    Ro = np.triu(QRo[0] + QRo[1])[:n]
    assert np.abs(R - Ro).max() <= 1e-24 * np.abs(Ro).max()


def test_qr_dd_refusals():
    A = torch.zeros((2, 10, 20), dtype=torch.float64, device=DEV)
    tau = torch.zeros((2, 20), dtype=torch.float64, device=DEV)
    ws = torch.empty(1 << 20, dtype=torch.uint8, device=DEV)
    lib = md.lib()
    assert lib.mdgemm_qr_dd(10, 20, 8, A.data_ptr(), tau.data_ptr(), ws.data_ptr(), ws.numel(), None) == \
        md.MDGEMM_EINVAL  # m < n
    assert lib.mdgemm_qr_dd(20, 10, 65, A.data_ptr(), tau.data_ptr(), ws.data_ptr(), ws.numel(), None) == \
        md.MDGEMM_EINVAL  # nb > 64
    need = lib.mdgemm_qr_dd_workspace_bytes(20, 10, 8)
    assert lib.mdgemm_qr_dd(20, 10, 8, A.data_ptr(), tau.data_ptr(), ws.data_ptr(), need - 1, None) == \
        md.MDGEMM_EWORKSPACE


@pytest.mark.parametrize("m,n,nb", [(600, 100, 32), (200, 90, 64)])
def test_qr_dd_triangular_and_zero_columns(m, n, nb):
    # an upper triangular A with a diagonal of mixed signs and a zero column:
    # every column has nothing below its pivot (sigma = 0), so each reflection
    # is the identity (tau = 0, x_1 >= 0) or flips the row (tau = 2, v = e_1),
    # and the stored vectors are zero.  R is A with the rows of negative pivots
    # negated.  Within the first panel the arithmetic is exact (the oracle agrees
    # bit for bit); the later columns pass through the trailing products, whose
    # digits on each line's grid keep the error within the product's bound, so
    # there the high limbs are exact and the low limbs within 1e-28 of each
    # entry (tall panels take the multi-workgroup path at m = 600)
    print(f"[case] qr dd triangular {m}x{n} nb={nb}", flush=True)
    rng = np.random.default_rng(m + n)
    A = workloads.make_operand(rng, 2, m, n, "normal")
    A[:, np.tril_indices(m, -1, n)[0], np.tril_indices(m, -1, n)[1]] = 0.0
    A[:, :, 7] = 0.0
    QRg, taug = md.mdgemm_qr_dd(torch.from_numpy(A).to(DEV).clone(), nb=nb)
    torch.cuda.synchronize()
    QR, tau = QRg.cpu().numpy(), taug.cpu().numpy()
    QRo, tauo = coracle.qr_dd(A)
    flip = A[0][np.arange(n), np.arange(n)] < 0.0
    assert np.array_equal(tau, tauo)
    assert np.array_equal(tau[0], np.where(flip, 2.0, 0.0)) and not tau[1].any()
    assert np.array_equal(QR[:, :, :nb], QRo[:, :, :nb])
    assert not np.tril(QR[0], -1).any() and not np.tril(QR[1], -1).any()
    R = np.where(flip[None, :, None], -A[:, :n], A[:, :n])
    assert np.array_equal(np.triu(QR[0][:n]), np.triu(R[0]))
    lo = np.abs(np.triu(QR[1][:n]) - np.triu(R[1]))
    assert (lo <= 1e-28 * np.abs(np.triu(R[0]))).all()


def test_qr_dd_rank_deficient():
    # repeated columns: after the first copy is eliminated the second has (nearly)
    # nothing left below its pivot; the factorization stays orthogonal and exact
    # to double-double level
    m, n = 500, 60
    print("[case] qr dd rank deficient", flush=True)
    rng = np.random.default_rng(21)
    A = workloads.make_operand(rng, 2, m, n, "normal")
    A[:, :, 30:40] = A[:, :, 0:10]
    A[:, :, 50] = 2.0 * A[:, :, 3]
    QRg, taug = md.mdgemm_qr_dd(torch.from_numpy(A).to(DEV).clone(), nb=32)
    torch.cuda.synchronize()
    QR, tau = QRg.cpu().numpy(), taug.cpu().numpy()
    assert np.isfinite(QR).all() and np.isfinite(tau).all()
    assert nonoverlap_all(QR) and nonoverlap_all(tau)
    res, orth, _ = coracle.qr_dd_check(A, QR, tau)
    print(f"[result] qr rank deficient: residual {res:.2e}, orthogonality {orth:.2e}", flush=True)
    assert res < 1e-28 and orth < 1e-28
