"""GPU checks of the Taylor-series solver (mdgemm_taylor_dd): the coefficients
of X(t) with A(t) X(t) = B(t) modulo t^(d+1), by the QR of A_0 and two products
on mdgemm_ex per degree.

* A(t) = I - t N with N strictly upper triangular and integer data: the QR of I
  leaves R = Q = I and every product is exact, so X must equal the Neumann
  series sum_j N^j B_{k-j} bit for bit (integers, checked in int64).
* Random well-conditioned systems (one and several QR panels, r = 1, d = 0,
  n = 1, a ragged n): X against the oracle's degree-by-degree QR solve in
  double-double, to a relative 1e-27 (both are accurate to the conditioning of
  A_0 times the double-double unit roundoff, 1e-30 here).
* n = 2100 (QR panels taller than 2048 rows, 33 back-substitution blocks): a
  banded nilpotent case exact in integers, and a random system whose identity
  A(t) X(t) = B(t) holds to float64 rounding (the oracle is too slow there).
"""

import numpy as np
import pytest
import torch

from oracle import coracle
from paper_2607_06881_amd import mdgemm as md

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _dd(rng, shape, scale=1.0):
    hi = rng.standard_normal(shape) * scale
    lo = hi * 2.0**-60 * rng.uniform(-1, 1, size=shape)
    return hi, lo


def test_taylor_nilpotent_exact():
    n, r, d = 100, 5, 5
    print(f"[case] taylor nilpotent n={n} r={r} d={d}", flush=True)
    rng = np.random.default_rng(17)
    N = np.triu(rng.integers(-2, 3, size=(n, n)), 1)
    Bi = rng.integers(-50, 50, size=(d + 1, n, r))
    A = np.zeros((d + 1, 2, n, n))
    A[0, 0] = np.eye(n)
    A[1, 0] = -N
    B = np.zeros((d + 1, 2, n, r))
    B[:, 0] = Bi
    X = md.mdgemm_taylor_dd(torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV))
    torch.cuda.synchronize()
    Xh = X.cpu().numpy()
    P = np.eye(n, dtype=np.int64)
    powers = [P]
    for _ in range(d):
        powers.append(powers[-1] @ N)
    for k in range(d + 1):
        want = sum(powers[j] @ Bi[k - j] for j in range(k + 1))
        assert np.abs(want).max() < 2**52
        assert np.array_equal(Xh[k, 0], want.astype(np.float64)), k
        assert not Xh[k, 1].any(), k


@pytest.mark.parametrize("n,r,d,seed", [(64, 4, 4, 1), (100, 7, 3, 2), (200, 16, 2, 3), (130, 1, 6, 4),
                                        (70, 33, 0, 5), (1, 3, 5, 6), (257, 2, 2, 7)])
def test_taylor_against_the_oracle(n, r, d, seed):
    print(f"[case] taylor n={n} r={r} d={d}", flush=True)
    rng = np.random.default_rng(seed)
    A = np.zeros((d + 1, 2, n, n))
    B = np.zeros((d + 1, 2, n, r))
    for k in range(d + 1):
        A[k, 0], A[k, 1] = _dd(rng, (n, n), 1.0 / np.sqrt(n))
        B[k, 0], B[k, 1] = _dd(rng, (n, r))
    A[0, 0] += 2.0 * np.eye(n)  # well conditioned A_0
    X = md.mdgemm_taylor_dd(torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV))
    torch.cuda.synchronize()
    Xh = X.cpu().numpy()
    Xo = coracle.taylor_dd(A, B)
    assert np.isfinite(Xh).all()
    for k in range(d + 1):
        got = Xh[k, 0] + Xh[k, 1]
        want = Xo[k, 0] + Xo[k, 1]
        err = np.abs((Xh[k, 0] - Xo[k, 0]) + (Xh[k, 1] - Xo[k, 1])).max()
        scale = np.abs(want).max()
        print(f"[result] taylor n={n} k={k}: max |X - X_oracle| / max |X| = {err / scale:.2e}", flush=True)
        assert err <= 1e-27 * scale, (k, err / scale)
        assert np.allclose(got, want, rtol=1e-12, atol=1e-14 * scale)


def test_taylor_large_banded_nilpotent_exact():
    # n above 2048: the first QR panels take 32-row workgroups, 33 back-substitution
    # blocks; N has three superdiagonals, so its powers stay small integers
    n, r, d = 2100, 3, 4
    print(f"[case] taylor banded nilpotent n={n} r={r} d={d}", flush=True)
    rng = np.random.default_rng(23)
    N = np.zeros((n, n), dtype=np.int64)
    for off in (1, 2, 3):
        N += np.diag(rng.integers(-1, 2, size=n - off), off)
    Bi = rng.integers(-50, 50, size=(d + 1, n, r))
    A = np.zeros((d + 1, 2, n, n))
    A[0, 0] = np.eye(n)
    A[1, 0] = -N
    B = np.zeros((d + 1, 2, n, r))
    B[:, 0] = Bi
    X = md.mdgemm_taylor_dd(torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV))
    torch.cuda.synchronize()
    Xh = X.cpu().numpy()
    # want[k] = sum_j N^j B_{k-j} = B_k + N want[k-1], exact in int64
    want = [Bi[0]]
    for k in range(1, d + 1):
        want.append(Bi[k] + N @ want[-1])
    for k in range(d + 1):
        assert np.array_equal(Xh[k, 0], want[k].astype(np.float64)), k
        assert not Xh[k, 1].any(), k


def test_taylor_large_random_residual():
    # a random well-conditioned system at n = 2100: the identity A(t) X(t) = B(t)
    # holds to float64 rounding (the double-double accuracy is the oracle tests')
    n, r, d = 2100, 3, 2
    print(f"[case] taylor random n={n} r={r} d={d}", flush=True)
    rng = np.random.default_rng(29)
    A = np.zeros((d + 1, 2, n, n))
    B = np.zeros((d + 1, 2, n, r))
    for k in range(d + 1):
        A[k, 0], A[k, 1] = _dd(rng, (n, n), 1.0 / np.sqrt(n))
        B[k, 0], B[k, 1] = _dd(rng, (n, r))
    A[0, 0] += 2.0 * np.eye(n)
    X = md.mdgemm_taylor_dd(torch.from_numpy(A).to(DEV), torch.from_numpy(B).to(DEV))
    torch.cuda.synchronize()
    Xh = X.cpu().numpy()
    assert np.isfinite(Xh).all()
    for k in range(d + 1):
        res = sum(A[i, 0] @ Xh[k - i, 0] for i in range(k + 1)) - B[k, 0]
        scale = np.abs(B[k, 0]).max() + sum(np.abs(A[i, 0]).max() * np.abs(Xh[k - i, 0]).max() * np.sqrt(n)
                                           for i in range(k + 1))
        print(f"[result] taylor n={n} k={k}: float64 residual / scale = {np.abs(res).max() / scale:.2e}", flush=True)
        assert np.abs(res).max() <= 1e-13 * scale, k
