"""Pins of the oracle's Taylor-series solver (coracle.taylor_dd): the
coefficients X_k of the solution of A(t) X(t) = B(t) modulo t^(d+1), formed
degree by degree with the QR of A_0 in double-double.

Each pin is fixed by something other than the recurrence the solver follows:
closed forms of scalar series ((1 - t)^-1 and (1 - t)^-2 have the coefficients
1 and k + 1), the Neumann series of I - t N for a nilpotent N
(X_k = sum_j N^j B_{k-j}, checked exactly in integers), and the exact residual
of the defining identity sum_i A_i X_{k-i} = B_k in rational arithmetic for
random well-conditioned data.  A dropped term, a wrong sign of the convolution
or a transposed coefficient fails one of them.
"""

from fractions import Fraction

import numpy as np

from oracle import coracle


def _scalar(coeffs, d):
    out = np.zeros((d + 1, 2, 1, 1))
    for k, c in enumerate(coeffs):
        out[k, 0, 0, 0] = c
    return out


def test_geometric_series():
    d = 12
    X = coracle.taylor_dd(_scalar([1.0, -1.0], d), _scalar([1.0], d))
    assert X[:, 0, 0, 0].tolist() == [1.0] * (d + 1) and not X[:, 1].any()


def test_square_of_the_geometric_series():
    d = 10
    X = coracle.taylor_dd(_scalar([1.0, -2.0, 1.0], d), _scalar([1.0], d))
    assert X[:, 0, 0, 0].tolist() == [float(k + 1) for k in range(d + 1)] and not X[:, 1].any()


def test_constant_matrix_series_divides_exactly():
    d = 4
    rng = np.random.default_rng(3)
    b = rng.integers(-1000, 1000, size=d + 1).astype(np.float64)
    X = coracle.taylor_dd(_scalar([2.0], d), _scalar(b, d))
    assert X[:, 0, 0, 0].tolist() == (b / 2).tolist() and not X[:, 1].any()


def test_nilpotent_neumann_series_exact():
    # A(t) = I - t N, N strictly upper triangular: X(t) = sum_j t^j N^j B(t)
    n, r, d = 6, 3, 5
    rng = np.random.default_rng(11)
    N = np.triu(rng.integers(-2, 3, size=(n, n)), 1)
    Bi = rng.integers(-50, 50, size=(d + 1, n, r))
    A = np.zeros((d + 1, 2, n, n))
    A[0, 0] = np.eye(n)
    A[1, 0] = -N
    B = np.zeros((d + 1, 2, n, r))
    B[:, 0] = Bi
    X = coracle.taylor_dd(A, B)
    powers = [np.eye(n, dtype=np.int64)]
    for _ in range(d):
        powers.append(powers[-1] @ N)
    for k in range(d + 1):
        want = sum(powers[j] @ Bi[k - j] for j in range(k + 1))
        assert np.array_equal(X[k, 0], want.astype(np.float64)), k
        assert not X[k, 1].any()


def _exact(x):
    return Fraction(float(x))


def test_random_system_exact_residual():
    # well-conditioned A_0 (diagonally dominant), double-double data with low limbs
    n, r, d = 5, 3, 4
    rng = np.random.default_rng(5)
    A = np.zeros((d + 1, 2, n, n))
    B = np.zeros((d + 1, 2, n, r))
    for k in range(d + 1):
        A[k, 0] = rng.standard_normal((n, n)) + (4.0 * np.eye(n) if k == 0 else 0.0)
        A[k, 1] = A[k, 0] * 2.0**-60 * rng.uniform(-1, 1, size=(n, n))
        B[k, 0] = rng.standard_normal((n, r))
        B[k, 1] = B[k, 0] * 2.0**-60 * rng.uniform(-1, 1, size=(n, r))
    X = coracle.taylor_dd(A, B)
    scale = np.abs(A[:, 0]).max() * np.abs(X[:, 0]).max() * n * (d + 1)
    worst = 0.0
    for k in range(d + 1):
        for i in range(n):
            for c in range(r):
                s = -(_exact(B[k, 0, i, c]) + _exact(B[k, 1, i, c]))
                for a in range(k + 1):
                    for l in range(n):
                        s += (_exact(A[a, 0, i, l]) + _exact(A[a, 1, i, l])) * \
                             (_exact(X[k - a, 0, l, c]) + _exact(X[k - a, 1, l, c]))
                worst = max(worst, abs(float(s)))
    assert worst <= 1e-30 * scale, worst / scale
    # and the leading limbs agree with a float64 solve of the same recurrence's first step
    X0 = np.linalg.solve(A[0, 0], B[0, 0])
    assert np.allclose(X[0, 0], X0, rtol=1e-12, atol=1e-12)
