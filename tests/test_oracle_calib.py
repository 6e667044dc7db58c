"""Pins of the oracle's calibration step (table step 1): the fp64 Jacobi eigendecomposition and the
query variance along each key eigendirection (CPU only)."""
import math

import numpy as np
import pytest

from oracle import calib
from oracle.native import jacobi_eigh


def _spd(rng, d, spread=1.0):
    Q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    lam = np.sort(rng.uniform(0.01, 1.0, d) ** spread)[::-1]
    return Q @ np.diag(lam) @ Q.T, lam


def test_jacobi_two_by_two_closed_form():
    # eigenvalues of [[a, b], [b, c]]: (a + c)/2 +- sqrt(((a - c)/2)^2 + b^2); eigenvector of the
    # larger one along (b, lam1 - a)
    for a, b, c in ((2.0, 1.0, 3.0), (1.0, -0.5, 1.0), (5.0, 1e-3, -2.0), (0.0, 2.0, 0.0)):
        lam, U, _ = jacobi_eigh(np.array([[a, b], [b, c]]))
        m, r = (a + c) / 2, math.hypot((a - c) / 2, b)
        assert lam[0] == pytest.approx(m + r, rel=1e-15, abs=1e-15)
        assert lam[1] == pytest.approx(max(m - r, 0.0), rel=1e-15, abs=1e-15)
        v = np.array([b, m + r - a])
        v = v / np.linalg.norm(v)
        v = v * np.sign(v[np.argmax(np.abs(v))])
        assert np.allclose(U[:, 0], v, atol=1e-15)


def test_jacobi_diagonal_is_exact_and_sorted():
    D = np.diag([0.5, 3.0, 1.0, 3.0, 0.0])
    lam, U, sweeps = jacobi_eigh(D)
    assert list(lam) == [3.0, 3.0, 1.0, 0.5, 0.0]
    # ties keep the diagonal index order: eigen index 0 -> e_1, 1 -> e_3
    assert np.array_equal(U, np.eye(5)[:, [1, 3, 2, 0, 4]])
    assert sweeps == 1


@pytest.mark.parametrize("d,spread", [(8, 1.0), (64, 3.0), (128, 1.0), (128, 6.0)])
def test_jacobi_matches_library_eigh(d, spread):
    rng = np.random.default_rng(d + int(spread))
    S, lam_true = _spd(rng, d, spread)
    lam, U, _ = jacobi_eigh(S)
    ref, V = np.linalg.eigh(S)
    ref, V = ref[::-1], V[:, ::-1]
    assert np.max(np.abs(lam - ref)) <= 1e-13 * lam[0]
    assert np.max(np.abs(lam - lam_true)) <= 1e-13 * lam[0]
    # eigenvectors up to sign (eigenvalues here are separated by far more than the rounding)
    gaps = np.minimum(np.abs(np.diff(ref, prepend=np.inf)), np.abs(np.diff(ref, append=-np.inf)))
    err = np.abs(np.abs(np.sum(U * V, axis=0)) - 1.0)
    assert np.all(err <= 1e-20 + 1e-12 * (lam[0] / gaps) ** 2)
    # orthonormal and reproduces S; fixed sign convention
    assert np.max(np.abs(U.T @ U - np.eye(d))) <= 1e-13
    assert np.max(np.abs(U @ np.diag(lam) @ U.T - S)) <= 1e-13 * lam[0]
    j = np.argmax(np.abs(U), axis=0)
    assert np.all(U[j, np.arange(d)] > 0)


def test_jacobi_batched_equals_one_by_one():
    rng = np.random.default_rng(7)
    S = np.stack([_spd(rng, 32)[0] for _ in range(5)])
    lam, U, sw = jacobi_eigh(S)
    for h in range(5):
        l1, U1, s1 = jacobi_eigh(S[h])
        assert np.array_equal(lam[h], l1) and np.array_equal(U[h], U1) and sw[h] == s1


def test_query_variance_special_cases():
    rng = np.random.default_rng(3)
    S_k, lam = _spd(rng, 16)
    _, U, _ = jacobi_eigh(S_k)
    # isotropic queries: variance 1 along every direction
    assert np.allclose(calib.query_variance(U, [np.eye(16)]), 1.0, atol=1e-14)
    # queries distributed like the keys: variance lambda_i along eigendirection i
    assert np.allclose(calib.query_variance(U, [S_k]), np.sort(lam)[::-1], rtol=1e-12)
    # mean over the query heads of a group
    S2 = 3.0 * np.eye(16)
    assert np.allclose(calib.query_variance(U, [np.eye(16), S2]), 2.0, atol=1e-14)


def test_query_variance_matches_monte_carlo():
    # sigma^2_Q,i = E[(u_i . q)^2] for zero-mean queries (Section 2), estimated from samples
    rng = np.random.default_rng(11)
    d = 32
    S_k, _ = _spd(rng, d)
    F = [rng.standard_normal((d, d)) / math.sqrt(d) for _ in range(3)]
    S_q = [f @ f.T for f in F]
    _, U, _ = jacobi_eigh(S_k)
    est = np.zeros(d)
    for f in F:
        qs = rng.standard_normal((200_000, d)) @ f.T
        est += np.mean((qs @ U) ** 2, axis=0)
    est /= 3
    assert np.allclose(est, calib.query_variance(U, S_q), rtol=0.02)


def test_sample_covariance_is_centred():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((1000, 6)) + 7.0
    S = calib.sample_covariance(x)
    xc = x - x.mean(axis=0)
    assert np.allclose(S, xc.T @ xc / 1000, rtol=1e-13)
    assert np.allclose(calib.sample_covariance(x - 7.0), S, rtol=1e-12)
