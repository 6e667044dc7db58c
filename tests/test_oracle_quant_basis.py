"""Pins of the oracle's quantizer and fused basis against closed forms, published
values, invariants and exact rational arithmetic (CPU only)."""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import basis as ob
from oracle import quant as oq

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- quantizer

def test_one_bit_step_closed_form():
    # 2-level mid-rise quantizer of N(0,1): levels +-step/2, optimum at step/2 = E|X| = sqrt(2/pi)
    assert abs(oq.optimal_step(1) - 2.0 * math.sqrt(2.0 / math.pi)) < 1e-7
    assert oq.delta_b(1) == 1.596


def test_steps_match_max_1960_table():
    rows = []
    with open(os.path.join(GOLDEN, "max1960_uniform_steps.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                b, n, s = line.split()
                rows.append((int(b), int(n), float(s)))
    assert len(rows) == 5
    for b, n, s in rows:
        assert n == 2 ** b
        assert abs(oq.delta_b(b) - s) <= 1e-4 * s + 1e-12, (b, oq.delta_b(b), s)


def test_steps_are_stationary_points_for_all_b():
    for b in range(1, 9):
        s = oq.optimal_step(b)
        h = s * 1e-3
        f0, fm, fp = (oq.gaussian_midrise_mse(v, b) for v in (s, s - h, s + h))
        assert fm > f0 and fp > f0
    # decreasing step with more bits
    steps = [oq.delta_b(b) for b in range(1, 9)]
    assert all(a > c for a, c in zip(steps, steps[1:]))


def test_gaussian_mse_matches_monte_carlo():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(2_000_000)
    for b in (1, 2, 3, 5, 8):
        step = oq.delta_b(b)
        h = 2 ** (b - 1)
        k = np.clip(np.floor(x / step) + h, 0, 2 ** b - 1)
        mc = np.mean((x - (k - h + 0.5) * step) ** 2)
        exact = oq.gaussian_midrise_mse(step, b)
        assert abs(mc - exact) < 5e-3 * exact + 1e-6, (b, mc, exact)


def test_fine_quantizer_mse_is_granular_noise():
    # many levels, step small: clipping vanishes and MSE -> step^2 / 12
    step = 0.01
    assert abs(oq.gaussian_midrise_mse(step, 12) - step * step / 12) < 1e-4 * step * step / 12


def test_code_exact_error_bound_and_clamp():
    rng = np.random.default_rng(2)
    for b in range(1, 9):
        step = Fraction(3, 7)
        h = 2 ** (b - 1)
        for _ in range(200):
            y = Fraction(int(rng.integers(-10 ** 6, 10 ** 6)), 10 ** 5)
            k = oq.code_exact(y, step, b)
            assert 0 <= k < 2 ** b
            level = (k - h + Fraction(1, 2)) * step
            if -h * step <= y < h * step:
                assert abs(y - level) <= step / 2
            elif y >= h * step:
                assert k == 2 ** b - 1
            else:
                assert k == 0
        # exact thresholds: y = j*step lands in cell j (floor), j-epsilon in j-1
        for j in range(-h + 1, h):
            assert oq.code_exact(j * step, step, b) == j + h
            assert oq.code_exact(j * step - Fraction(1, 10 ** 30), step, b) == j + h - 1


def test_head_step_constant_spectrum():
    for b in (1, 4, 8):
        st = oq.head_step([2.25] * 16, b)
        assert st == np.float32(1.5 * oq.delta_b(b))


def test_q_model_normalisation():
    assert oq.q_model(1) == 1.0 / 48.0
    assert oq.q_model(4) == 2.0 ** -8 / 12.0
    assert abs(oq.q_model(2.5) - 2.0 ** -5 / 12.0) < 1e-18


# ---------------------------------------------------------------- basis

EVEN_R = list(range(2, 129, 2))


def test_block_sizes_binary_expansion():
    for r in EVEN_R:
        s = ob.block_sizes(r)
        assert sum(s) == r and all(x & (x - 1) == 0 for x in s) and s == sorted(set(s), reverse=True)


@pytest.mark.parametrize("r", EVEN_R)
def test_rotation_is_orthogonal_in_integers(r):
    H = ob.rotation_matrix(r)
    n = ob.row_block_size(r)
    assert np.array_equal(H @ H.T, np.diag(n))          # rows orthogonal, squared norm = block size
    assert np.array_equal(np.abs(H).sum(axis=0), np.array([n[np.nonzero(H[:, i])[0][0]] for i in range(r)]))


def test_power_of_two_rotation_is_sylvester():
    for r in (2, 4, 8, 16, 32, 64, 128):
        assert np.array_equal(ob.rotation_matrix(r), ob.sylvester(r))


def test_deal_interleaves_blocks():
    # r = 96 = 64 + 32: two of every three positions go to the 64-block
    d = ob.deal(96)
    blocks = [j for j, _ in d]
    assert blocks.count(0) == 64 and blocks.count(1) == 32
    for k in range(0, 96, 3):
        assert sorted(blocks[k:k + 3]) == [0, 0, 1]
    # every block's columns are 0..n-1 in order
    for r in EVEN_R:
        seen = {}
        for j, c in ob.deal(r):
            assert c == seen.get(j, 0)
            seen[j] = c + 1


def _rand_orth(d, rng):
    Q, R = np.linalg.qr(rng.standard_normal((d, d)))
    return Q * np.sign(np.diag(R))


@pytest.mark.parametrize("r", [2, 6, 16, 50, 96, 128])
def test_fused_basis_orthonormal_and_spans_retained(r):
    rng = np.random.default_rng(r)
    d = 128
    U = _rand_orth(d, rng)
    order = rng.permutation(d)
    sign = rng.integers(0, 2, size=d) * 2 - 1
    P = ob.fused_basis_f64(U, order, r, sign)
    assert np.allclose(P @ P.T, np.eye(r), atol=1e-13)
    Ur = U[:, order[:r]]
    assert np.allclose(P.T @ P, Ur @ Ur.T, atol=1e-13)


def test_hadamard_equalises_variance_power_of_two():
    # Appendix A, Lemma lem:head-dist step 4: diag(H diag(lam) H^T) = mean(lam) for r = 2^k
    rng = np.random.default_rng(5)
    d = 128
    U = _rand_orth(d, rng)
    lam = np.sort(rng.uniform(0, 3, d))[::-1]
    Sigma = U @ np.diag(lam) @ U.T
    for r in (4, 32, 128):
        sign = rng.integers(0, 2, size=d) * 2 - 1
        P = ob.fused_basis_f64(U, np.arange(d), r, sign)
        v = np.diag(P @ Sigma @ P.T)
        assert np.allclose(v, lam[:r].mean(), rtol=1e-11)


def test_fp16_rounding_is_correctly_rounded():
    # compare numpy's fp64 -> fp16 conversion with exact round-to-nearest-even on rationals
    rng = np.random.default_rng(7)
    all_h = np.arange(0, 0x7C00, dtype=np.uint16).view(np.float16).astype(np.float64)   # finite positives
    vals = list(rng.uniform(-2, 2, 3000)) + list(rng.uniform(-1e-5, 1e-5, 3000))
    # exact midpoints between neighbouring fp16 values (ties) and values next to them
    for k in rng.integers(0, len(all_h) - 1, 500):
        mid = (all_h[k] + all_h[k + 1]) / 2.0
        vals += [mid, np.nextafter(mid, 0), np.nextafter(mid, 10), -mid]
    vals = np.array(vals)
    got = ob.fp16_bits(vals).view(np.float16).astype(np.float64)
    for v, g in zip(vals, got):
        fv = Fraction(float(v))
        a = abs(fv)
        i = np.searchsorted(all_h, float(a))
        cands = [all_h[j] for j in (i - 1, i) if 0 <= j < len(all_h)]
        best = min(cands, key=lambda c: (abs(Fraction(float(c)) - a),
                                         int(np.float16(c).view(np.uint16)) & 1))
        expect = best if fv >= 0 else -best
        assert g == expect, (v, g, expect)


def test_make_basis_step_uses_retained_eigenvalues():
    rng = np.random.default_rng(11)
    d = 128
    U = _rand_orth(d, rng)
    lam = np.sort(rng.uniform(0.01, 2, d))[::-1]
    order = rng.permutation(d)
    r, b = 24, 3
    sign = rng.integers(0, 2, size=d) * 2 - 1
    Pbits, step = ob.make_basis(U, order, lam, r, b, sign)
    assert Pbits.shape == (r, d) and Pbits.dtype == np.uint16
    s = 0.0
    for v in lam[order[:r]]:
        s += float(v)
    assert step == np.float32(math.sqrt(s / r) * 0.586)
