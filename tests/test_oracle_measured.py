"""Pins of the measured distortion tables and of the exact DP over them (CPU only)."""
import math

import numpy as np
import pytest

from oracle import alloc as oa
from oracle import attention as oatt
from oracle import calib
from oracle import measured as om
from oracle import quant as oq
from oracle.native import encode_codes
from paper_2609_24298_amd import synth


def _head(seed=0, n=512):
    c = synth.head_cov(seed, 0, 1, 2)
    lam_k, U_k, sq, _, _ = calib.head_calibration(c.S_k, c.S_v, c.S_q)
    rng = np.random.default_rng(seed)
    x = synth.draw_tokens_np(c.F_k, n, rng).view(np.uint16)
    order = oa.importance_order(oa.kl_weights(lam_k, sq))
    return x, U_k, order, lam_k, c.sign_k, sq


@pytest.mark.parametrize("r,b", [(2, 3), (16, 2), (40, 1), (64, 4), (98, 2), (128, 6)])
def test_mse_table_equals_direct_reconstruction_error(r, b):
    # with unit weights the measured D(r, b) is the mean squared reconstruction error of the deployed
    # quantizer, computed here the long way: encode, reconstruct x_hat = P^T z_hat, average ||x - x_hat||^2
    x, U, order, lam, sign, _ = _head()
    ones = np.ones(128)
    D, _, _ = om.measured_table(x, U, order, lam, sign, ones, [r], [b])
    P, step = om.make_basis(U, order, lam, r, b, sign)
    xhat = oatt.reconstruct(encode_codes(P, step, b, x), P, step, b)
    direct = np.mean(np.sum((oatt.fp16_to_f64(x) - xhat) ** 2, axis=1))
    # P's fp16 rounding leaves its rows orthonormal to about 1e-3
    assert D[0, 0] == pytest.approx(direct, rel=2e-3)


@pytest.mark.parametrize("b", [1, 2, 3, 4])
def test_isotropic_gaussian_matches_closed_form(b):
    # Sigma = s^2 I: every rotated coordinate is N(0, s^2) and the step is s delta_b, so
    # quant(r, b) / r -> s^2 mse_b (the exact Gaussian mid-rise MSE) and trunc(r) -> (d - r) s^2
    s2, d, n, r = 0.25, 128, 6000, 32
    rng = np.random.default_rng(b)
    x = (rng.standard_normal((n, d)) * math.sqrt(s2)).astype(np.float16).view(np.uint16)
    U, lam, order, sign = np.eye(d), np.full(d, s2), list(range(d)), np.where(rng.random(d) < 0.5, -1, 1)
    D, T, Q = om.measured_table(x, U, order, lam, sign, np.ones(d), [r], [b])
    step = oq.head_step([s2] * r, b) / math.sqrt(s2)
    expect = s2 * oq.gaussian_midrise_mse(step, b)
    assert Q[0, 0] / r == pytest.approx(expect, rel=0.03)
    assert T[r] == pytest.approx((d - r) * s2, rel=0.02)


def test_kl_weighted_table_matches_direct_weighted_error():
    # the block-weight form equals, in expectation, the error weighted along each eigendirection:
    # sum_i wt_i (u_i . (x - x_hat))^2 averaged over tokens (Gaussian data, uncorrelated coordinate errors)
    d, n = 128, 4000
    rng = np.random.default_rng(3)
    Q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    lam = np.arange(1, d + 1) ** -0.8
    x = ((rng.standard_normal((n, d)) * np.sqrt(lam)) @ Q.T).astype(np.float16).view(np.uint16)
    wt = rng.uniform(0.2, 3.0, d)
    order = list(range(d))
    sign = np.where(rng.random(d) < 0.5, -1, 1)
    for r, b in ((64, 2), (48, 3), (128, 1)):
        D, _, _ = om.measured_table(x, Q, order, lam, sign, wt, [r], [b])
        P, step = om.make_basis(Q, order, lam, r, b, sign)
        xhat = oatt.reconstruct(encode_codes(P, step, b, x), P, step, b)
        e = (oatt.fp16_to_f64(x) - xhat) @ Q
        direct = np.mean(np.sum(wt[None, :] * e * e, axis=1))
        assert D[0, 0] == pytest.approx(direct, rel=0.03), (r, b)


def test_row_weights_average_each_block():
    # r = 6 = 4 + 2: rows 0-3 form the 4-block, rows 4-5 the 2-block; positions dealt 0->4blk, 1->2blk, ...
    wt = np.arange(1.0, 129.0)
    order = list(range(128))
    c = om.row_weights(6, order, wt)
    members = {0: [], 1: []}
    for i, (j, _) in enumerate(om.deal(6)):
        members[j].append(i)
    assert sorted(members[0] + members[1]) == list(range(6)) and len(members[0]) == 4
    assert np.allclose(c[:4], np.mean(wt[members[0]])) and np.allclose(c[4:], np.mean(wt[members[1]]))


@pytest.mark.parametrize("bpd", [0.5, 1.0, 2.5])
def test_dp_over_tables_equals_exhaustive(bpd):
    rng = np.random.default_rng(int(bpd * 10))
    o = oa.AllocOpts(d=8, bpd=bpd, b_max=4)
    for _ in range(4):
        # measured tables need not follow the model: random, decreasing in r and b only on average
        tables = [np.sort(rng.uniform(0, 1, (4, 4)), axis=None)[::-1].reshape(4, 4) + rng.uniform(0, 0.3, (4, 4))
                  for _ in range(3)]
        budgets, allocs, total = oa.dp_tables(tables, o)
        assert sum(budgets) <= math.floor(bpd * 24)
        assert total == pytest.approx(oa.brute_force_tables(tables, o), rel=1e-14)
        for bh, a in zip(budgets, allocs):
            assert a[0] * a[1] <= bh


def test_table_of_the_model_reproduces_c1():
    # with the model itself as the table, the per-head optimum over all feasible pairs is C1's
    o = oa.AllocOpts(d=128)
    w = [3.0 * (i + 1) ** -1.2 for i in range(128)]
    table = [[oa.distortion(w, r, b) for b in range(1, 9)] for r in range(2, 129, 2)]
    for B in (2.0, 17.5, 64.0, 256.0, 511.0, 1024.0):
        assert oa.c1_table(table, B, o)[2] == oa.c1(w, B, o)[2]
