"""Pins of the oracle allocator (C1, C2, DP) against closed forms, exhaustive
search and invariants (CPU only)."""
import math

import numpy as np
import pytest

from oracle import alloc as oa
from oracle.quant import q_model


def power_law(d, alpha, scale=1.0):
    return [scale * (i + 1) ** (-alpha) for i in range(d)]


def test_truncation_term_is_eckart_young_trace():
    # Lemma lem:trunc: E||x - U_r U_r^T x||^2 = sum_{i>r} lambda_i = tr((I - U_r U_r^T) Sigma)
    rng = np.random.default_rng(0)
    d = 32
    Q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    lam = np.sort(rng.uniform(0, 2, d))[::-1]
    Sigma = Q @ np.diag(lam) @ Q.T
    for r in (0, 2, 10, 31, 32):
        Ur = Q[:, :r]
        trace = np.trace((np.eye(d) - Ur @ Ur.T) @ Sigma)
        assert abs(oa.tail_sum(list(lam), r) - trace) < 1e-12
        # D(r, b) with b -> infinity tends to the trace (q(b) -> 0)
        assert abs(oa.distortion(list(lam), r, 60) - trace) < 1e-12 if r > 0 else True


def test_distortion_endpoints():
    w = power_law(16, 1.2)
    # r = d keeps everything: only quantisation loss q(b) * sum w
    assert oa.distortion(w, 16, 3) == pytest.approx(q_model(3) * sum(w), rel=1e-15)


@pytest.mark.parametrize("alpha", [0.5, 1.0, 1.5, 2.0])
def test_c1_equals_exhaustive_search(alpha):
    o = oa.AllocOpts(d=128)
    w = power_law(128, alpha, 3.0)
    for B in [2.0, 3.5, 17.0, 64.0, 100.3, 256.0, 300.7, 512.0, 1000.0, 1024.0, 2000.0]:
        a = oa.c1(w, B, o)
        e = oa.brute_force_head(w, B, o)
        assert a[2] == e[2], (B, a, e)
        assert a[0] * a[1] <= B


def test_c1_forward_difference_identity():
    # Eq. eq:c1-foc: f(r+2) - f(r) with b = B/r (continuous) equals the closed form
    w = power_law(128, 1.3)
    B = 256.0
    f = lambda r: oa.tail_sum(w, r) + q_model(B / r) * oa.head_sum(w, r)
    for r in range(2, 126, 2):
        lhs = f(r + 2) - f(r)
        qa, qb = q_model(B / (r + 2)), q_model(B / r)
        rhs = -(w[r] + w[r + 1]) * (1 - qa) + (qa - qb) * oa.head_sum(w, r)
        assert abs(lhs - rhs) < 1e-13 * max(1.0, abs(lhs)), r


def test_c1_relaxed_argmin_satisfies_two_sided_foc():
    for alpha in (0.7, 1.1, 1.9):
        w = power_law(128, alpha)
        for B in (64.0, 256.0, 512.0):
            f = lambda r: oa.tail_sum(w, r) + q_model(B / r) * oa.head_sum(w, r)
            grid = list(range(2, 129, 2))
            r_star = min(grid, key=f)
            df = lambda r: f(r + 2) - f(r)
            if r_star > 2:
                assert df(r_star - 2) <= 0
            if r_star < 128:
                assert df(r_star) >= 0


def test_c2_fixed_point_identical_heads():
    o = oa.AllocOpts(d=64, bpd=1.5)
    w = power_law(64, 1.0)
    B, allocs = oa.c2_damped([list(w) for _ in range(6)], o)
    assert all(b == 1.5 * 64 for b in B)
    assert len({a for a in allocs}) == 1


def test_c2_conserves_budget_and_moves_toward_high_distortion():
    rng = np.random.default_rng(3)
    o = oa.AllocOpts(d=128, bpd=1.0, rounds=1)
    W = [power_law(128, a, s) for a, s in zip(rng.uniform(0.5, 2, 20), rng.uniform(0.1, 10, 20))]
    B, _ = oa.c2_damped(W, o)
    assert abs(sum(B) - 20 * 128 * 1.0) < 1e-9
    D0 = [oa.c1(w, 128.0, o)[2] for w in W]
    Dbar = sum(D0) / len(D0)
    for b, d0 in zip(B, D0):
        if d0 > 1.5 * Dbar:
            assert b > 128.0
        if d0 < 0.5 * Dbar:
            assert b < 128.0


def test_c2_lowers_total_distortion_vs_uniform():
    rng = np.random.default_rng(4)
    o = oa.AllocOpts(d=128, bpd=1.0)
    W = [power_law(128, a, s) for a, s in zip(rng.uniform(0.5, 2, 32), rng.uniform(0.1, 10, 32))]
    _, allocs = oa.c2_damped(W, o)
    uni = sum(oa.c1(w, 128.0, o)[2] for w in W)
    assert sum(a[2] for a in allocs) < uni


@pytest.mark.parametrize("bpd", [0.5, 1.0, 2.0, 3.75])
def test_dp_equals_exhaustive_on_tiny_instances(bpd):
    rng = np.random.default_rng(int(bpd * 100))
    o = oa.AllocOpts(d=8, bpd=bpd, solver=oa.SOLVER_DP)
    for _ in range(3):
        W = [sorted(rng.uniform(0, 1, 8) ** rng.uniform(1, 4), reverse=True) for _ in range(3)]
        budgets, allocs, total = oa.dp_exact(W, o)
        assert sum(budgets) <= math.floor(bpd * 24)
        assert total == pytest.approx(sum(a[2] for a in allocs), rel=1e-15)
        assert total == pytest.approx(oa.brute_force_global(W, o), rel=1e-14)
        for bh, a in zip(budgets, allocs):
            assert a[0] * a[1] <= bh


def test_dp_is_no_worse_than_damped():
    rng = np.random.default_rng(9)
    o = oa.AllocOpts(d=32, bpd=1.0)
    W = [power_law(32, a, s) for a, s in zip(rng.uniform(0.5, 2, 6), rng.uniform(0.1, 10, 6))]
    _, damped = oa.c2_damped(W, o)
    _, _, dp_total = oa.dp_exact(W, o)
    assert dp_total <= sum(a[2] for a in damped) + 1e-15


def test_kl_weights_and_stable_reorder():
    lam = [4.0, 2.0, 1.0, 1.0, 0.5]
    sq = [0.1, 1.0, 2.0, 2.0, 8.0]
    w = oa.kl_weights(lam, sq)
    assert w == [0.4, 2.0, 2.0, 2.0, 4.0]
    assert oa.importance_order(w) == [4, 1, 2, 3, 0]


def test_kl_query_variance_matches_monte_carlo():
    # sigma_Q,i^2 = E[(u_i . q)^2] along each key eigendirection (Proposition prop:kl-bound (c))
    # on a synthetic head: the oracle's calibration of its exact covariances against samples
    from oracle import calib
    from paper_2609_24298_amd import synth
    c = synth.head_cov(0, 0, 0, 4, d=128)
    _, U_k, sig2, _, _ = calib.head_calibration(c.S_k, c.S_v, c.S_q)
    rng = np.random.default_rng(1)
    est = np.zeros(128)
    for F in c.F_q:
        q = rng.standard_normal((200_000, 128)) @ F.T
        est += np.mean((q @ U_k) ** 2, axis=0)
    est /= 4
    assert np.allclose(est, sig2, rtol=0.03, atol=1e-3 * sig2.max())


def test_allocate_c1_only_and_infeasible_fallback():
    o = oa.AllocOpts(d=16, bpd=0.05, solver=oa.SOLVER_C1_ONLY)   # B = 0.8 < r_min * b_min
    out = oa.allocate([power_law(16, 1.0)], None, o)
    assert out["r"][0] == 2 and out["b"][0] == 1


# ---------------------------------------------------------------- C2 update, worked by hand
#
# Three heads, d = 4 (ranks 2 and 4), bpd = 1: B_h = 4 at the start, B_tot = 12, B_bar = 4,
# eta B_bar = 1.2. Weights: A = (192, 0, 0, 0), B = (6, 6, 6, 6), C = (48, 0, 0, 0).
# C1 by hand (q(b) = 4^-b / 12, b = floor(B_h / r)):
#   A, C (one nonzero weight): r = 2 always wins, D = w_1 q(floor(B/2));
#   B (flat): for B_h in [4, 8) r = 4, b = 1, D = 24/48 = 0.5; for B_h in [2, 4) only r = 2 is
#   feasible, b = 1, D = 12 + 12/48 = 12.25.
# Round 1 (B = 4, 4, 4): D = (1, 0.5, 0.25), D_bar = 7/12;
#   B'_h = 4 + 1.2 (sqrt(D_h / D_bar) - 1) = 4 + 1.2 (sqrt(12/7), sqrt(6/7), sqrt(3/7)) - 1.2,
#   then B_h = B'_h * 12 / sum B'.
# Round 2 at those budgets (4.42, 3.95, 3.63): D = (1, 12.25, 1), D_bar = 4.75; each head moves by
#   1.2 (sqrt(D_h / 4.75) - 1) from its own budget (eta times the mean budget, not its own), C falls
#   to 2.976, which the floor B_min = 3 (second case) raises to 3 before renormalising.
# Final C1: A (r, b) = (2, 1), B = (4, 1), C = (2, 1). The literals below are those numbers to 16
# digits; a dropped square root, eta B_h for eta B_bar, renormalising before the clamp or a missing
# clamp each change them in the third digit or earlier.
C2_HAND = {
    (1, 2.0): [4.419884282818997, 3.9545709611535416, 3.6255447560274607],
    (2, 2.0): [3.9591044405021916, 4.9158683300781805, 3.1250272294196257],
    (2, 3.0): [3.950856704883234, 4.905627432690046, 3.1435158624267183],
}


@pytest.mark.parametrize("rounds,B_min", sorted(C2_HAND))
def test_c2_damped_update_worked_by_hand(rounds, B_min):
    o = oa.AllocOpts(d=4, bpd=1.0, rounds=rounds, B_min=B_min)
    W = [[192.0, 0.0, 0.0, 0.0], [6.0] * 4, [48.0, 0.0, 0.0, 0.0]]
    B, allocs = oa.c2_damped(W, o)
    assert np.allclose(B, C2_HAND[(rounds, B_min)], rtol=1e-14, atol=0)
    assert abs(sum(B) - 12.0) < 1e-12
    if rounds == 2:
        assert [(a[0], a[1]) for a in allocs] == [(2, 1), (4, 1), (2, 1)]
        assert [a[2] for a in allocs] == pytest.approx([4.0, 0.5, 1.0], rel=1e-15)
