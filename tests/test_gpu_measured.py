"""GPU parity of the measured distortion tables (Appendix D, exact DP over measured distortion).

* kvc_measured_quant (quantization term of every candidate (r, b), fp32 on the device) against the
  oracle's fp64 tables from exact codes, on synthetic heads, within 1e-3 relative (the device decides
  codes in fp32, so a few elements on a threshold may take the neighbouring code);
* the truncation term from kvc_covariance and kvc_query_variance against the oracle's sample variances;
* the whole measured path of the pipeline on a 16-head workload: every head gets a feasible (r, b), the
  budget holds, and on the measured tables the DP's total is no larger than that of the damped
  allocation on the model (the DP is exact for the tables).
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import alloc as oa
from oracle import measured as om
from paper_2609_24298_amd import kvc, pipeline, synth

from oracle_stats import oracle_stats

pytestmark = pytest.mark.gpu

RANKS = (2, 6, 14, 16, 18, 64, 66, 96, 126, 128)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _calib_tokens(stats, n, seed, side=kvc.SIDE_K):
    x = torch.empty((len(stats), n, 128), dtype=torch.float16, device="cuda")
    for h, s in enumerate(stats):
        x[h] = synth.draw_tokens_torch(s.F_k if side == kvc.SIDE_K else s.F_v, n, (seed, 5150, h, side), "cuda")
    return x


@pytest.mark.parametrize("side", [kvc.SIDE_K, kvc.SIDE_V])
def test_measured_tables_match_oracle(side):
    w = synth.Workload("meas", 1, 4, 4, 1, 1, 1.0)
    st = oracle_stats(w, 2)
    n = 1024
    x = _calib_tokens(st, n, 2, side)
    quant, trunc_w, order = pipeline.measured_tables(st, x, n, side)
    xb = x.view(torch.int16).cpu().numpy().view(np.uint16)
    grid = kvc.rank_grid()
    worst_q = worst_t = 0.0
    for h, s in enumerate(st):
        U, lam, sign = (s.U_k, s.lam_k, s.sign_k) if side == kvc.SIDE_K else (s.U_v, s.lam_v, s.sign_v)
        wt = s.sigma2_q if side == kvc.SIDE_K else np.ones(128)
        assert list(order[h]) == oa.importance_order([a * b for a, b in zip(wt, lam)])
        Q = om.quant_table(xb[h], U, order[h], lam, sign, wt, RANKS, range(1, 9))
        for k, r in enumerate(RANKS):
            ri = grid.index(r)
            e = np.abs(quant[h, ri] - Q[k]) / Q[k]
            worst_q = max(worst_q, float(e.max()))
            assert np.all(e <= 1e-3), (h, r, e)
        lam_hat = om.sample_variances(xb[h], U)
        ref = wt * lam_hat
        e = np.abs(trunc_w[h] - ref) / ref.max()
        worst_t = max(worst_t, float(e.max()))
        assert np.all(e <= 1e-5), h
    log(f"[measured side {side}] quant term within {worst_q:.1e} relative, truncation within {worst_t:.1e}")


def test_measured_dp_allocation_on_a_workload():
    w = synth.Workload("meas_dp", 2, 8, 4, 1, 1, 1.0)
    st = oracle_stats(w, 4)
    n = 2048
    x = _calib_tokens(st, n, 4)
    quant, trunc_w, order = pipeline.measured_tables(st, x, n, kvc.SIDE_K)
    am = kvc.kvc_allocate_measured(quant, trunc_w, order, kvc.alloc_opts(w.bpd))
    dm = kvc.kvc_allocate(np.stack([s.lam_k for s in st]), np.stack([s.sigma2_q for s in st]), kvc.alloc_opts(w.bpd))
    H = len(st)
    assert np.sum(am["r"] * am["b"]) <= w.bpd * H * 128
    assert np.all(am["r"] * am["b"] <= am["B"])
    grid = kvc.rank_grid()

    def total(r, b):
        t = 0.0
        for h in range(H):
            T = om.truncation_terms(order[h], trunc_w[h], np.ones(128))
            t += T[r[h]] + quant[h, grid.index(int(r[h])), int(b[h]) - 1]
        return t

    t_dp, t_damped = total(am["r"], am["b"]), total(dm["r"], dm["b"])
    log(f"[measured DP] total measured distortion {t_dp:.5e} (damped on the model: {t_damped:.5e}); "
        f"(r, b) changed on {np.mean((am['r'] != dm['r']) | (am['b'] != dm['b'])):.0%} of heads")
    assert t_dp <= t_damped * (1 + 1e-12)
    # the cache builds from the measured tables
    cache = pipeline.Cache(w, seed=4, stats=st, capacity=64, measured=(quant, trunc_w, order))
    assert np.array_equal(cache.k_tab.r, am["r"]) and np.array_equal(cache.k_tab.b, am["b"])
