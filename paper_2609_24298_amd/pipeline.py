"""Assemble a KV-COBRA compressed cache for a synthetic workload through libkvc.

The synthetic generator (synth) supplies exact covariances and draws tokens;
calibration (table step 1: eigendecomposition, query variance), allocation,
basis construction, encode, decode attention and reconstruction are library
calls. Layout of units: u = (layer * batch + sequence) * kv_heads + head; the
sequences of one (layer, head) share its basis.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import kvc, synth


@dataclass
class HeadStats:
    """Calibration record of one (layer, KV head): its covariances (and token factors) plus the
    results of table step 1 in fp64 arrays (eigenvalues descending, eigenvectors as columns)."""
    cov: synth.HeadCov
    lam_k: np.ndarray
    U_k: np.ndarray
    sigma2_q: np.ndarray
    lam_v: np.ndarray
    U_v: np.ndarray

    @property
    def F_k(self):
        return self.cov.F_k

    @property
    def F_v(self):
        return self.cov.F_v

    @property
    def F_q(self):
        return self.cov.F_q

    @property
    def sign_k(self):
        return self.cov.sign_k

    @property
    def sign_v(self):
        return self.cov.sign_v


def calibrate(covs, device="cuda", batch: int = 1024):
    """Table step 1 on the device for every head: kvc_eigh of the key and value covariances and
    kvc_query_variance of the query heads along the key eigendirections (fp32, as the paper states)."""
    import torch
    dev = torch.device(device)
    H, d = len(covs), covs[0].S_k.shape[0]
    out = {k: np.zeros((H, d)) for k in ("lam_k", "lam_v", "sigma2_q")}
    out.update({k: np.zeros((H, d, d)) for k in ("U_k", "U_v")})
    for h0 in range(0, H, batch):
        hs = covs[h0:h0 + batch]
        n = len(hs)
        for side in ("k", "v"):
            S = torch.as_tensor(np.stack([getattr(c, "S_" + side) for c in hs]).astype(np.float32), device=dev)
            lam = torch.empty((n, d), dtype=torch.float32, device=dev)
            U = torch.empty((n, d, d), dtype=torch.float32, device=dev)
            kvc.kvc_eigh(S, lam, U)
            if side == "k":
                Sq = torch.as_tensor(np.stack([np.stack(c.S_q) for c in hs]).astype(np.float32), device=dev)
                sig = torch.empty((n, d), dtype=torch.float32, device=dev)
                kvc.kvc_query_variance(U, Sq, sig)
                out["sigma2_q"][h0:h0 + n] = sig.cpu().numpy()
            out["lam_" + side][h0:h0 + n] = lam.cpu().numpy()
            out["U_" + side][h0:h0 + n] = U.cpu().numpy()
    return [HeadStats(c, out["lam_k"][h], out["U_k"][h], out["sigma2_q"][h], out["lam_v"][h], out["U_v"][h])
            for h, c in enumerate(covs)]


@dataclass
class SideTables:
    r: np.ndarray          # per head
    b: np.ndarray
    order: np.ndarray      # per head x d
    P: list                # per head: (r x d) uint16 fp16 bits
    delta: np.ndarray      # per head, float32


def measured_tables(stats, x_cal, n_tok: int, side: int = kvc.SIDE_K, r_min: int = 2, r_step: int = 2,
                    threads: int = 16):
    """Measured distortion tables of every head (Appendix D, exact DP over measured distortion), for
    kvc_allocate_measured: the candidate records on the host (kvc_make_candidates, heads in parallel
    threads), the quantization term on the device (kvc_measured_quant over the calibration activations
    x_cal, fp16 (H, >= n_tok, d) on the device), and the truncation term from the measured variance along
    each eigendirection (kvc_covariance without centring, then kvc_query_variance with G = 1). The K side
    weighs with sigma2_q (the attention-KL objective), the V side with 1 (MSE).
    Returns (quant (H, n_r, 8), trunc_w (H, d), order (H, d))."""
    import concurrent.futures as cf

    import torch
    dev = x_cal.device
    H, d = len(stats), stats[0].lam_k.shape[0]
    lam = np.stack([s.lam_k if side == kvc.SIDE_K else s.lam_v for s in stats])
    U = np.stack([s.U_k if side == kvc.SIDE_K else s.U_v for s in stats])
    wt = np.stack([s.sigma2_q for s in stats]) if side == kvc.SIDE_K else np.ones((H, d))
    sq = wt if side == kvc.SIDE_K else None
    order = kvc.kvc_allocate(lam, sq, kvc.alloc_opts(1.0, kvc.SOLVER_C1_ONLY))["order"]
    sign = [s.sign_k if side == kvc.SIDE_K else s.sign_v for s in stats]
    with cf.ThreadPoolExecutor(max_workers=threads) as ex:  # the host calls release the GIL
        cands = list(ex.map(lambda h: kvc.kvc_make_candidates(U[h], order[h], lam[h], wt[h], sign[h], r_min, r_step),
                            range(H)))
    P_all = torch.as_tensor(np.stack([c[0] for c in cands]).view(np.int16), device=dev)
    delta_all = torch.as_tensor(np.stack([c[1] for c in cands]), device=dev)
    rw_all = torch.as_tensor(np.stack([c[2] for c in cands]), device=dev)
    n_r = delta_all.shape[1]
    quant = torch.empty((H, n_r, 8), dtype=torch.float32, device=dev)
    kvc.kvc_measured_quant(x_cal, n_tok, P_all, delta_all, rw_all, quant, r_min, r_step)
    C = torch.empty((H, d, d), dtype=torch.float32, device=dev)
    kvc.kvc_covariance(x_cal, n_tok, C, centered=False)
    lam_hat = torch.empty((H, d), dtype=torch.float32, device=dev)
    kvc.kvc_query_variance(torch.as_tensor(U.astype(np.float32), device=dev), C.view(H, 1, d, d), lam_hat)
    trunc_w = wt * lam_hat.cpu().numpy().astype(np.float64)
    return quant.cpu().numpy().astype(np.float64), trunc_w, order


def allocate_workload(w: synth.Workload, stats, bpd: float | None = None, solver: int = kvc.SOLVER_DAMPED,
                      uniform=None, measured=None):
    """Joint K+V tables: K with attention-KL weights and C1+C2, V with MSE weights and C1 only.

    measured = (quant, trunc_w, order) from measured_tables takes the K side from the exact DP over
    measured distortion tables instead of C1 + C2 on the model.

    uniform = (r_K, b_K, r_V, b_V) replaces the allocator's (r, b) by one pair per side for every head
    (the coordinate order and the bases are still built per head): a measurement case that isolates
    one code shape, not the method's allocation."""
    bpd = w.bpd if bpd is None else bpd
    lam_k = np.stack([s.lam_k for s in stats])
    sq = np.stack([s.sigma2_q for s in stats])
    lam_v = np.stack([s.lam_v for s in stats])
    ak = kvc.kvc_allocate(lam_k, sq, kvc.alloc_opts(bpd, solver))
    av = kvc.kvc_allocate(lam_v, None, kvc.alloc_opts(bpd, kvc.SOLVER_C1_ONLY))
    if measured is not None:  # K side from the exact DP over measured tables (quant, trunc_w, order)
        quant, trunc_w, order = measured
        am = kvc.kvc_allocate_measured(quant, trunc_w, order, kvc.alloc_opts(bpd))
        ak = {"r": am["r"], "b": am["b"], "B": am["B"], "D": am["D"], "order": order}
    if uniform is not None:
        rk, bk, rv, bv = (int(x) for x in uniform)
        for a, r, b in ((ak, rk, bk), (av, rv, bv)):
            a["r"] = np.full_like(a["r"], r)
            a["b"] = np.full_like(a["b"], b)
    sides = []
    for a, lam_key, U_key, sign_key in ((ak, "lam_k", "U_k", "sign_k"), (av, "lam_v", "U_v", "sign_v")):
        Ps, ds = [], []
        for h, s in enumerate(stats):
            P, dl = kvc.kvc_make_basis(getattr(s, U_key), a["order"][h], getattr(s, lam_key), int(a["r"][h]),
                                       int(a["b"][h]), getattr(s, sign_key))
            Ps.append(P)
            ds.append(dl)
        sides.append(SideTables(a["r"], a["b"], a["order"], Ps, np.array(ds, dtype=np.float32)))
    return sides[0], sides[1]


def build_side(side: int, tab: SideTables, w: synth.Workload, capacity: int, device="cuda") -> kvc.Side:
    offs = np.zeros(len(tab.P), dtype=np.int64)
    if len(tab.P) > 1:
        offs[1:] = np.cumsum([p.size for p in tab.P])[:-1]
    flat = np.concatenate([p.reshape(-1) for p in tab.P])
    heads = np.array([w.head_of_unit(u) for u in range(w.n_units)], dtype=np.int64)
    return kvc.Side(side, tab.r[heads], tab.b[heads], tab.delta[heads], flat, offs[heads], capacity, device)


def draw_unit_tokens(w: synth.Workload, stats, side: int, n_tok: int, seed: int, device, units=None):
    """fp16 tokens (len(units), n_tok, d) for the given units, drawn on `device`."""
    import torch
    units = range(w.n_units) if units is None else units
    units = list(units)
    x = torch.empty((len(units), n_tok, w.d), dtype=torch.float16, device=device)
    for k, u in enumerate(units):
        h = w.head_of_unit(u)
        F = stats[h].F_k if side == kvc.SIDE_K else stats[h].F_v
        x[k] = synth.draw_tokens_torch(F, n_tok, (seed, synth.KIND_TOK, side, u), device)
    return x


def draw_queries(w: synth.Workload, stats, seed: int, device, scale: float = 1.0):
    """fp16 queries (n_units, G, d): query head g of unit u from N(0, Sigma_Q,g) of its KV head."""
    import torch
    q = np.zeros((w.n_units, w.group, w.d), dtype=np.float16)
    for u in range(w.n_units):
        h = w.head_of_unit(u)
        rng = synth.rng_for(seed, synth.KIND_QVEC, u)
        for g in range(w.group):
            q[u, g] = (stats[h].F_q[g] @ rng.standard_normal(w.d) * scale).astype(np.float16)
    return torch.as_tensor(q.view(np.int16), device=device).view(torch.float16)


class Cache:
    """A compressed K/V cache for a workload plus its decode buffers."""

    def __init__(self, w: synth.Workload, seed: int = 0, device="cuda", bpd: float | None = None,
                 capacity: int | None = None, solver: int = kvc.SOLVER_DAMPED, stats=None, uniform=None,
                 measured=None):
        import torch
        self.w = w
        self.seed = seed
        self.device = torch.device(device)
        self.stats = calibrate(synth.workload_covs(w, seed), device) if stats is None else stats
        self.k_tab, self.v_tab = allocate_workload(w, self.stats, bpd, solver, uniform, measured)
        self.capacity = w.tokens if capacity is None else capacity
        self.K = build_side(kvc.SIDE_K, self.k_tab, w, self.capacity, device)
        self.V = build_side(kvc.SIDE_V, self.v_tab, w, self.capacity, device)

    def encode(self, xk, xv, t0: int, n_tok: int, stream=None):
        kvc.kvc_encode_kv(self.K, self.V, xk, xv, t0, n_tok, stream)

    def decode_buffers(self, max_seq_len: int):
        import torch
        nbytes = kvc.kvc_decode_attn_workspace(self.K, self.V, self.w.group, max_seq_len)
        ws = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        out = torch.empty((self.w.n_units, self.w.group, self.w.d), dtype=torch.float32, device=self.device)
        return ws, out

    def decode(self, q, seq_len, max_seq_len: int, out, ws, stream=None):
        kvc.kvc_decode_attn(self.K, self.V, q, self.w.group, seq_len, max_seq_len, out, ws, stream)

    def step(self, xk, xv, t_new: int, q, seq_len, max_seq_len: int, out, ws, stream=None):
        """Fused decode step: append (xk, xv) at t_new to every unit, then decode attention."""
        kvc.kvc_decode_step(self.K, self.V, xk, xv, t_new, q, self.w.group, seq_len, max_seq_len, out, ws, stream)

    def layer_sides(self, layer: int):
        """Descriptors of one layer's units (u = (layer * batch + sequence) * kv_heads + head is
        layer-major, so they are one contiguous range) for per-layer calls."""
        upl = self.w.batch * self.w.kv_heads
        return kvc.SideRange(self.K, layer * upl, upl), kvc.SideRange(self.V, layer * upl, upl)

    def code_bytes(self, n_tok: int) -> int:
        """Algorithmic bytes of the K and V code streams holding n_tok tokens per unit."""
        return int(sum(self.K.stream_bytes(u, n_tok) + self.V.stream_bytes(u, n_tok) for u in range(self.w.n_units)))
