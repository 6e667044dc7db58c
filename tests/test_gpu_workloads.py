"""GPU parity on the shapes of the measured workloads, through the C ABI.

* every query-group size the decode kernel is instantiated for (G = 1, 2, 8, 16);
* the 8B-shaped 32-layer, batch-8, 32768-token, 2 bpd workload at full size, in the launch
  configuration bench.py times (append one token, decode over 32769), checked on sampled units;
* the long-context 0.5 bpd shape (131072 tokens; 2 of the 32 layers) and the 70B shape
  (G = 8, 65536 tokens, 1 bpd; 2 of the 80 layers), checked on sampled units;
* the bit-rate sweep (0.5 .. 4 bpd) on a reduced 8B shape: tables, codes, decode outputs and
  reconstruction MSE (GPU vs oracle vs the distortion model D(r, b)) for every unit.

Reduced layer counts keep every per-unit shape (tokens, G, budget) of the full workload; the
allocation then couples fewer heads, which is immaterial for kernel parity. The oracle builds
its own tables, bases and codes from the same seeded fp16 inputs.
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import alloc as oa
from oracle import attention as oatt
from oracle import native as onat
from oracle import quant as oq
from paper_2609_24298_amd import kvc, pipeline, synth

from test_gpu_parity import TOL, OracleTables, normwise, x_bits

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _build(w, T, capacity, seed=0, bpd=None):
    cache = pipeline.Cache(w, seed=seed, bpd=bpd, capacity=capacity)
    xk = pipeline.draw_unit_tokens(w, cache.stats, kvc.SIDE_K, T, seed, "cuda")
    xv = pipeline.draw_unit_tokens(w, cache.stats, kvc.SIDE_V, T, seed, "cuda")
    return cache, xk, xv


def _check_units(w, cache, ot, xk, xv, q, seq, got, units, tag, n_enc):
    """Streams of the n_enc encoded tokens bit-exact; outputs over seq[u] tokens within TOL."""
    worst = 0.0
    for u in units:
        h = w.head_of_unit(u)
        n = int(seq[u])
        res = {}
        for side, S, x in ((kvc.SIDE_K, cache.K, xk), (kvc.SIDE_V, cache.V, xv)):
            r, b = ot.rb(side, h)
            assert (int(S.r_h[u]), int(S.b_h[u])) == (r, b)
            P, dl = ot.basis(side, h)
            codes = onat.encode_codes(P, dl, b, x_bits(x[u][:n_enc]))
            exp = onat.pack(codes, r, b, side)
            assert np.array_equal(S.unit_codes(u, n_enc).cpu().numpy(), exp), (tag, side, u)
            res[side] = (codes[:n], P, dl, b)
        (ck, Pk, dk, bk), (cv, Pv, dv, bv) = res[kvc.SIDE_K], res[kvc.SIDE_V]
        qb = q[u].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        ref = oatt.decode_attention(ck, cv, Pk, Pv, dk, dv, bk, bv, qb, n)
        for g in range(w.group):
            e = normwise(got[u, g], ref[g])
            worst = max(worst, e)
            assert e <= TOL, (tag, u, g, e)
    log(f"[{tag}] units {list(units)}: codes bit-exact, max normwise error {worst:.2e}")


@pytest.mark.parametrize("G", [1, 2, 8, 16])
def test_decode_every_group_size(G):
    w = synth.Workload(f"g{G}", layers=1, kv_heads=2, group=G, batch=2, tokens=1000, bpd=2.0)
    log(f"[G={G}] build")
    cache, xk, xv = _build(w, w.tokens, w.tokens)
    cache.encode(xk, xv, 0, w.tokens)
    ot = OracleTables(w, cache.stats)
    q = pipeline.draw_queries(w, cache.stats, 3, "cuda", scale=4.0)
    seq = np.array([1000, 777, 64, 1][: w.n_units], dtype=np.int32)
    ws, out = cache.decode_buffers(w.tokens)
    cache.decode(q, torch.as_tensor(seq, device="cuda"), w.tokens, out, ws)
    torch.cuda.synchronize()
    _check_units(w, cache, ot, xk, xv, q, seq, out.cpu().numpy(), range(w.n_units), f"G={G}", w.tokens)


@pytest.mark.parametrize("G", [1, 4, 8, 16])
def test_decode_many_chunks_every_group_size(G):
    # two units over 65 tiles: the context splits into more than 32 chunks, so the combine runs with
    # its widest block for the group size (8 wavefronts for G <= 4, 4 for G = 8, 2 for G = 16) and the
    # query projection on eight wavefronts per unit
    w = synth.Workload(f"chunks_g{G}", layers=1, kv_heads=1, group=G, batch=2, tokens=4100, bpd=2.0)
    log(f"[chunks G={G}] build")
    cache, xk, xv = _build(w, w.tokens, w.tokens)
    cache.encode(xk, xv, 0, w.tokens)
    ot = OracleTables(w, cache.stats)
    q = pipeline.draw_queries(w, cache.stats, 5, "cuda", scale=6.0)
    seq = np.array([4100, 2345], dtype=np.int32)
    ws, out = cache.decode_buffers(w.tokens)
    cache.decode(q, torch.as_tensor(seq, device="cuda"), w.tokens, out, ws)
    torch.cuda.synchronize()
    _check_units(w, cache, ot, xk, xv, q, seq, out.cpu().numpy(), range(w.n_units), f"chunks G={G}", w.tokens)


def _sampled_full(w, T, units, seed=0, qscale=1.0):
    """Bench launch configuration: encode T tokens, append one, decode over T + 1; check `units`."""
    log(f"[{w.name}] build cache + draw {2 * w.n_units * T} tokens")
    cache, xk, xv = _build(w, T + 1, T + kvc.TILE, seed)
    cache.encode(xk, xv, 0, T)  # rows past T are not read
    cache.encode(xk[:, T:T + 1].contiguous(), xv[:, T:T + 1].contiguous(), T, 1)
    q = pipeline.draw_queries(w, cache.stats, seed + 1, "cuda", scale=qscale)
    seq = np.full(w.n_units, T + 1, dtype=np.int32)
    ws, out = cache.decode_buffers(T + 1)
    log(f"[{w.name}] decode")
    cache.decode(q, torch.as_tensor(seq, device="cuda"), T + 1, out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert np.isfinite(got).all()
    ot = OracleTables(w, cache.stats)
    _check_units(w, cache, ot, xk, xv, q, seq, got, units, w.name, T + 1)


def test_bench_workload_sampled_parity():
    w = synth.WORKLOADS["llama8b_b8_t32k_2bpd"]
    _sampled_full(w, w.tokens, [0, 777, w.n_units - 1])


def test_long_context_half_bpd_sampled_parity():
    w0 = synth.WORKLOADS["llama8b_b1_t128k_0.5bpd"]
    w = synth.Workload("llama8b_b1_t128k_0.5bpd_2layers", 2, w0.kv_heads, w0.group, w0.batch, w0.tokens, w0.bpd)
    _sampled_full(w, w.tokens, [3, w.n_units - 2], qscale=4.0)


def test_70b_shape_sampled_parity():
    w0 = synth.WORKLOADS["llama70b_b4_t64k_1bpd"]
    w = synth.Workload("llama70b_b4_t64k_1bpd_2layers", 2, w0.kv_heads, w0.group, w0.batch, w0.tokens, w0.bpd)
    _sampled_full(w, w.tokens, [5, w.n_units - 1])


@pytest.mark.parametrize("bpd", [0.5, 1.0, 2.0, 3.0, 4.0])
def test_bitrate_sweep_parity_and_mse(bpd):
    w = synth.Workload(f"sweep_{bpd}", layers=1, kv_heads=8, group=4, batch=2, tokens=1100, bpd=bpd)
    cache, xk, xv = _build(w, w.tokens, w.tokens, bpd=bpd)
    cache.encode(xk, xv, 0, w.tokens)
    ot = OracleTables(w, cache.stats, bpd=bpd)
    for side, tab, a in ((kvc.SIDE_K, cache.k_tab, ot.ak), (kvc.SIDE_V, cache.v_tab, ot.av)):
        assert np.array_equal(tab.r, a["r"]) and np.array_equal(tab.b, a["b"]), (bpd, side)
    q = pipeline.draw_queries(w, cache.stats, 5, "cuda", scale=2.0)
    seq = np.full(w.n_units, w.tokens, dtype=np.int32)
    ws, out = cache.decode_buffers(w.tokens)
    cache.decode(q, torch.as_tensor(seq, device="cuda"), w.tokens, out, ws)
    torch.cuda.synchronize()
    _check_units(w, cache, ot, xk, xv, q, seq, out.cpu().numpy(), range(w.n_units), f"sweep {bpd}", w.tokens)
    # reconstruction MSE per unit and side: GPU, oracle and the model D(r, b) / d
    for side, S, x in ((kvc.SIDE_K, cache.K, xk), (kvc.SIDE_V, cache.V, xv)):
        rec = torch.empty((w.n_units, w.tokens, w.d), dtype=torch.float32, device="cuda")
        kvc.kvc_reconstruct(S, 0, w.tokens, rec)
        torch.cuda.synchronize()
        rec = rec.cpu().numpy().astype(np.float64)
        xs = x.float().cpu().numpy().astype(np.float64)
        rows = []
        for u in range(w.n_units):
            h = w.head_of_unit(u)
            r, b = ot.rb(side, h)
            P, dl = ot.basis(side, h)
            codes = onat.encode_codes(P, dl, b, x_bits(x[u]))
            ref = oatt.reconstruct(codes, P, dl, b)
            mse_gpu = float(np.mean((rec[u] - xs[u]) ** 2))
            mse_orc = float(np.mean((ref - xs[u]) ** 2))
            st = cache.stats[h]
            lam = st.lam_k if side == kvc.SIDE_K else st.lam_v
            a = ot.ak if side == kvc.SIDE_K else ot.av
            lam_o = lam[a["order"][h]]
            model = (np.sum(lam_o[r:]) + oq.q_model(b) * np.sum(lam_o[:r])) / w.d
            assert abs(mse_gpu - mse_orc) <= 1e-5 * mse_orc + 1e-12, (bpd, side, u, mse_gpu, mse_orc)
            rows.append((r, b, mse_gpu, mse_orc, model))
        m = np.array([row[2:] for row in rows])
        log(f"[sweep {bpd}] side {'KV'[side]}: mean MSE gpu {m[:, 0].mean():.4e} oracle {m[:, 1].mean():.4e} "
            f"model D/d {m[:, 2].mean():.4e}; (r,b) {sorted(set((r, b) for r, b, *_ in rows))}")
