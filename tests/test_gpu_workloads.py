"""GPU parity on the shapes of the measured workloads, through the C ABI.

* every query-group size the decode kernel is instantiated for (G = 1, 2, 8, 16);
* the 8B-shaped 32-layer, batch-8, 32768-token, 2 bpd workload at full size, in the launch
  configuration bench.py times (append one token, decode over 32769), checked on sampled units;
* the long-context 0.5 bpd workload at full size (32 layers, 131072 tokens) and the 70B shape
  (G = 8, 65536 tokens, 1 bpd; 2 of the 80 layers), checked on sampled units;
* peaky attention on the sampled units of those launches and of G = 1 and 16 over long chunks:
  planted sink keys 12 and 16 nats above every other logit, and queries scaled to a logit
  standard deviation of 1, 2 and 4 nats;
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

from oracle_stats import oracle_stats
from test_gpu_parity import TOL, OracleTables, normwise, x_bits

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _build(w, T, capacity, seed=0, bpd=None):
    cache = pipeline.Cache(w, seed=seed, bpd=bpd, capacity=capacity, stats=oracle_stats(w, seed))
    xk = pipeline.draw_unit_tokens(w, cache.stats, kvc.SIDE_K, T, seed, "cuda")
    xv = pipeline.draw_unit_tokens(w, cache.stats, kvc.SIDE_V, T, seed, "cuda")
    return cache, xk, xv


def _oracle_units(w, cache, ot, xk, xv, units, tag, n_enc):
    """The oracle's codes of the n_enc encoded tokens of each unit, checked bit-exact against the
    GPU streams on the way: {u: (codes_K, P_K, step_K, b_K, codes_V, P_V, step_V, b_V)}."""
    data = {}
    for u in units:
        h = w.head_of_unit(u)
        res = {}
        for side, S, x in ((kvc.SIDE_K, cache.K, xk), (kvc.SIDE_V, cache.V, xv)):
            r, b = ot.rb(side, h)
            assert (int(S.r_h[u]), int(S.b_h[u])) == (r, b)
            P, dl = ot.basis(side, h)
            codes = onat.encode_codes(P, dl, b, x_bits(x[u][:n_enc]))
            exp = onat.pack(codes, r, b, side)
            assert np.array_equal(S.unit_codes(u, n_enc).cpu().numpy(), exp), (tag, side, u)
            res[side] = (codes, P, dl, b)
        data[u] = res[kvc.SIDE_K] + res[kvc.SIDE_V]
    return data


def q_bits_of(q, u):
    return q[u].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def _check_outputs(data, q, seq, got, tag, G):
    """Outputs of the units in `data` over seq[u] tokens within TOL of the oracle's fp64 decode."""
    worst = 0.0
    for u, (ck, Pk, dk, bk, cv, Pv, dv, bv) in data.items():
        n = int(seq[u])
        ref = oatt.decode_attention(ck, cv, Pk, Pv, dk, dv, bk, bv, q_bits_of(q, u), n)
        for g in range(G):
            e = normwise(got[u, g], ref[g])
            worst = max(worst, e)
            assert e <= TOL, (tag, u, g, e)
    log(f"[{tag}] units {list(data)}: max normwise error {worst:.2e}")
    return worst


def _check_units(w, cache, ot, xk, xv, q, seq, got, units, tag, n_enc):
    """Streams of the n_enc encoded tokens bit-exact; outputs over seq[u] tokens within TOL."""
    data = _oracle_units(w, cache, ot, xk, xv, units, tag, n_enc)
    _check_outputs(data, q, seq, got, tag, w.group)
    log(f"[{tag}] codes bit-exact")
    return data


# ---------------------------------------------------------------- peaky attention
#
# Flat attention over a long context is a weak test of the softmax: every weight is close to the
# largest. Two constructions make it peaky on the units that are checked:
#  * sink keys: for query head g a seeded sign pattern s over the K rank coordinates; the key at
#    position pos_g is replaced by P_K^T (2^(b-1) step s), whose codes saturate along s, and the query
#    by kappa P_K^T s, with kappa chosen (from the oracle's logits) so that this key's logit is `gap`
#    nats above the largest logit of every other token;
#  * a query-scale sweep: every query multiplied by one factor that puts the median logit standard
#    deviation of the checked heads at 1, 2 or 4 nats.

def sink_positions(T, G):
    return [(g * T) // G + 3 for g in range(G)]


def plant_sink_keys(w, ot, xk, units, T, seed):
    """Writes the sink keys into xk (device fp16) for `units`; returns {u: sign patterns (G x r_K)}."""
    signs = {}
    for u in units:
        h = w.head_of_unit(u)
        rk, bk = ot.rb(kvc.SIDE_K, h)
        Pk, dk = ot.basis(kvc.SIDE_K, h)
        P = oatt.fp16_to_f64(Pk)
        rng = np.random.default_rng([seed, 77, u])
        sg = rng.integers(0, 2, (w.group, rk)) * 2.0 - 1.0
        for g, pos in enumerate(sink_positions(T, w.group)):
            key = (P.T @ (sg[g] * float(2 ** (bk - 1)) * float(dk))).astype(np.float16)
            xk[u, pos] = torch.as_tensor(key.view(np.int16), device=xk.device).view(torch.float16)
        signs[u] = sg
    return signs


def sink_queries(w, data, signs, q, T, gap):
    """q with the checked units' heads replaced by kappa P_K^T s (see above); logs the achieved gaps."""
    qs = q.clone()
    stats = []
    for u, (ck, Pk, dk, bk, *_rest) in data.items():
        P = oatt.fp16_to_f64(Pk)
        pos = sink_positions(T, w.group)
        base = (signs[u] @ P).astype(np.float64)               # G x d: P_K^T s per head
        s1 = oatt.decode_logits(ck, Pk, dk, bk, base.astype(np.float16).view(np.uint16), T)
        for g in range(w.group):
            rest = np.delete(s1[g], pos[g])
            g1 = s1[g, pos[g]] - rest.max()
            assert g1 > 0, (u, g, g1)
            kappa = gap / g1
            qs[u, g] = torch.as_tensor((kappa * base[g]).astype(np.float16).view(np.int16),
                                       device=q.device).view(torch.float16)
        s = oatt.decode_logits(ck, Pk, dk, bk, q_bits_of(qs, u), T)
        for g in range(w.group):
            rest = np.delete(s[g], pos[g])
            stats.append((s[g, pos[g]] - rest.max(), rest.std()))
    st = np.array(stats)
    log(f"[sink gap {gap}] achieved gap over the rest {st[:, 0].min():.2f}..{st[:, 0].max():.2f} nats, "
        f"tail logit std {st[:, 1].min():.2f}..{st[:, 1].max():.2f}")
    return qs


def logit_std(data, q, T, G):
    return float(np.median([oatt.decode_logits(ck, Pk, dk, bk, q_bits_of(q, u), T).std(axis=1)
                            for u, (ck, Pk, dk, bk, *_r) in data.items()]))


def _peaky_checks(w, cache, data, q, seq, n_att, ws, out, signs, T_sink, tag):
    """Query-scale sweep and sink keys on the checked units, in the launch configuration of `seq`."""
    std1 = logit_std(data, q, n_att, w.group)
    for target in (1.0, 2.0, 4.0):
        qs = (q.float() * (target / std1)).to(torch.float16)
        cache.decode(qs, torch.as_tensor(seq, device="cuda"), n_att, out, ws)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        assert np.isfinite(got).all()
        log(f"[{tag}] logit std {logit_std(data, qs, n_att, w.group):.2f} nats (target {target})")
        _check_outputs(data, qs, seq, got, f"{tag} logit std {target}", w.group)
    for gap in (12.0, 16.0):
        qs = sink_queries(w, data, signs, q, n_att, gap)
        cache.decode(qs, torch.as_tensor(seq, device="cuda"), n_att, out, ws)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        assert np.isfinite(got).all()
        _check_outputs(data, qs, seq, got, f"{tag} sink +{gap}", w.group)


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


def _sampled_full(w, T, units, seed=0, qscale=1.0, peaky=False):
    """Bench launch configuration: encode T tokens, append one, decode over T + 1; check `units`.
    peaky: sink keys planted in the checked units, then the query-scale sweep and the sink queries
    decoded in the same launch configuration (every unit attends over T + 1 tokens)."""
    log(f"[{w.name}] build cache + draw {2 * w.n_units * T} tokens")
    cache, xk, xv = _build(w, T + 1, T + kvc.TILE, seed)
    ot = OracleTables(w, cache.stats)
    signs = plant_sink_keys(w, ot, xk, units, T + 1, seed) if peaky else None
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
    data = _check_units(w, cache, ot, xk, xv, q, seq, got, units, w.name, T + 1)
    if peaky:
        _peaky_checks(w, cache, data, q, seq, T + 1, ws, out, signs, T + 1, w.name)


def test_bench_workload_sampled_parity():
    # 2048 units at 32768 tokens: few long context chunks per unit (the split the bench times)
    w = synth.WORKLOADS["llama8b_b8_t32k_2bpd"]
    _sampled_full(w, w.tokens, [0, 777, w.n_units - 1], peaky=True)


def test_long_context_half_bpd_sampled_parity():
    # the whole 32-layer, 131072-token workload (256 units, chunks of ~10^4 tokens)
    w = synth.WORKLOADS["llama8b_b1_t128k_0.5bpd"]
    _sampled_full(w, w.tokens, [3, w.n_units - 2], qscale=4.0, peaky=True)


def test_70b_shape_sampled_parity():
    w0 = synth.WORKLOADS["llama70b_b4_t64k_1bpd"]
    w = synth.Workload("llama70b_b4_t64k_1bpd_2layers", 2, w0.kv_heads, w0.group, w0.batch, w0.tokens, w0.bpd)
    _sampled_full(w, w.tokens, [5, w.n_units - 1], peaky=True)


@pytest.mark.parametrize("G,T,bpd", [(16, 32768, 2.0), (1, 131072, 1.0)])
def test_peaky_attention_long_chunks_other_group_sizes(G, T, bpd):
    # 256 units, so the context splits into few long chunks, with the general-width partials kernel
    w = synth.Workload(f"peaky_g{G}_t{T}", 32, 8, G, 1, T, bpd)
    _sampled_full(w, T, [1, 200], peaky=True)


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
