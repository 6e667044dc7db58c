"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Codes and streams: bit-exact. Attention outputs and reconstructions: max
normwise relative error <= 2e-3 per (unit, query head), i.e.
max|out - ref| / max|ref| (fp32 accumulation from fp16 inputs).
The oracle never sees a value the GPU produced: it builds its own tables,
bases and codes from the same seeded fp16 inputs.
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import alloc as oa
from oracle import attention as oatt
from oracle import basis as ob
from oracle import native as onat
from paper_2609_24298_amd import kvc, pipeline, synth

from oracle_stats import oracle_stats

pytestmark = pytest.mark.gpu
TOL = 2e-3


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def normwise(out, ref):
    out = np.asarray(out, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return np.max(np.abs(out - ref)) / max(np.max(np.abs(ref)), 1e-30)


class OracleTables:
    """The oracle's own allocation and bases for a workload (same rules as the library)."""

    def __init__(self, w, stats, bpd=None, solver=oa.SOLVER_DAMPED):
        bpd = w.bpd if bpd is None else bpd
        lam_k = np.stack([s.lam_k for s in stats])
        sq = np.stack([s.sigma2_q for s in stats])
        lam_v = np.stack([s.lam_v for s in stats])
        self.ak = oa.allocate(lam_k, sq, oa.AllocOpts(bpd=bpd, solver=solver))
        self.av = oa.allocate(lam_v, None, oa.AllocOpts(bpd=bpd, solver=oa.SOLVER_C1_ONLY))
        self.stats = stats
        self._bases = {}

    def basis(self, side, h):
        key = (side, h)
        if key not in self._bases:
            a = self.ak if side == kvc.SIDE_K else self.av
            s = self.stats[h]
            U, lam, sign = (s.U_k, s.lam_k, s.sign_k) if side == kvc.SIDE_K else (s.U_v, s.lam_v, s.sign_v)
            self._bases[key] = ob.make_basis(U, a["order"][h], lam, int(a["r"][h]), int(a["b"][h]), sign)
        return self._bases[key]

    def rb(self, side, h):
        a = self.ak if side == kvc.SIDE_K else self.av
        return int(a["r"][h]), int(a["b"][h])


def x_bits(x_unit):
    return x_unit.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


@pytest.fixture(scope="module")
def small():
    w = synth.WORKLOADS["small_l1_h8_t4k"]
    log("[small] build cache", w)
    cache = pipeline.Cache(w, seed=0, stats=oracle_stats(w, 0))
    xk = pipeline.draw_unit_tokens(w, cache.stats, kvc.SIDE_K, w.tokens, 0, "cuda")
    xv = pipeline.draw_unit_tokens(w, cache.stats, kvc.SIDE_V, w.tokens, 0, "cuda")
    cache.encode(xk, xv, 0, w.tokens)
    torch.cuda.synchronize()
    ot = OracleTables(w, cache.stats)
    return w, cache, xk, xv, ot


def test_small_tables_match_oracle(small):
    w, cache, _, _, ot = small
    for side, tab, a in ((kvc.SIDE_K, cache.k_tab, ot.ak), (kvc.SIDE_V, cache.v_tab, ot.av)):
        assert np.array_equal(tab.r, a["r"]) and np.array_equal(tab.b, a["b"])
        for h in range(w.n_heads):
            P, dl = ot.basis(side, h)
            assert np.array_equal(tab.P[h], P) and np.float32(tab.delta[h]) == np.float32(dl)


def test_small_encode_streams_bit_exact(small):
    w, cache, xk, xv, ot = small
    for side, S, x in ((kvc.SIDE_K, cache.K, xk), (kvc.SIDE_V, cache.V, xv)):
        for u in range(w.n_units):
            h = w.head_of_unit(u)
            r, b = ot.rb(side, h)
            P, dl = ot.basis(side, h)
            log(f"[small] encode parity side={side} unit={u} r={r} b={b}")
            codes = onat.encode_codes(P, dl, b, x_bits(x[u]))
            exp = onat.pack(codes, r, b, side)
            got = S.unit_codes(u, w.tokens).cpu().numpy()
            assert np.array_equal(got, exp), (side, u, int(np.sum(got != exp)))


def _oracle_decode(w, ot, cache, xk, xv, q, seq):
    outs = np.zeros((w.n_units, w.group, w.d))
    for u in range(w.n_units):
        h = w.head_of_unit(u)
        (rk, bk), (rv, bv) = ot.rb(kvc.SIDE_K, h), ot.rb(kvc.SIDE_V, h)
        Pk, dk = ot.basis(kvc.SIDE_K, h)
        Pv, dv = ot.basis(kvc.SIDE_V, h)
        ck = onat.encode_codes(Pk, dk, bk, x_bits(xk[u][: seq[u]]))
        cv = onat.encode_codes(Pv, dv, bv, x_bits(xv[u][: seq[u]]))
        qb = q[u].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        outs[u] = oatt.decode_attention(ck, cv, Pk, Pv, dk, dv, bk, bv, qb, int(seq[u]))
    return outs


@pytest.mark.parametrize("qscale", [1.0, 8.0])
def test_small_decode_attention_parity(small, qscale):
    w, cache, xk, xv, ot = small
    q = pipeline.draw_queries(w, cache.stats, 1, "cuda", scale=qscale)
    seq = np.array([w.tokens] * w.n_units, dtype=np.int32)
    ws, out = cache.decode_buffers(w.tokens)
    log(f"[small] decode qscale={qscale}")
    cache.decode(q, torch.as_tensor(seq, device="cuda"), w.tokens, out, ws)
    got = out.cpu().numpy()
    ref = _oracle_decode(w, ot, cache, xk, xv, q, seq)
    worst = 0.0
    for u in range(w.n_units):
        for g in range(w.group):
            e = normwise(got[u, g], ref[u, g])
            worst = max(worst, e)
            assert e <= TOL, (u, g, e)
    log(f"[small] decode qscale={qscale}: max normwise error {worst:.2e}")


def test_small_decode_ragged_lengths(small):
    w, cache, xk, xv, ot = small
    q = pipeline.draw_queries(w, cache.stats, 2, "cuda", scale=4.0)
    seq = np.array([1, 63, 64, 65, 1000, 4095, 4096, 2049], dtype=np.int32)
    ws, out = cache.decode_buffers(w.tokens)
    log("[small] decode ragged", seq.tolist())
    cache.decode(q, torch.as_tensor(seq, device="cuda"), w.tokens, out, ws)
    got = out.cpu().numpy()
    ref = _oracle_decode(w, ot, cache, xk, xv, q, seq)
    for u in range(w.n_units):
        for g in range(w.group):
            assert normwise(got[u, g], ref[u, g]) <= TOL, (u, g, seq[u])
    # a single attended token returns its reconstructed value
    u = 0
    h = w.head_of_unit(u)
    Pv, dv = ot.basis(kvc.SIDE_V, h)
    rv, bv = ot.rb(kvc.SIDE_V, h)
    cv = onat.encode_codes(Pv, dv, bv, x_bits(xv[u][:1]))
    v0 = oatt.reconstruct(cv, Pv, dv, bv)[0]
    for g in range(w.group):
        assert normwise(got[u, g], v0) <= 1e-5


def test_small_decode_clamps_lengths(small):
    # seq_len is device data: 0 (or negative) attends to nothing and gives zeros, values past max_seq_len
    # attend to max_seq_len tokens
    w, cache, xk, xv, ot = small
    q = pipeline.draw_queries(w, cache.stats, 4, "cuda", scale=4.0)
    n_max = 700
    seq = np.array([0, -5, n_max + 50, n_max, 1, 3, 64, 129][: w.n_units], dtype=np.int32)
    ws, out = cache.decode_buffers(n_max)
    cache.decode(q, torch.as_tensor(seq, device="cuda"), n_max, out, ws)
    got = out.cpu().numpy()
    assert np.all(got[0] == 0.0) and np.all(got[1] == 0.0)
    eff = np.clip(seq, 0, n_max)
    ref = _oracle_decode(w, ot, cache, xk, xv, q, np.maximum(eff, 1))
    for u in range(2, w.n_units):
        for g in range(w.group):
            assert normwise(got[u, g], ref[u, g]) <= TOL, (u, g, seq[u])


def test_small_decode_is_deterministic(small):
    w, cache, _, _, _ = small
    q = pipeline.draw_queries(w, cache.stats, 3, "cuda")
    seq = torch.full((w.n_units,), w.tokens, dtype=torch.int32, device="cuda")
    ws, out1 = cache.decode_buffers(w.tokens)
    cache.decode(q, seq, w.tokens, out1, ws)
    out2 = torch.empty_like(out1)
    ws.fill_(0xAB)
    cache.decode(q, seq, w.tokens, out2, ws)
    assert torch.equal(out1, out2)


def test_small_reconstruct_parity(small):
    w, cache, xk, xv, ot = small
    t0, n = 37, 700
    for side, S in ((kvc.SIDE_K, cache.K), (kvc.SIDE_V, cache.V)):
        out = torch.empty((w.n_units, n, w.d), dtype=torch.float32, device="cuda")
        log(f"[small] reconstruct side={side}")
        kvc.kvc_reconstruct(S, t0, n, out)
        got = out.cpu().numpy()
        x = xk if side == kvc.SIDE_K else xv
        for u in range(w.n_units):
            h = w.head_of_unit(u)
            r, b = ot.rb(side, h)
            P, dl = ot.basis(side, h)
            codes = onat.encode_codes(P, dl, b, x_bits(x[u][t0:t0 + n]))
            ref = oatt.reconstruct(codes, P, dl, b)
            assert normwise(got[u], ref) <= 1e-5, (side, u)


def test_encode_append_ragged_pieces(small):
    # appending in ragged pieces reproduces the one-shot stream (read-modify-write of partial tiles)
    w, cache, xk, xv, _ = small
    T = 1000
    K2 = pipeline.build_side(kvc.SIDE_K, cache.k_tab, w, T)
    V2 = pipeline.build_side(kvc.SIDE_V, cache.v_tab, w, T)
    for a, e in ((0, 1), (1, 63), (63, 64), (64, 200), (200, 333), (333, 1000)):
        xs_k = xk[:, a:e].contiguous()
        xs_v = xv[:, a:e].contiguous()
        kvc.kvc_encode(K2, xs_k, a, e - a)
        kvc.kvc_encode(V2, xs_v, a, e - a)
    torch.cuda.synchronize()
    for u in range(w.n_units):
        for S2, S in ((K2, cache.K), (V2, cache.V)):
            n_full = T // 64 * 64
            got = S2.unit_codes(u, T).cpu().numpy()
            ref_full = S.unit_codes(u, w.tokens).cpu().numpy()
            # whole tiles are identical; the last partial tile holds the same codes for t < T
            nb = S.stream_bytes(u, n_full)
            assert np.array_equal(got[:nb], ref_full[:nb])
            r, b = int(S.r_h[u]), int(S.b_h[u])
            c2 = onat.unpack(got, T, r, b, S.side)
            c1 = onat.unpack(ref_full, T, r, b, S.side)
            assert np.array_equal(c1, c2)


def test_encode_kv_equals_per_side_encode(small):
    # both sides in one call (one launch for the append path, the bulk encoder beyond) write exactly the
    # bytes of two per-side kvc_encode calls, piece by piece
    w, cache, xk, xv, _ = small
    T = 300
    K1, V1 = (pipeline.build_side(s, t, w, T) for s, t in ((kvc.SIDE_K, cache.k_tab), (kvc.SIDE_V, cache.v_tab)))
    K2, V2 = (pipeline.build_side(s, t, w, T) for s, t in ((kvc.SIDE_K, cache.k_tab), (kvc.SIDE_V, cache.v_tab)))
    for a, e in ((0, 1), (1, 3), (3, 7), (7, 64), (64, 67), (67, 200), (200, 204), (204, 300)):
        xs_k, xs_v = xk[:, a:e].contiguous(), xv[:, a:e].contiguous()
        kvc.kvc_encode(K1, xs_k, a, e - a)
        kvc.kvc_encode(V1, xs_v, a, e - a)
        kvc.kvc_encode_kv(K2, V2, xs_k, xs_v, a, e - a)
    torch.cuda.synchronize()
    for S1, S2 in ((K1, K2), (V1, V2)):
        assert torch.equal(S1.codes, S2.codes)


def _custom_side(side, Ps, deltas, rs, bs, capacity):
    flat = np.concatenate([p.reshape(-1) for p in Ps])
    offs = np.concatenate([[0], np.cumsum([p.size for p in Ps])[:-1]]).astype(np.int64)
    return kvc.Side(side, rs, bs, deltas, flat, offs, capacity)


@pytest.mark.parametrize("side", [kvc.SIDE_K, kvc.SIDE_V])
def test_encode_every_rank_and_width(side):
    rng = np.random.default_rng(10 + side)
    combos = [(r, b) for b in range(1, 9) for r in (2, 4, 6, 14, 16, 18, 30, 50, 64, 66, 98, 126, 128)]
    Ps, ds, rs, bs = [], [], [], []
    for r, b in combos:
        Q, _ = np.linalg.qr(rng.standard_normal((128, 128)))
        Ps.append(Q[:r].astype(np.float16).view(np.uint16))
        ds.append(np.float32(rng.uniform(0.3, 1.2) * 1.596 / 2 ** (b - 1)))
        rs.append(r)
        bs.append(b)
    T = 130
    S = _custom_side(side, Ps, np.array(ds, np.float32), rs, bs, T)
    x = (rng.standard_normal((len(combos), T, 128)) * rng.uniform(0.1, 4, (len(combos), 1, 1))).astype(np.float16)
    xt = torch.as_tensor(x.view(np.int16), device="cuda").view(torch.float16)
    log(f"[sweep] side={side} units={len(combos)}")
    kvc.kvc_encode(S, xt, 0, T)
    torch.cuda.synchronize()
    for u, (r, b) in enumerate(combos):
        codes = onat.encode_codes(Ps[u], ds[u], b, x[u].view(np.uint16))
        exp = onat.pack(codes, r, b, side)
        got = S.unit_codes(u, T).cpu().numpy()
        assert np.array_equal(got, exp), (r, b, int(np.sum(got != exp)))


@pytest.mark.parametrize("side", [kvc.SIDE_K, kvc.SIDE_V])
def test_append_few_tokens_every_rank_and_width(side):
    # appends of 1..4 tokens (the decode-step path) across a tile boundary equal the oracle's stream
    rng = np.random.default_rng(20 + side)
    combos = [(r, b) for b in range(1, 9) for r in (2, 6, 16, 18, 34, 62, 96, 126, 128)]
    Ps, ds, rs, bs = [], [], [], []
    for r, b in combos:
        Q, _ = np.linalg.qr(rng.standard_normal((128, 128)))
        Ps.append(Q[:r].astype(np.float16).view(np.uint16))
        ds.append(np.float32(rng.uniform(0.3, 1.2) * 1.596 / 2 ** (b - 1)))
        rs.append(r)
        bs.append(b)
    T = 75
    S = _custom_side(side, Ps, np.array(ds, np.float32), rs, bs, T)
    x = (rng.standard_normal((len(combos), T, 128)) * rng.uniform(0.1, 4, (len(combos), 1, 1))).astype(np.float16)
    xt = torch.as_tensor(x.view(np.int16), device="cuda").view(torch.float16)
    log(f"[append] side={side} units={len(combos)}")
    a, k = 0, 0
    while a < T:
        n = min(1 + k % 4, T - a)
        kvc.kvc_encode(S, xt[:, a:a + n].contiguous(), a, n)
        a, k = a + n, k + 1
    torch.cuda.synchronize()
    for u, (r, b) in enumerate(combos):
        codes = onat.encode_codes(Ps[u], ds[u], b, x[u].view(np.uint16))
        exp = onat.pack(codes, r, b, side)
        got = S.unit_codes(u, T).cpu().numpy()
        assert np.array_equal(got, exp), (r, b, int(np.sum(got != exp)))


def test_encode_exact_thresholds_and_subnormals():
    # dyadic basis, power-of-two step and dyadic inputs put many projections exactly on
    # quantizer thresholds: the fp32 path cannot decide them, the exact path must
    rng = np.random.default_rng(5)
    r, b, T = 16, 6, 256
    P = (rng.integers(-4, 5, (r, 128)) / 16.0).astype(np.float16)
    x = (rng.integers(-8, 9, (1, T, 128)) / 2.0).astype(np.float16)
    x[0, ::7, ::3] = np.float16(2.0 ** -20)          # subnormal fp16 inputs
    x[0, 5] = 0
    step = np.float32(0.25)
    S = _custom_side(kvc.SIDE_K, [P.view(np.uint16)], np.array([step]), [r], [b], T)
    xt = torch.as_tensor(x.view(np.int16), device="cuda").view(torch.float16)
    kvc.kvc_encode(S, xt, 0, T)
    S1 = _custom_side(kvc.SIDE_K, [P.view(np.uint16)], np.array([step]), [r], [b], T)
    for a in range(0, T, 3):  # the few-token append path decides the same ties
        n = min(3, T - a)
        kvc.kvc_encode(S1, xt[:, a:a + n].contiguous(), a, n)
    torch.cuda.synchronize()
    codes = onat.encode_codes(P.view(np.uint16), step, b, x[0].view(np.uint16))
    y = x[0].astype(np.float64) @ P.astype(np.float64).T
    assert np.mean(np.abs(y / 0.25 - np.round(y / 0.25)) < 1e-12) > 0.05     # many exact ties exercised
    exp = onat.pack(codes, r, b, kvc.SIDE_K)
    assert np.array_equal(S.unit_codes(0, T).cpu().numpy(), exp)
    assert np.array_equal(S1.unit_codes(0, T).cpu().numpy(), exp)


def test_invalid_arguments_raise_before_launch(small):
    w, cache, xk, _, _ = small
    with pytest.raises(kvc.KvcError) as ei:
        kvc.kvc_encode(cache.K, xk, w.tokens - 10, 11)          # beyond capacity
    assert ei.value.code == kvc.KVC_ENOSPACE
    q = pipeline.draw_queries(w, cache.stats, 1, "cuda")
    seq = torch.full((w.n_units,), w.tokens, dtype=torch.int32, device="cuda")
    ws, out = cache.decode_buffers(w.tokens)
    with pytest.raises(kvc.KvcError) as ei:
        kvc.kvc_decode_attn(cache.K, cache.V, q, w.group, seq, w.tokens, out, ws[: ws.numel() - 256])
    assert ei.value.code == kvc.KVC_ENOSPACE
    # the C ABI itself rejects an unsupported group size (the binding's shape checks are bypassed)
    import ctypes
    rc = kvc.lib().kvc_decode_attn(ctypes.byref(cache.K.desc), ctypes.byref(cache.V.desc),
                                   ctypes.c_void_p(q.data_ptr()), 3, ctypes.c_void_p(seq.data_ptr()), w.tokens,
                                   ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ws.data_ptr()), ws.numel(), None)
    assert rc == kvc.KVC_EUNSUPPORTED
    rc = kvc.lib().kvc_decode_attn(ctypes.byref(cache.K.desc), ctypes.byref(cache.V.desc),
                                   ctypes.c_void_p(q.data_ptr()), w.group, ctypes.c_void_p(seq.data_ptr()),
                                   w.tokens + 1, ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ws.data_ptr()),
                                   ws.numel(), None)
    assert rc == kvc.KVC_ENOSPACE
