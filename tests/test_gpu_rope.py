"""GPU parity of RoPE-aware decode attention (kvc_decode_attn_rope) against the oracle's fp64
decode_attention_rope: the keys' codes hold pre-RoPE keys, the kernel reconstructs them, rotates each at
its stream index and scores the rotated query. Every query-group size, ragged lengths, both common
rotary bases, one layer of the 8B-shaped 32k workload, and every pair of code widths (the 512-unit
table of test_gpu_widths)."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import attention as oatt
from oracle import native as onat
from paper_2609_24298_amd import kvc, pipeline, synth

from oracle_stats import oracle_stats
from test_gpu_parity import TOL, OracleTables, normwise, x_bits

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _run(w, T, seq, base, q_scale=1.0, units=None, seed=5):
    st = oracle_stats(w, seed)
    cache = pipeline.Cache(w, seed=seed, stats=st, capacity=T)
    xk = pipeline.draw_unit_tokens(w, st, kvc.SIDE_K, T, seed, "cuda")
    xv = pipeline.draw_unit_tokens(w, st, kvc.SIDE_V, T, seed, "cuda")
    cache.encode(xk, xv, 0, T)
    rng = np.random.default_rng(seed)
    q = (rng.standard_normal((w.n_units, w.group, 128)) * q_scale).astype(np.float16)
    qt = torch.as_tensor(q.view(np.int16), device="cuda").view(torch.float16)
    ws, out = cache.decode_buffers(T)
    kvc.kvc_decode_attn_rope(cache.K, cache.V, qt, w.group, torch.as_tensor(seq, device="cuda"), T, base, out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert np.isfinite(got).all()
    ot = OracleTables(w, st)
    worst = 0.0
    for u in (range(w.n_units) if units is None else units):
        h = w.head_of_unit(u)
        n = int(seq[u])
        res = {}
        for side, x in ((kvc.SIDE_K, xk), (kvc.SIDE_V, xv)):
            r, b = ot.rb(side, h)
            P, dl = ot.basis(side, h)
            res[side] = (onat.encode_codes(P, dl, b, x_bits(x[u][:n])), P, dl, b)
        (ck, Pk, dk, bk), (cv, Pv, dv, bv) = res[kvc.SIDE_K], res[kvc.SIDE_V]
        ref = oatt.decode_attention_rope(ck, cv, Pk, Pv, dk, dv, bk, bv, q[u].view(np.uint16), n, base)
        for g in range(w.group):
            e = normwise(got[u, g], ref[g])
            worst = max(worst, e)
            assert e <= TOL, (u, g, n, e)
    return worst


@pytest.mark.parametrize("G", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("base", [10000.0, 500000.0])
def test_rope_decode_every_group_size(G, base):
    w = synth.Workload(f"rope_g{G}", 1, 4, G, 1, 2000, 2.0)
    seq = np.array([2000, 1999, 65, 1][: w.n_units], dtype=np.int32)
    worst = _run(w, w.tokens, seq, base, q_scale=3.0)
    log(f"[rope G={G} base={base:g}] max normwise error {worst:.1e}")


def test_rope_decode_one_layer_of_the_8b_workload():
    w0 = synth.WORKLOADS["llama8b_b8_t32k_2bpd"]
    w = synth.Workload("rope_8b_l1", 1, w0.kv_heads, w0.group, w0.batch, w0.tokens, w0.bpd)
    seq = np.full(w.n_units, w.tokens, dtype=np.int32)
    worst = _run(w, w.tokens, seq, 500000.0, q_scale=2.0, units=[0, 33, w.n_units - 1])
    log(f"[rope 8B layer, 32k] max normwise error {worst:.1e}")
