"""Per-layer decode calls and their HIP-graph capture, through the C ABI.

A decode step issued as one kvc_decode_attn call per layer (unit ranges of the cache, see
kvc.SideRange) must give the oracle's outputs for every unit, like the all-layers call; the same
loop captured in one HIP graph must reproduce the eager outputs bit for bit on every replay, with
other GPU work between the replays.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2609_24298_amd import kvc, pipeline, synth

from test_gpu_parity import OracleTables
from test_gpu_workloads import _build, _check_units, log

pytestmark = pytest.mark.gpu


def _layer_loop(cache, w, q, seq, n_att, out, ws):
    upl = w.batch * w.kv_heads
    for l in range(w.layers):
        k, v = cache.layer_sides(l)
        sl = slice(l * upl, (l + 1) * upl)
        kvc.kvc_decode_attn(k, v, q[sl], w.group, seq[sl], n_att, out[sl], ws)


def _setup():
    w = synth.Workload("layers3", layers=3, kv_heads=2, group=4, batch=2, tokens=700, bpd=2.0)
    cache, xk, xv = _build(w, w.tokens, w.tokens)
    cache.encode(xk, xv, 0, w.tokens)
    q = pipeline.draw_queries(w, cache.stats, 9, "cuda", scale=3.0)
    seq_np = np.array([700, 513, 64, 1, 650, 700, 129, 300, 700, 2, 333, 64][: w.n_units], dtype=np.int32)
    seq = torch.as_tensor(seq_np, device="cuda")
    upl = w.batch * w.kv_heads
    nbytes = max(kvc.kvc_decode_attn_workspace(*cache.layer_sides(l), w.group, w.tokens) for l in range(w.layers))
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    assert upl * w.layers == w.n_units
    return w, cache, xk, xv, q, seq, seq_np, ws


def test_per_layer_calls_match_oracle():
    w, cache, xk, xv, q, seq, seq_np, ws = _setup()
    out = torch.full((w.n_units, w.group, w.d), float("nan"), dtype=torch.float32, device="cuda")
    _layer_loop(cache, w, q, seq, w.tokens, out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert np.isfinite(got).all()
    ot = OracleTables(w, cache.stats)
    _check_units(w, cache, ot, xk, xv, q, seq_np, got, range(w.n_units), "per-layer", w.tokens)


def test_per_layer_graph_replays_equal_eager():
    w, cache, xk, xv, q, seq, seq_np, ws = _setup()
    eager = torch.empty((w.n_units, w.group, w.d), dtype=torch.float32, device="cuda")
    _layer_loop(cache, w, q, seq, w.tokens, eager, ws)
    torch.cuda.synchronize()
    ref = eager.clone()
    out = torch.zeros_like(eager)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        _layer_loop(cache, w, q, seq, w.tokens, out, ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _layer_loop(cache, w, q, seq, w.tokens, out, ws)
    scratch = torch.empty((w.n_units, w.group, w.d), dtype=torch.float32, device="cuda")
    for rep in range(3):
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), rep
        # eager work between replays: the same calls into another buffer, and an all-layers call
        _layer_loop(cache, w, q, seq, w.tokens, scratch, ws)
        wsa, outa = cache.decode_buffers(w.tokens)
        cache.decode(q, seq, w.tokens, outa, wsa)
        torch.cuda.synchronize()
        assert torch.equal(scratch, ref), rep
    log(f"[per-layer graph] 3 replays equal the eager outputs")
