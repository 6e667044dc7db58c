"""GPU test of kvc_decode_attn_noalloc, the decode entry point that allocates nothing: through the C
ABI, its outputs equal kvc_decode_attn's (same kernels, caller workspace) bit for bit on two calls in
a row, the second with fewer units and a shorter context; a need beyond the fixed workspace is
rejected before any launch."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2609_24298_amd import kvc, pipeline, synth

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _decode_both(k, v, q, G, seq, n_max):
    nbytes = kvc.kvc_decode_attn_workspace(k, v, G, n_max)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    ref = torch.empty((k.n_units, G, 128), dtype=torch.float32, device="cuda")
    got = torch.full_like(ref, float("nan"))
    kvc.kvc_decode_attn(k, v, q, G, seq, n_max, ref, ws)
    kvc.kvc_decode_attn_noalloc(k, v, q, G, seq, n_max, got)
    torch.cuda.synchronize()
    return ref, got, nbytes


def test_noalloc_equals_workspace_entry_point_on_two_calls():
    w = synth.Workload("noalloc_l2_h8", 2, 8, 4, 2, 3000, 2.0)
    cache = pipeline.Cache(w, seed=11)
    xk = pipeline.draw_unit_tokens(w, cache.stats, kvc.SIDE_K, w.tokens, 11, "cuda")
    xv = pipeline.draw_unit_tokens(w, cache.stats, kvc.SIDE_V, w.tokens, 11, "cuda")
    cache.encode(xk, xv, 0, w.tokens)
    q = pipeline.draw_queries(w, cache.stats, 12, "cuda", scale=20.0)
    # call 1: every unit, ragged lengths up to the whole context
    seq = torch.as_tensor(np.array([w.tokens - 37 * u for u in range(w.n_units)], dtype=np.int32), device="cuda")
    ref, got, nb1 = _decode_both(cache.K, cache.V, q, w.group, seq, w.tokens)
    assert torch.isfinite(ref).all() and torch.equal(ref, got)
    # call 2: the first layer's units only, a shorter context (a smaller workspace need)
    k1, v1 = cache.layer_sides(0)
    n = k1.n_units
    seq2 = torch.full((n,), 700, dtype=torch.int32, device="cuda")
    ref2, got2, nb2 = _decode_both(k1, v1, q[:n].contiguous(), w.group, seq2, 700)
    assert nb2 < nb1
    assert torch.isfinite(ref2).all() and torch.equal(ref2, got2)
    log(f"[noalloc] two calls equal the workspace entry point (workspace needs {nb1} then {nb2} bytes)")


def test_noalloc_rejects_a_need_beyond_its_scratch():
    # 20000 tiny units at G = 16 need ~160 MB for the query limbs alone
    U, G = 20000, 16
    P = np.zeros((2, 128), dtype=np.float16)
    P[0, 0] = P[1, 1] = 1.0
    flat = P.view(np.uint16).reshape(-1)
    ks = kvc.Side(kvc.SIDE_K, [2] * U, [1] * U, [0.5] * U, flat, [0] * U, 64)
    vs = kvc.Side(kvc.SIDE_V, [2] * U, [1] * U, [0.5] * U, flat, [0] * U, 64)
    need = kvc.kvc_decode_attn_workspace(ks, vs, G, 64)
    assert need > kvc.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((U, G, 128), dtype=torch.float16, device="cuda")
    seq = torch.full((U,), 64, dtype=torch.int32, device="cuda")
    out = torch.zeros((U, G, 128), dtype=torch.float32, device="cuda")
    with pytest.raises(kvc.KvcError) as ei:
        kvc.kvc_decode_attn_noalloc(ks, vs, q, G, seq, 64, out)
    assert ei.value.code == kvc.KVC_ENOSPACE
    torch.cuda.synchronize()
    assert torch.count_nonzero(out).item() == 0
