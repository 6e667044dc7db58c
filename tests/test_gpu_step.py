"""GPU parity of the fused decode step (kvc_decode_step: the new token's append in the same launch as the
query projection) against the two-call step (kvc_encode_kv of one token, then kvc_decode_attn): code
arenas and outputs identical bit for bit, and outputs within the parity bound of the oracle's fp64
decode from its own codes, for every query-group size, over several consecutive steps."""
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


@pytest.mark.parametrize("G", [1, 4, 8, 16])
def test_fused_step_equals_two_calls(G):
    w = synth.Workload(f"step_g{G}", 4, 8, G, 4, 2000, 2.0)
    st = oracle_stats(w, 3)
    T0, steps = 1990, 3       # the steps cross into a new tile at token 1984.. and end at 1993
    A = pipeline.Cache(w, seed=3, stats=st, capacity=w.tokens)
    B = pipeline.Cache(w, seed=3, stats=st, capacity=w.tokens)
    xk = pipeline.draw_unit_tokens(w, st, kvc.SIDE_K, T0 + steps, 3, "cuda")
    xv = pipeline.draw_unit_tokens(w, st, kvc.SIDE_V, T0 + steps, 3, "cuda")
    for c in (A, B):
        c.encode(xk, xv, 0, T0)
    q = pipeline.draw_queries(w, st, 4, "cuda", scale=20.0)
    ws, outA = A.decode_buffers(T0 + steps)
    outB = torch.empty_like(outA)
    for s in range(steps):
        t = T0 + s
        seq = torch.full((w.n_units,), t + 1, dtype=torch.int32, device="cuda")
        xk1, xv1 = xk[:, t:t + 1].contiguous(), xv[:, t:t + 1].contiguous()
        A.encode(xk1, xv1, t, 1)
        A.decode(q, seq, T0 + steps, outA, ws)
        B.step(xk1, xv1, t, q, seq, T0 + steps, outB, ws)
        torch.cuda.synchronize()
        assert torch.equal(A.K.codes, B.K.codes) and torch.equal(A.V.codes, B.V.codes), s
        assert torch.equal(outA, outB), s
    # the last step against the oracle on a few units
    ot = OracleTables(w, st)
    n = T0 + steps
    got = outB.cpu().numpy()
    worst = 0.0
    for u in (0, 37, w.n_units - 1):
        h = w.head_of_unit(u)
        res = {}
        for side, x in ((kvc.SIDE_K, xk), (kvc.SIDE_V, xv)):
            r, b = ot.rb(side, h)
            P, dl = ot.basis(side, h)
            res[side] = (onat.encode_codes(P, dl, b, x_bits(x[u][:n])), P, dl, b)
        (ck, Pk, dk, bk), (cv, Pv, dv, bv) = res[kvc.SIDE_K], res[kvc.SIDE_V]
        qb = q[u].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        ref = oatt.decode_attention(ck, cv, Pk, Pv, dk, dv, bk, bv, qb, n)
        for g in range(G):
            e = normwise(got[u, g], ref[g])
            worst = max(worst, e)
            assert e <= TOL, (u, g, e)
    log(f"[step G={G}] fused step equals the two-call step over {steps} steps; vs oracle {worst:.1e}")


def test_fused_step_rejects_position_beyond_capacity():
    w = synth.Workload("step_cap", 1, 2, 4, 1, 128, 2.0)
    c = pipeline.Cache(w, seed=1, stats=oracle_stats(w, 1), capacity=128)
    x = torch.zeros((w.n_units, 1, 128), dtype=torch.float16, device="cuda")
    q = torch.zeros((w.n_units, 4, 128), dtype=torch.float16, device="cuda")
    ws, out = c.decode_buffers(128)
    seq = torch.full((w.n_units,), 128, dtype=torch.int32, device="cuda")
    with pytest.raises(kvc.KvcError) as ei:
        c.step(x, x, 128, q, seq, 128, out, ws)
    assert ei.value.code == kvc.KVC_ENOSPACE
