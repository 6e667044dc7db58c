"""Host-side tests of libkvc (no GPU): the library loads and exports every
symbol include/kvc.h declares; kvc_allocate and kvc_make_basis are bit-exact
against the oracle on synthetic workloads; argument validation returns the
documented error codes before any launch."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import alloc as oa
from oracle import basis as ob
from paper_2609_24298_amd import kvc, synth

from oracle_stats import oracle_stats

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "kvc.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w]+\s*\*?\s*(kvc_\w+)\s*\(", src, flags=re.M)))


def test_library_exports_every_declared_symbol():
    names = header_functions()
    assert {"kvc_allocate", "kvc_make_basis", "kvc_encode", "kvc_decode_attn", "kvc_decode_attn_workspace",
            "kvc_reconstruct", "kvc_last_error", "kvc_version", "kvc_alloc_opts_default"} <= set(names)
    L = kvc.lib()
    for n in names:
        assert hasattr(L, n), n
    assert L.kvc_version() == 1


def test_struct_layouts_match_header():
    # offsets of the C structs as the binding lays them out (x86-64 SysV)
    assert ctypes.sizeof(kvc.AllocOpts) == 8 * 4 + 4 * 8
    assert ctypes.sizeof(kvc.HeadAlloc) == 24
    assert kvc.StreamDesc.codes_bytes.offset == kvc.StreamDesc.codes.offset + 8
    assert ctypes.sizeof(kvc.StreamDesc) == 16 + 14 * 8


def _oracle_opts(o: kvc.AllocOpts) -> oa.AllocOpts:
    return oa.AllocOpts(d=o.d, r_min=o.r_min, r_step=o.r_step, b_min=o.b_min, b_max=o.b_max, solver=o.solver,
                        rounds=o.rounds, reorder=bool(o.reorder), bpd=o.bpd, eta=o.eta, B_min=o.B_min, B_max=o.B_max)


def _stats(n_layers, group=4, seed=0):
    w = synth.Workload("t", n_layers, 8, group, 1, 64, 2.0)
    return oracle_stats(w, seed)


@pytest.mark.parametrize("bpd", [0.5, 1.0, 2.0, 3.0, 4.0])
def test_allocate_damped_kl_bit_exact(bpd):
    st = _stats(4)
    lam = np.stack([s.lam_k for s in st])
    sq = np.stack([s.sigma2_q for s in st])
    o = kvc.alloc_opts(bpd)
    got = kvc.kvc_allocate(lam, sq, o)
    exp = oa.allocate(lam, sq, _oracle_opts(o))
    assert np.array_equal(got["order"], exp["order"])
    assert np.array_equal(got["r"], exp["r"]) and np.array_equal(got["b"], exp["b"])
    assert np.array_equal(got["B"], exp["B"]) and np.array_equal(got["D"], exp["D"])
    # realised bits never exceed the budget
    assert np.sum(got["r"] * got["b"]) <= bpd * 128 * len(st) + 1e-9


def test_allocate_large_workload_bit_exact():
    # 256 heads, the 8B-shaped calibration
    st = _stats(32)
    lam = np.stack([s.lam_k for s in st])
    sq = np.stack([s.sigma2_q for s in st])
    o = kvc.alloc_opts(2.0)
    got = kvc.kvc_allocate(lam, sq, o)
    exp = oa.allocate(lam, sq, _oracle_opts(o))
    for k in ("r", "b", "B", "D", "order"):
        assert np.array_equal(got[k], exp[k]), k
    # heterogeneous table
    assert len(set(zip(got["r"].tolist(), got["b"].tolist()))) > 10


@pytest.mark.parametrize("bpd", [0.5, 2.0])
def test_allocate_c1_only_mse_bit_exact(bpd):
    st = _stats(2)
    lam = np.stack([s.lam_v for s in st])
    o = kvc.alloc_opts(bpd, kvc.SOLVER_C1_ONLY)
    got = kvc.kvc_allocate(lam, None, o)
    exp = oa.allocate(lam, None, _oracle_opts(o))
    for k in ("r", "b", "B", "D", "order"):
        assert np.array_equal(got[k], exp[k]), k
    assert np.all(got["B"] == bpd * 128)


def test_allocate_dp_bit_exact_and_exhaustive():
    rng = np.random.default_rng(3)
    # moderate instance for the oracle's full-enumeration DP
    lam = np.stack([np.sort(rng.uniform(0, 1, 16) ** rng.uniform(1, 5))[::-1] for _ in range(5)])
    o = kvc.alloc_opts(1.0, kvc.SOLVER_DP, d=16, B_max=64.0)
    got = kvc.kvc_allocate(lam, None, o)
    exp = oa.allocate(lam, None, _oracle_opts(o))
    for k in ("r", "b", "B", "D"):
        assert np.array_equal(got[k], exp[k]), k
    # tiny instance: equals exhaustive search over every (r, b) vector
    lam3 = np.stack([np.sort(rng.uniform(0, 1, 8))[::-1] for _ in range(3)])
    o3 = kvc.alloc_opts(1.5, kvc.SOLVER_DP, d=8, B_max=64.0)
    g3 = kvc.kvc_allocate(lam3, None, o3)
    assert g3["D"].sum() == pytest.approx(oa.brute_force_global([list(x) for x in lam3], _oracle_opts(o3)), rel=1e-14)


def test_allocate_dp_no_worse_than_damped_at_scale():
    st = _stats(8)
    lam = np.stack([s.lam_k for s in st])
    sq = np.stack([s.sigma2_q for s in st])
    dp = kvc.kvc_allocate(lam, sq, kvc.alloc_opts(1.0, kvc.SOLVER_DP))
    dm = kvc.kvc_allocate(lam, sq, kvc.alloc_opts(1.0))
    assert dp["D"].sum() <= dm["D"].sum()
    assert np.sum(dp["r"] * dp["b"]) <= 128 * 64


@pytest.mark.parametrize("r,b", [(2, 1), (6, 3), (16, 8), (50, 2), (96, 4), (100, 5), (128, 7), (126, 6)])
def test_make_basis_bit_exact(r, b):
    st = _stats(1)[r % 8]
    o = kvc.alloc_opts(2.0)
    order = kvc.kvc_allocate(st.lam_k[None], st.sigma2_q[None], o)["order"][0]
    P, delta = kvc.kvc_make_basis(st.U_k, order, st.lam_k, r, b, st.sign_k)
    Pe, de = ob.make_basis(st.U_k, order, st.lam_k, r, b, st.sign_k)
    assert np.array_equal(P, Pe)
    assert np.float32(delta).tobytes() == np.float32(de).tobytes()


def test_make_basis_many_random_bases_bit_exact():
    rng = np.random.default_rng(17)
    for trial in range(6):
        U, _ = np.linalg.qr(rng.standard_normal((128, 128)))
        U = U * rng.uniform(0.5, 3.0)          # exercise a wide range of fp16 exponents
        lam = np.sort(rng.uniform(1e-3, 5, 128))[::-1]
        order = rng.permutation(128).astype(np.int32)
        sign = (rng.integers(0, 2, 128) * 2 - 1).astype(np.int8)
        r = int(rng.integers(1, 65)) * 2
        b = int(rng.integers(1, 9))
        P, delta = kvc.kvc_make_basis(U, order, lam, r, b, sign)
        Pe, de = ob.make_basis(U, order, lam, r, b, sign)
        assert np.array_equal(P, Pe), (trial, r, b)
        assert np.float32(delta) == np.float32(de)


def test_error_codes_without_gpu():
    L = kvc.lib()
    o = kvc.alloc_opts(2.0)
    out = (kvc.HeadAlloc * 1)()
    lam = np.ones((1, 128))
    assert L.kvc_allocate(None, None, 1, ctypes.byref(o), ctypes.cast(out, ctypes.c_void_p), None) == kvc.KVC_EINVAL
    bad = kvc.alloc_opts(2.0, b_max=9)
    assert L.kvc_allocate(lam.ctypes.data_as(ctypes.c_void_p), None, 1, ctypes.byref(bad),
                          ctypes.cast(out, ctypes.c_void_p), None) == kvc.KVC_EINVAL
    assert b"bit range" in L.kvc_last_error()
    U = np.eye(128)
    order = np.arange(128, dtype=np.int32)
    sign = np.ones(128, dtype=np.int8)
    for r, b, code in [(3, 2, kvc.KVC_EUNSUPPORTED), (130, 2, kvc.KVC_EUNSUPPORTED), (4, 0, kvc.KVC_EUNSUPPORTED),
                       (4, 9, kvc.KVC_EUNSUPPORTED)]:
        with pytest.raises(kvc.KvcError) as ei:
            kvc.kvc_make_basis(U, order, np.ones(128), r, b, sign)
        assert ei.value.code == code
    with pytest.raises(kvc.KvcError) as ei:      # step below 2^-24
        kvc.kvc_make_basis(U, order, np.full(128, 1e-20), 4, 8, sign)
    assert ei.value.code == kvc.KVC_EUNSUPPORTED
    # device entry points validate descriptors on the host before any HIP call
    d = kvc.StreamDesc(n_units=1, d=64, capacity=64, side=0)
    assert L.kvc_encode(ctypes.byref(d), None, 0, 0, 1, None) == kvc.KVC_EUNSUPPORTED
    d.d = 128
    assert L.kvc_encode(ctypes.byref(d), None, 0, 0, 1, None) == kvc.KVC_EINVAL   # null tables
    assert L.kvc_encode(None, None, 0, 0, 1, None) == kvc.KVC_EINVAL
    assert L.kvc_reconstruct(None, 0, 1, None, None) == kvc.KVC_EINVAL
    assert L.kvc_decode_attn(None, None, None, 4, None, 1, None, None, 0, None) == kvc.KVC_EINVAL
    assert L.kvc_decode_attn_workspace(None, None, 4, 1) == 0


def test_descriptor_validation_ranges_without_gpu():
    # host mirrors are checked before anything touches the device pointers
    L = kvc.lib()
    r = np.array([4], dtype=np.int32)
    b = np.array([3], dtype=np.int32)
    off = np.array([0], dtype=np.int64)
    boff = np.array([0], dtype=np.int64)
    dl = np.array([0.5], dtype=np.float32)
    fake = ctypes.c_void_p(16)          # never dereferenced: validation fails first

    def desc(**kw):
        d = kvc.StreamDesc(n_units=1, d=128, capacity=64, side=0, r_host=r.ctypes.data, b_host=b.ctypes.data,
                           code_off_host=off.ctypes.data, basis_off_host=boff.ctypes.data, delta_host=dl.ctypes.data,
                           r=fake, b=fake, code_off=fake, basis_off=fake, delta=fake, codes=fake,
                           codes_bytes=8 * 4 * 3, basis=fake, basis_elems=4 * 128)
        for k, v in kw.items():
            setattr(d, k, v)
        return d

    r[0] = 5
    assert L.kvc_reconstruct(ctypes.byref(desc()), 0, 1, fake, None) == kvc.KVC_EUNSUPPORTED
    r[0] = 4
    b[0] = 9
    assert L.kvc_reconstruct(ctypes.byref(desc()), 0, 1, fake, None) == kvc.KVC_EUNSUPPORTED
    b[0] = 3
    assert L.kvc_reconstruct(ctypes.byref(desc(codes_bytes=95)), 0, 1, fake, None) == kvc.KVC_ENOSPACE
    assert L.kvc_reconstruct(ctypes.byref(desc(basis_elems=511)), 0, 1, fake, None) == kvc.KVC_ENOSPACE
    off[0] = 8
    assert L.kvc_reconstruct(ctypes.byref(desc()), 0, 1, fake, None) == kvc.KVC_EINVAL
    off[0] = 0
    dl[0] = 1e-9
    assert L.kvc_reconstruct(ctypes.byref(desc()), 0, 1, fake, None) == kvc.KVC_EUNSUPPORTED
    dl[0] = 0.5
    assert L.kvc_reconstruct(ctypes.byref(desc()), 0, 65, fake, None) == kvc.KVC_ENOSPACE
    assert L.kvc_reconstruct(ctypes.byref(desc()), -1, 1, fake, None) == kvc.KVC_EINVAL


def test_decode_rejects_misaligned_query_without_gpu():
    # q is read as 16-byte operand fragments; a misaligned pointer is refused before any launch
    L = kvc.lib()
    r = np.array([4], dtype=np.int32)
    b = np.array([3], dtype=np.int32)
    off = np.array([0], dtype=np.int64)
    boff = np.array([0], dtype=np.int64)
    dl = np.array([0.5], dtype=np.float32)
    fake = ctypes.c_void_p(256)          # never dereferenced
    dk, dv = (kvc.StreamDesc(n_units=1, d=128, capacity=64, side=side, r_host=r.ctypes.data, b_host=b.ctypes.data,
                             code_off_host=off.ctypes.data, basis_off_host=boff.ctypes.data,
                             delta_host=dl.ctypes.data, r=fake, b=fake, code_off=fake, basis_off=fake, delta=fake,
                             codes=fake, codes_bytes=8 * 4 * 3, basis=fake, basis_elems=4 * 128) for side in (0, 1))
    rc = L.kvc_decode_attn(ctypes.byref(dk), ctypes.byref(dv), ctypes.c_void_p(258), 4, fake, 1, fake, fake, 1 << 20, None)
    assert rc == kvc.KVC_EINVAL
    assert b"16-byte" in L.kvc_last_error()


def test_read_probe_validates_arguments_without_gpu():
    # the bandwidth probe refuses misaligned or null arguments before any launch; zero bytes launch nothing
    L = kvc.lib()
    fake = ctypes.c_void_p(256)          # never dereferenced
    assert L.kvc_read_probe(ctypes.c_void_p(264), 1024, fake, None) == kvc.KVC_EINVAL
    assert L.kvc_read_probe(fake, 1000, fake, None) == kvc.KVC_EINVAL
    assert L.kvc_read_probe(fake, 1024, ctypes.c_void_p(258), None) == kvc.KVC_EINVAL
    assert L.kvc_read_probe(None, 1024, fake, None) == kvc.KVC_EINVAL
    assert b"16 bytes" in L.kvc_last_error()
    assert L.kvc_read_probe(fake, 0, fake, None) == kvc.KVC_OK


def test_encode_kv_rejects_swapped_sides_without_gpu():
    L = kvc.lib()
    r = np.array([4], dtype=np.int32)
    b = np.array([3], dtype=np.int32)
    off = np.array([0], dtype=np.int64)
    dl = np.array([0.5], dtype=np.float32)
    fake = ctypes.c_void_p(256)          # never dereferenced
    dk, dv = (kvc.StreamDesc(n_units=1, d=128, capacity=64, side=side, r_host=r.ctypes.data, b_host=b.ctypes.data,
                             code_off_host=off.ctypes.data, basis_off_host=off.ctypes.data,
                             delta_host=dl.ctypes.data, r=fake, b=fake, code_off=fake, basis_off=fake, delta=fake,
                             codes=fake, codes_bytes=8 * 4 * 3, basis=fake, basis_elems=4 * 128) for side in (0, 1))
    rc = L.kvc_encode_kv(ctypes.byref(dv), ctypes.byref(dk), fake, 128, fake, 128, 0, 1, None)
    assert rc == kvc.KVC_EINVAL and b"sides" in L.kvc_last_error()
    rc = L.kvc_encode_kv(ctypes.byref(dk), ctypes.byref(dv), ctypes.c_void_p(258), 128, fake, 128, 0, 1, None)
    assert rc == kvc.KVC_EINVAL and b"16-byte" in L.kvc_last_error()
    rc = L.kvc_encode_kv(ctypes.byref(dk), ctypes.byref(dv), fake, 128, fake, 128, 60, 5, None)
    assert rc == kvc.KVC_ENOSPACE


def test_noalloc_scratch_size_matches_header():
    src = open(os.path.join(ROOT, "include", "kvc.h")).read()
    m = re.search(r"#define KVC_NOALLOC_SCRATCH_BYTES \((\d+)ll << (\d+)\)", src)
    assert m and int(m.group(1)) << int(m.group(2)) == kvc.NOALLOC_SCRATCH_BYTES


def test_make_candidates_bit_exact():
    from oracle import measured as om
    st = _stats(1)[3]
    order = kvc.kvc_allocate(st.lam_k[None], st.sigma2_q[None], kvc.alloc_opts(2.0))["order"][0]
    P_all, dl, rw = kvc.kvc_make_candidates(st.U_k, order, st.lam_k, st.sigma2_q, st.sign_k)
    po = wo = 0
    for ri, r in enumerate(kvc.rank_grid()):
        if r in (2, 6, 16, 18, 48, 66, 100, 128):
            for b in (1, 3, 8):
                Pe, de = ob.make_basis(st.U_k, order, st.lam_k, r, b, st.sign_k)
                assert np.array_equal(P_all[po:po + r * 128].reshape(r, 128), Pe), (r, b)
                assert np.float32(dl[ri, b - 1]).tobytes() == np.float32(de).tobytes(), (r, b)
            assert np.array_equal(rw[wo:wo + r], om.row_weights(r, order, st.sigma2_q).astype(np.float32)), r
        po += r * 128
        wo += r


@pytest.mark.parametrize("bpd", [0.5, 1.0, 3.0])
def test_allocate_measured_bit_exact(bpd):
    # tables shaped like measured ones (noisy, not the model) on 12 heads; the oracle's exact DP over them
    from oracle import measured as om
    rng = np.random.default_rng(int(bpd * 7))
    st = _stats(2)[:12]
    ranks = kvc.rank_grid()
    quant = np.zeros((12, len(ranks), 8))
    tw = np.zeros((12, 128))
    orders = []
    for h, s in enumerate(st):
        lam_hat = s.lam_k * rng.uniform(0.9, 1.1, 128)
        tw[h] = s.sigma2_q * lam_hat
        order = oa.importance_order(oa.kl_weights(s.lam_k, s.sigma2_q))
        orders.append(order)
        S = np.cumsum(tw[h][order])
        for ri, r in enumerate(ranks):
            for b in range(1, 9):
                quant[h, ri, b - 1] = S[r - 1] * 2.0 ** (-2 * b) / 12 * rng.uniform(0.8, 2.0)
    o = kvc.alloc_opts(bpd)
    got = kvc.kvc_allocate_measured(quant, tw, np.array(orders, dtype=np.int32), o)
    oo = _oracle_opts(o)
    tables = []
    for h in range(12):
        T = om.truncation_terms(orders[h], tw[h], np.ones(128))
        tables.append([[T[r] + quant[h, ri, b] for b in range(8)] for ri, r in enumerate(ranks)])
    budgets, allocs, _ = oa.dp_tables(tables, oo)
    assert np.array_equal(got["r"], [a[0] for a in allocs]) and np.array_equal(got["b"], [a[1] for a in allocs])
    assert np.array_equal(got["B"], budgets) and np.array_equal(got["D"], [a[2] for a in allocs])
