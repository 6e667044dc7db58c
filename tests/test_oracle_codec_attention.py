"""Pins of the oracle's exact encode, packed layout, reconstruction and decode
attention (CPU only): exact rational arithmetic, hand-derived bit positions,
round trips, Lemma lem:head-dist and dense softmax attention."""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import attention as oatt
from oracle import basis as ob
from oracle import layout as ol
from oracle import native as onat
from oracle import quant as oq


def half_fraction(bits: int) -> Fraction:
    return Fraction(float(np.array([bits], dtype=np.uint16).view(np.float16)[0]))


def encode_fraction(P_bits, step, b, x_bits):
    r, d = P_bits.shape
    out = np.zeros((x_bits.shape[0], r), dtype=np.uint8)
    st = Fraction(float(np.float32(step)))
    for t in range(x_bits.shape[0]):
        xs = [half_fraction(int(v)) for v in x_bits[t]]
        for i in range(r):
            y = sum(half_fraction(int(P_bits[i, j])) * xs[j] for j in range(d))
            out[t, i] = oq.code_exact(y, st, b)
    return out


def rand_half_bits(rng, shape, scale=1.0, subnormal_frac=0.05):
    v = (rng.standard_normal(shape) * scale).astype(np.float16).view(np.uint16)
    mask = rng.uniform(size=shape) < subnormal_frac
    v[mask] = rng.integers(0, 1024, size=mask.sum()) | (rng.integers(0, 2, size=mask.sum()) << 15)
    return v


@pytest.mark.parametrize("b", [1, 2, 3, 5, 8])
def test_c_exact_encode_matches_rationals(b):
    rng = np.random.default_rng(b)
    r, d = 6, 16
    P = rand_half_bits(rng, (r, d), 0.3)
    x = rand_half_bits(rng, (20, d), 2.0)
    step = np.float32(0.37 / (1 << (b - 1)))
    assert np.array_equal(onat.encode_codes(P, step, b, x), encode_fraction(P, step, b, x))


def test_c_exact_encode_on_exact_thresholds():
    # y lands exactly on multiples of the step: codes must follow floor exactly
    d, b = 8, 4
    P = np.zeros((2, d), dtype=np.float16)
    P[0, 0] = 1.0
    P[1, :2] = [0.5, -0.25]
    step = np.float32(0.125)
    xs = []
    for j in range(-9, 10):
        x = np.zeros(d, dtype=np.float16)
        x[0] = np.float16(j * 0.125)
        x[1] = np.float16(j * 0.25 * 0.5)
        xs.append(x)
    x = np.stack(xs)
    got = onat.encode_codes(P.view(np.uint16), step, b, x.view(np.uint16))
    exp = encode_fraction(P.view(np.uint16), step, b, x.view(np.uint16))
    assert np.array_equal(got, exp)
    # hand check: y0 = j/8 exactly -> floor = j -> code j + 8 clamped to [0, 15]
    assert list(got[:, 0]) == [max(0, min(15, j + 8)) for j in range(-9, 10)]


def test_layout_hand_derived_bit_positions():
    # K side, r = 2, b = 1 (tail group only): slot(t=0, i=1) = 0*2 + 1 = 1 -> bit 1 of byte 0
    c = np.zeros((64, 2), dtype=np.uint8)
    c[0, 1] = 1
    s = onat.pack(c, 2, 1, ol.SIDE_K)
    assert s.size == 16 and list(np.nonzero(s)[0]) == [0] and s[0] == 2
    # K side, r = 2, b = 1: slot(t=2, i=0) = 4 -> bit 4 of byte 0
    c[:] = 0
    c[2, 0] = 1
    s = onat.pack(c, 2, 1, ol.SIDE_K)
    assert list(np.nonzero(s)[0]) == [0] and s[0] == 16
    # V side, r = 2, b = 1: coord 1, token 0 -> slot 64 -> bit 64 -> byte 8
    c[:] = 0
    c[0, 1] = 1
    s = onat.pack(c, 2, 1, ol.SIDE_V)
    assert list(np.nonzero(s)[0]) == [8] and s[8] == 1
    # V side, b = 1: token 6 (quarter 0, item 6) -> position 4*2 + 1 = 9 -> bit 9 -> byte 1, bit 1;
    # token 17 (quarter 1, item 1) -> slot 16 + 4 = 20 -> byte 2, bit 4
    c[:] = 0
    c[6, 0] = 1
    c[17, 0] = 1
    s = onat.pack(c, 2, 1, ol.SIDE_V)
    assert list(np.nonzero(s)[0]) == [1, 2] and s[1] == 2 and s[2] == 16
    # V side, b = 2: token 13 -> position 4*1 + 3 = 7 -> bits 14, 15 -> byte 1, value 3 << 6
    c[:] = 0
    c[13, 0] = 3
    s = onat.pack(c, 2, 2, ol.SIDE_V)
    assert list(np.nonzero(s)[0]) == [1] and s[1] == 0xC0
    # V side, b = 4: token 5 -> position 8*0 + 2*1 + 1 = 3 -> bits 12..15 -> high nibble of byte 1
    c[:] = 0
    c[5, 0] = 0xA
    s = onat.pack(c, 2, 4, ol.SIDE_V)
    assert list(np.nonzero(s)[0]) == [1] and s[1] == 0xA0
    # V side, b = 8: natural token order, one byte per slot: coord 1, token 37 -> slot 64 + 37
    c8 = np.zeros((64, 2), dtype=np.uint8)
    c8[37, 1] = 200
    s = onat.pack(c8, 2, 8, ol.SIDE_V)
    assert list(np.nonzero(s)[0]) == [101] and s[101] == 200
    # K side with a tail group, r = 18 (one group of 16 + 2 tail coordinates), b = 8 (plain bytes):
    # token 1, coordinate 3 -> slot 0*1024 + 1*16 + 3 = 19; token 1, coordinate 17 -> slot 1024 + 1*2 + 1 = 1027
    c18 = np.zeros((64, 18), dtype=np.uint8)
    c18[1, 3] = 7
    c18[1, 17] = 9
    s = onat.pack(c18, 18, 8, ol.SIDE_K)
    assert list(np.nonzero(s)[0]) == [19, 1027] and s[19] == 7 and s[1027] == 9
    # K side, r = 18, b = 2: token 3, coordinate 17 -> tail slot 1024 + 3*2 + 1 = 1031 -> bits 2062, 2063
    # -> byte 257, bits 6..7
    c18[:] = 0
    c18[3, 17] = 2
    s = onat.pack(c18, 18, 2, ol.SIDE_K)
    assert list(np.nonzero(s)[0]) == [257] and s[257] == 0x80
    # b = 8 on the K side with r < 16 is plain bytes in token-major order
    c = np.arange(64 * 2, dtype=np.uint8).reshape(64, 2)
    s = onat.pack(c, 2, 8, ol.SIDE_K)
    assert np.array_equal(s, np.arange(128, dtype=np.uint8))
    # b = 3 = planes (2, 1): the 2-bit plane holds the high bits, then the 1-bit plane
    c = np.zeros((64, 2), dtype=np.uint8)
    c[0, 0] = 0b110
    s = onat.pack(c, 2, 3, ol.SIDE_K)
    assert s.size == 48 and s[0] == 0b11 and np.count_nonzero(s) == 1


def test_layout_v_groups_hand_derived():
    # V side, r = 40: N-tiles 0, 1 full and 2 holding coordinates 32..39 (ct = 8). For p = 1 and 2 the
    # three N-tiles are one group (g = 8 and 4), stored by L = 4 c + q, then N-tile; columns c < 8
    # have three fields, columns 8..15 two.
    # b = 2, coordinate 17 (n = 1, c = 1), token 0 (q = 0, position 0): L = 4; 4 lanes x 3 fields
    # before it, then n = 0 -> field 13 -> byte 4 * 13 = 52, bits 0..1
    c = np.zeros((64, 40), dtype=np.uint8)
    c[0, 17] = 3
    s = onat.pack(c, 40, 2, ol.SIDE_V)
    assert s.size == 8 * 40 * 2 and list(np.nonzero(s)[0]) == [52] and s[52] == 3
    # b = 2, coordinate 9 (n = 0, c = 9), token 16 (q = 1, position 0): L = 37. Before it: L < 32 (c < 8)
    # 32 x 3 = 96 fields, L = 32..35 (c = 8) 4 x 2, L = 36 (c = 9, q = 0) 2 -> field 106 -> byte 424
    c[:] = 0
    c[16, 9] = 2
    s = onat.pack(c, 40, 2, ol.SIDE_V)
    assert list(np.nonzero(s)[0]) == [424] and s[424] == 2
    # b = 1, the same code position: 2-byte fields -> byte 212
    c[:] = 0
    c[16, 9] = 1
    s = onat.pack(c, 40, 1, ol.SIDE_V)
    assert s.size == 8 * 40 and list(np.nonzero(s)[0]) == [212] and s[212] == 1
    # b = 3 = planes (2, 1) at r = 40: the 2-bit plane (640 bytes) then the 1-bit plane; coordinate 33
    # (n = 2, c = 1), token 5 (q = 0, position 4 * 1 + 1 = 5): L = 4, field 4 * 3 + 2 = 14 ->
    # 2-bit plane byte 56 + 10 // 8 = 57, bits 2..3; 1-bit plane byte 640 + 28 + 5 // 8 = 668, bit 5
    c[:] = 0
    c[5, 33] = 0b111
    s = onat.pack(c, 40, 3, ol.SIDE_V)
    assert list(np.nonzero(s)[0]) == [57, 668] and s[57] == 0b1100 and s[668] == 1 << 5
    # r = 128, b = 2: groups of four N-tiles, 1024 bytes each. Coordinate 80 (n = 5, c = 0) token 0:
    # group 1, L = 0, j = 1 -> byte 1024 + 4 = 1028
    c128 = np.zeros((64, 128), dtype=np.uint8)
    c128[0, 80] = 1
    s = onat.pack(c128, 128, 2, ol.SIDE_V)
    assert list(np.nonzero(s)[0]) == [1028] and s[1028] == 1
    # r = 100, b = 2: N-tiles 4..6 form the last group (m = 3, ct = 4). Coordinate 99 (n = 6, c = 3),
    # token 63 (q = 3, position 4 * 3 + 3 = 15): L = 15, field 15 * 3 + 2 = 47 ->
    # byte 1024 + 4 * 47 + 30 // 8 = 1215, bits 6..7
    c100 = np.zeros((64, 100), dtype=np.uint8)
    c100[63, 99] = 2
    s = onat.pack(c100, 100, 2, ol.SIDE_V)
    assert list(np.nonzero(s)[0]) == [1215] and s[1215] == 2 << 6
    # r = 100, b = 4 (g = 2): N-tile 6 alone in the last group (m = 1, ct = 4); coordinate 97
    # (n = 6, c = 1), token 20 (q = 1, item 4: position 8 * 0 + 2 * 0 + 1 = 1): L = 5, field 5 ->
    # byte 3 * 1024 + 8 * 5 = 3112, bits 4..7
    c100[:] = 0
    c100[20, 97] = 0x9
    s = onat.pack(c100, 100, 4, ol.SIDE_V)
    assert list(np.nonzero(s)[0]) == [3112] and s[3112] == 0x90
    # r = 24, b = 8 (g = 1): coordinate-major fields; coordinate 20 (n = 1, c = 4), token 50 (q = 3,
    # position 2): field 64 + 4 * 4 + 3 = 83 -> byte 16 * 83 + 2 = 1330
    c24 = np.zeros((64, 24), dtype=np.uint8)
    c24[50, 20] = 77
    s = onat.pack(c24, 24, 8, ol.SIDE_V)
    assert list(np.nonzero(s)[0]) == [1330] and s[1330] == 77


def test_layout_v_group_closed_form():
    # The kernels address a value field by a closed form instead of the enumeration: for lane
    # L = 4 c + q and N-tile n = g Q + j, byte 2p (g L + j) of group Q (at 1024 Q) in a full group, and
    # 2p (m L - A + j) in the last one (m N-tiles, its last holding ct coordinates, A = 4 (c - ct) + q
    # for c >= ct, else 0). A lane's run of fields in a group starts at a multiple of 4 bytes except in
    # a 1-bit plane, where the fields still lie in the 16 bytes from the dword boundary below the start.
    for r in range(2, 129, 2):
        nvt = (r + 15) // 16
        ct = r - 16 * (nvt - 1)
        for p in (1, 2, 4, 8):
            tab = ol.v_field_bytes(r, p)
            g = 1 if p == 8 else 8 // p
            ql = (nvt - 1) // g
            m = nvt - g * ql
            for (n, c, q), off in tab.items():
                Q, j, L = n // g, n % g, 4 * c + q
                A = 4 * (c - ct) + q if c >= ct else 0
                start = 1024 * Q + (2 * p * (m * L - A) if Q == ql else 16 * L)
                assert off == start + 2 * p * j, (r, p, n, c, q)
                assert start % 4 == 0 or p == 1, (r, p, n, c, q)
                assert off + 2 * p <= (start & ~3) + 16, (r, p, n, c, q)


@pytest.mark.parametrize("r", [2, 16, 18, 40, 64, 84, 100, 126, 128])
@pytest.mark.parametrize("b", [1, 2, 3, 4, 5, 7, 8])
def test_layout_v_fields_tile_the_plane(r, b):
    # every V code of a tile has its own bits and together they fill every plane exactly
    for p in ol.plane_widths(b):
        tab = ol.v_field_bytes(r, p)
        seen = np.zeros(8 * r * p * 8, dtype=np.int32)
        for t in range(64):
            for i in range(r):
                bit = ol.plane_bit(ol.SIDE_V, t, i, r, b, p, tab)
                seen[bit:bit + p] += 1
        assert seen.min() == 1 and seen.max() == 1


@pytest.mark.parametrize("b", range(1, 9))
def test_v_token_order_is_a_permutation_of_each_quarter(b):
    pos = [ol.pos_b(b, m) for m in range(16)]
    assert sorted(pos) == list(range(16))
    if b != 4:
        assert all(ol.pos_b(b, ol.pos_b(b, m)) == m for m in range(16))


@pytest.mark.parametrize("side", [ol.SIDE_K, ol.SIDE_V])
@pytest.mark.parametrize("b", range(1, 9))
def test_pack_c_matches_python_and_round_trips(side, b):
    rng = np.random.default_rng(10 * b + side)
    for r, n in [(2, 64), (6, 70), (16, 5), (50, 130)]:
        codes = rng.integers(0, 1 << b, size=(n, r)).astype(np.uint8)
        s = onat.pack(codes, r, b, side)
        assert s.size == ol.stream_bytes(n, r, b) == ((n + 63) // 64) * 8 * r * b
        assert bytes(s) == ol.pack(codes.tolist(), r, b, side)
        assert np.array_equal(onat.unpack(s, n, r, b, side), codes)
        assert np.array_equal(np.array(ol.unpack(bytes(s), n, r, b, side), dtype=np.uint8), codes)


def test_storage_is_exactly_rb_over_d_bits_per_dimension():
    # Appendix E: r*b/d bits per dimension, no per-token metadata (whole tiles)
    for r in (2, 16, 100, 128):
        for b in range(1, 9):
            n = 64 * 7
            assert ol.stream_bytes(n, r, b) * 8 / (n * 128) == r * b / 128


def _head(rng, d=128, alpha=1.2):
    Q, R = np.linalg.qr(rng.standard_normal((d, d)))
    Q = Q * np.sign(np.diag(R))
    lam = np.arange(1, d + 1, dtype=np.float64) ** (-alpha)
    return Q, lam


def test_orthogonal_decomposition_per_token():
    # Lemma lem:head-dist step 1: ||x - x_hat||^2 = ||xi_1||^2 + ||xi_2||^2, deterministically
    rng = np.random.default_rng(21)
    U, lam = _head(rng)
    r, b = 40, 3
    sign = rng.integers(0, 2, 128) * 2 - 1
    Pbits, step = ob.make_basis(U, np.arange(128), lam, r, b, sign)
    x = ((rng.standard_normal((50, 128)) * np.sqrt(lam)) @ U.T).astype(np.float16)
    codes = onat.encode_codes(Pbits, step, b, x.view(np.uint16))
    xh = oatt.reconstruct(codes, Pbits, step, b)
    P = oatt.fp16_to_f64(Pbits)
    xf = x.astype(np.float64)
    # with the fp16-rounded basis the projector is P^T P (rows not exactly orthonormal): use its range
    Q, _ = np.linalg.qr(P.T)
    xi1 = xf - (Q @ (Q.T @ xf.T)).T
    xi2 = (xf - xh) - xi1
    tot = np.sum((xf - xh) ** 2, axis=1)
    assert np.allclose(tot, np.sum(xi1 ** 2, axis=1) + np.sum(xi2 ** 2, axis=1), rtol=1e-10)


@pytest.mark.parametrize("r,b", [(32, 3), (64, 4), (128, 5), (96, 6)])
def test_head_distortion_matches_lemma_with_actual_quantizer(r, b):
    # Lemma lem:head-dist: E||x - x_hat||^2 = sum_{i>r} lam + sum_i E[eps_i^2]; after the rotation every
    # channel is ~N(0, sigma_bar^2) so E[eps_i^2] = sigma_bar^2 * mse(delta_b) (Gaussian closed form)
    rng = np.random.default_rng(r + b)
    U, lam = _head(rng, alpha=1.0)
    sign = rng.integers(0, 2, 128) * 2 - 1
    Pbits, step = ob.make_basis(U, np.arange(128), lam, r, b, sign)
    n = 4000
    x = ((rng.standard_normal((n, 128)) * np.sqrt(lam)) @ U.T).astype(np.float16)
    codes = onat.encode_codes(Pbits, step, b, x.view(np.uint16))
    err = np.mean(np.sum((x.astype(np.float64) - oatt.reconstruct(codes, Pbits, step, b)) ** 2, axis=1))
    sigma2 = lam[:r].mean()
    model = lam[r:].sum() + r * sigma2 * oq.gaussian_midrise_mse(oq.delta_b(b), b)
    assert abs(err - model) < 0.08 * model, (err, model)


def test_full_rank_high_bits_reconstructs_within_step():
    rng = np.random.default_rng(5)
    U, lam = _head(rng, alpha=0.6)
    sign = rng.integers(0, 2, 128) * 2 - 1
    Pbits, step = ob.make_basis(U, np.arange(128), lam, 128, 8, sign)
    x = ((rng.standard_normal((200, 128)) * np.sqrt(lam)) @ U.T).astype(np.float16)
    codes = onat.encode_codes(Pbits, step, 8, x.view(np.uint16))
    y = x.astype(np.float64) @ oatt.fp16_to_f64(Pbits).T
    zh = oatt.dequantize(codes, step, 8)
    inside = np.abs(y) < 127 * float(step)
    assert np.all(np.abs(y - zh)[inside] <= float(step) / 2 * (1 + 1e-12))
    xh = oatt.reconstruct(codes, Pbits, step, 8)
    # sqrt(d) * step / 2 from quantisation plus the fp16 rounding of the basis
    bound = math.sqrt(128) * float(step) / 2 + 2e-3 * np.linalg.norm(x.astype(np.float64), axis=1)
    ok = np.all(inside, axis=1)            # tokens with no clipped coordinate
    assert ok.sum() > 150
    assert np.all((np.linalg.norm(x.astype(np.float64) - xh, axis=1) <= bound)[ok])


def test_brute_force_attention_closed_forms():
    rng = np.random.default_rng(1)
    V = rng.standard_normal((7, 16))
    K = rng.standard_normal((7, 16))
    assert np.allclose(oatt.brute_force_attention(np.zeros((1, 16)), K, V), V.mean(axis=0))
    assert np.allclose(oatt.brute_force_attention(rng.standard_normal((2, 16)), K[:1], V[:1]), V[:1])
    q = np.zeros((1, 16))
    q[0, 3] = 1e4
    K2 = np.zeros((7, 16))
    K2[4, 3] = 1.0
    assert np.allclose(oatt.brute_force_attention(q, K2, V), V[4])


def test_rank_space_attention_equals_dense_on_identity_basis():
    # codes -> z_hat with P = I and every value representable: equals softmax(q K^T / sqrt(d)) V
    rng = np.random.default_rng(3)
    d, T, b = 128, 300, 8
    step = np.float32(0.0625)
    ck = rng.integers(0, 256, (T, d)).astype(np.uint8)
    cv = rng.integers(0, 256, (T, d)).astype(np.uint8)
    I = np.eye(d, dtype=np.float16).view(np.uint16)
    q = (rng.standard_normal((4, d)) * 0.5).astype(np.float16)
    out = oatt.decode_attention(ck, cv, I, I, step, step, b, b, q.view(np.uint16), T)
    K = oatt.dequantize(ck, step, b)
    V = oatt.dequantize(cv, step, b)
    ref = oatt.brute_force_attention(q.astype(np.float64), K, V)
    assert np.allclose(out, ref, rtol=1e-12, atol=1e-13)


def test_rank_space_attention_equals_dense_on_reconstruction():
    rng = np.random.default_rng(4)
    U, lam = _head(rng)
    sk = rng.integers(0, 2, 128) * 2 - 1
    Pk, stk = ob.make_basis(U, np.arange(128), lam, 48, 3, sk)
    Pv, stv = ob.make_basis(U, np.arange(128), lam, 100, 2, sk)
    T = 500
    ck = rng.integers(0, 8, (T, 48)).astype(np.uint8)
    cv = rng.integers(0, 4, (T, 100)).astype(np.uint8)
    q = (rng.standard_normal((4, 128)) * 3).astype(np.float16)
    out = oatt.decode_attention(ck, cv, Pk, Pv, stk, stv, 3, 2, q.view(np.uint16), 321)
    Kh = oatt.reconstruct(ck, Pk, stk, 3)[:321]
    Vh = oatt.reconstruct(cv, Pv, stv, 2)[:321]
    ref = oatt.brute_force_attention(q.astype(np.float64), Kh, Vh)
    assert np.allclose(out, ref, rtol=1e-10, atol=1e-12)


# ---------------------------------------------------------------- RoPE-aware decode (oracle)

def test_rope_rotation_equals_complex_multiplication():
    # pair (j, j + d/2) as the complex number x_j + i x_{j+d/2}, multiplied by exp(i p theta_j)
    from oracle import attention as oatt
    rng = np.random.default_rng(0)
    X = rng.standard_normal((7, 128))
    pos = np.array([0, 1, 5, 64, 1000, 32767, 131071])
    base = 500000.0
    Y = oatt.rope_rotate(X, pos, base)
    z = (X[:, :64] + 1j * X[:, 64:]) * np.exp(1j * pos[:, None] * base ** (-np.arange(64) / 64.0)[None, :])
    assert np.allclose(Y[:, :64], z.real, atol=1e-12) and np.allclose(Y[:, 64:], z.imag, atol=1e-12)
    assert np.array_equal(oatt.rope_rotate(X, np.zeros(7), base), X)


def test_rope_logits_depend_on_relative_position_only():
    from oracle import attention as oatt
    rng = np.random.default_rng(1)
    q, K = rng.standard_normal((1, 128)), rng.standard_normal((50, 128))
    t = np.arange(50)
    for shift in (0, 7, 12345):
        s = oatt.rope_rotate(q, [60 + shift], 10000.0) @ oatt.rope_rotate(K, t + shift, 10000.0).T
        if shift == 0:
            s0 = s
        assert np.allclose(s, s0, atol=1e-9)


def test_rope_decode_on_identity_basis_equals_brute_force():
    # P = I, unquantized values: decode_attention_rope equals softmax(q' . rope(K)) V on dense inputs
    from oracle import attention as oatt
    rng = np.random.default_rng(2)
    T, G, b = 300, 4, 8
    step = 1.0
    codes = rng.integers(0, 256, (T, 128)).astype(np.uint8)
    I = np.eye(128).astype(np.float16).view(np.uint16)
    q = (rng.standard_normal((G, 128)) * 0.05).astype(np.float16)
    got = oatt.decode_attention_rope(codes, codes, I, I, step, step, b, b, q.view(np.uint16), T, 10000.0)
    K = (codes.astype(np.float64) - 128 + 0.5) * step
    Kr = oatt.rope_rotate(K, np.arange(T), 10000.0)
    ref = oatt.brute_force_attention(q.astype(np.float64), Kr, K)
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)
    # positions matter: without the rotation the output differs
    assert not np.allclose(got, oatt.brute_force_attention(q.astype(np.float64), K, K), atol=1e-6)
