"""Thin ctypes binding of libkvc (include/kvc.h): argument marshalling only.

Every computation runs in the library (host allocator / basis builder in C++,
everything else in HIP kernels). If libkvc.so is missing this module raises:
there is no fallback path. PyTorch is used only for device memory and streams.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvc.so")

KVC_OK, KVC_EINVAL, KVC_EUNSUPPORTED, KVC_ENOSPACE, KVC_EDEVICE = 0, 1, 2, 3, 4
SIDE_K, SIDE_V = 0, 1
SOLVER_DAMPED, SOLVER_DP, SOLVER_C1_ONLY = 0, 1, 2
TILE = 64
HEAD_DIM = 128
NOALLOC_SCRATCH_BYTES = 64 << 20  # KVC_NOALLOC_SCRATCH_BYTES of include/kvc.h


class KvcError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libkvc error {code}: {msg}")
        self.code = code


class AllocOpts(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("r_min", ctypes.c_int32), ("r_step", ctypes.c_int32),
                ("b_min", ctypes.c_int32), ("b_max", ctypes.c_int32), ("solver", ctypes.c_int32),
                ("rounds", ctypes.c_int32), ("reorder", ctypes.c_int32), ("bpd", ctypes.c_double),
                ("eta", ctypes.c_double), ("B_min", ctypes.c_double), ("B_max", ctypes.c_double)]


class HeadAlloc(ctypes.Structure):
    _fields_ = [("r", ctypes.c_int32), ("b", ctypes.c_int32), ("B", ctypes.c_double), ("D", ctypes.c_double)]


_p = ctypes.c_void_p


class StreamDesc(ctypes.Structure):
    _fields_ = [("n_units", ctypes.c_int32), ("d", ctypes.c_int32), ("capacity", ctypes.c_int32),
                ("side", ctypes.c_int32),
                ("r_host", _p), ("b_host", _p), ("code_off_host", _p), ("basis_off_host", _p), ("delta_host", _p),
                ("r", _p), ("b", _p), ("code_off", _p), ("basis_off", _p), ("delta", _p),
                ("codes", _p), ("codes_bytes", ctypes.c_int64), ("basis", _p), ("basis_elems", ctypes.c_int64)]


_lib = None


def lib():
    """Load libkvc.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_24298_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.kvc_alloc_opts_default.argtypes = [ctypes.POINTER(AllocOpts), ctypes.c_double]
        L.kvc_allocate.argtypes = [_p, _p, ctypes.c_int32, ctypes.POINTER(AllocOpts), _p, _p]
        L.kvc_make_basis.argtypes = [_p, _p, _p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _p, _p, _p]
        L.kvc_encode.argtypes = [ctypes.POINTER(StreamDesc), _p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _p]
        L.kvc_decode_attn.argtypes = [ctypes.POINTER(StreamDesc), ctypes.POINTER(StreamDesc), _p, ctypes.c_int32, _p,
                                      ctypes.c_int32, _p, _p, ctypes.c_size_t, _p]
        L.kvc_decode_attn_workspace.argtypes = [ctypes.POINTER(StreamDesc), ctypes.POINTER(StreamDesc),
                                                ctypes.c_int32, ctypes.c_int32]
        L.kvc_decode_attn_workspace.restype = ctypes.c_size_t
        L.kvc_decode_step.argtypes = [ctypes.POINTER(StreamDesc), ctypes.POINTER(StreamDesc), _p, ctypes.c_int64, _p,
                                      ctypes.c_int64, ctypes.c_int32, _p, ctypes.c_int32, _p, ctypes.c_int32, _p, _p,
                                      ctypes.c_size_t, _p]
        L.kvc_decode_attn_rope.argtypes = [ctypes.POINTER(StreamDesc), ctypes.POINTER(StreamDesc), _p, ctypes.c_int32, _p,
                                           ctypes.c_int32, ctypes.c_float, _p, _p, ctypes.c_size_t, _p]
        L.kvc_decode_attn_noalloc.argtypes = [ctypes.POINTER(StreamDesc), ctypes.POINTER(StreamDesc), _p,
                                              ctypes.c_int32, _p, ctypes.c_int32, _p, _p]
        L.kvc_reconstruct.argtypes = [ctypes.POINTER(StreamDesc), ctypes.c_int32, ctypes.c_int32, _p, _p]
        L.kvc_read_probe.argtypes = [_p, ctypes.c_size_t, _p, _p]
        L.kvc_encode_kv.argtypes = [ctypes.POINTER(StreamDesc), ctypes.POINTER(StreamDesc), _p, ctypes.c_int64, _p,
                                    ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _p]
        L.kvc_allocate_measured.argtypes = [_p, _p, _p, ctypes.c_int32, ctypes.POINTER(AllocOpts), _p]
        L.kvc_make_candidates.argtypes = [_p, _p, _p, _p, ctypes.c_int32, _p, ctypes.c_int32, ctypes.c_int32, _p, _p, _p]
        L.kvc_measured_quant.argtypes = [_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _p, ctypes.c_int64, _p, _p,
                                         ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _p, _p]
        L.kvc_covariance.argtypes = [_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _p, _p]
        L.kvc_eigh.argtypes = [_p, ctypes.c_int32, _p, _p, _p, _p]
        L.kvc_query_variance.argtypes = [_p, _p, ctypes.c_int32, ctypes.c_int32, _p, _p]
        L.kvc_last_error.restype = ctypes.c_char_p
        L.kvc_version.restype = ctypes.c_int32
        _lib = L
    return _lib


def _check(rc: int):
    if rc != KVC_OK:
        raise KvcError(rc, lib().kvc_last_error().decode())


def _np_ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


# ------------------------------------------------------------------ host calls

def alloc_opts(bpd: float, solver: int = SOLVER_DAMPED, **kw) -> AllocOpts:
    o = AllocOpts()
    _check(lib().kvc_alloc_opts_default(ctypes.byref(o), float(bpd)))
    o.solver = solver
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def kvc_allocate(lam: np.ndarray, sigma2_q: np.ndarray | None, opts: AllocOpts):
    lam = np.ascontiguousarray(lam, dtype=np.float64)
    n, d = lam.shape
    assert d == opts.d
    sq = None if sigma2_q is None else np.ascontiguousarray(sigma2_q, dtype=np.float64)
    out = (HeadAlloc * n)()
    order = np.zeros((n, d), dtype=np.int32)
    _check(lib().kvc_allocate(_np_ptr(lam), None if sq is None else _np_ptr(sq), n, ctypes.byref(opts),
                              ctypes.cast(out, ctypes.c_void_p), _np_ptr(order)))
    return {"r": np.array([h.r for h in out], dtype=np.int32), "b": np.array([h.b for h in out], dtype=np.int32),
            "B": np.array([h.B for h in out]), "D": np.array([h.D for h in out]), "order": order}


def kvc_allocate_measured(quant: np.ndarray, trunc_w: np.ndarray, order: np.ndarray, opts: AllocOpts):
    """quant (n_heads, n_r, n_b), trunc_w (n_heads, d), order (n_heads, d) -> dict of r, b, B, D arrays."""
    quant = np.ascontiguousarray(quant, dtype=np.float64)
    trunc_w = np.ascontiguousarray(trunc_w, dtype=np.float64)
    order = np.ascontiguousarray(order, dtype=np.int32)
    n = quant.shape[0]
    out = (HeadAlloc * n)()
    _check(lib().kvc_allocate_measured(_np_ptr(quant), _np_ptr(trunc_w), _np_ptr(order), n, ctypes.byref(opts),
                                       ctypes.cast(out, ctypes.c_void_p)))
    return {"r": np.array([h.r for h in out], dtype=np.int32), "b": np.array([h.b for h in out], dtype=np.int32),
            "B": np.array([h.B for h in out]), "D": np.array([h.D for h in out])}


def rank_grid(r_min: int = 2, r_step: int = 2, d: int = HEAD_DIM):
    return list(range(r_min, d + 1, r_step))


def kvc_make_candidates(U: np.ndarray, order: np.ndarray, lam: np.ndarray, wt: np.ndarray, sign: np.ndarray,
                        r_min: int = 2, r_step: int = 2):
    """Candidate records of one head: (P_all fp16 bits, delta_all (n_r, 8), row_w_all)."""
    U = np.ascontiguousarray(U, dtype=np.float64)
    d = U.shape[0]
    ranks = rank_grid(r_min, r_step, d)
    P = np.zeros(sum(ranks) * d, dtype=np.uint16)
    dl = np.zeros((len(ranks), 8), dtype=np.float32)
    rw = np.zeros(sum(ranks), dtype=np.float32)
    _check(lib().kvc_make_candidates(_np_ptr(U), _np_ptr(np.ascontiguousarray(order, dtype=np.int32)),
                                     _np_ptr(np.ascontiguousarray(lam, dtype=np.float64)),
                                     _np_ptr(np.ascontiguousarray(wt, dtype=np.float64)), d,
                                     _np_ptr(np.ascontiguousarray(sign, dtype=np.int8)), r_min, r_step, _np_ptr(P),
                                     _np_ptr(dl), _np_ptr(rw)))
    return P, dl, rw


def kvc_make_basis(U: np.ndarray, order: np.ndarray, lam: np.ndarray, r: int, b: int, sign: np.ndarray):
    U = np.ascontiguousarray(U, dtype=np.float64)
    d = U.shape[0]
    order = np.ascontiguousarray(order, dtype=np.int32)
    lam = np.ascontiguousarray(lam, dtype=np.float64)
    sign = np.ascontiguousarray(sign[:r], dtype=np.int8)
    P = np.zeros((r, d), dtype=np.uint16)
    delta = np.zeros(1, dtype=np.float32)
    _check(lib().kvc_make_basis(_np_ptr(U), _np_ptr(order), _np_ptr(lam), d, int(r), int(b), _np_ptr(sign),
                                _np_ptr(P), _np_ptr(delta)))
    return P, delta[0]


# ------------------------------------------------------------------ device side

class Side:
    """One side (K or V) of a compressed cache: per-unit tables, code arena and basis arena.

    r, b, delta: per unit; basis: (n_bases x r_max x d) uint16 fp16 bits or a flat
    array with basis_off giving each unit's element offset.
    """

    def __init__(self, side: int, r, b, delta, basis_flat, basis_off, capacity: int, device="cuda", codes=None):
        import torch
        self.side = side
        self.capacity = int(capacity)
        self.r_h = np.ascontiguousarray(r, dtype=np.int32)
        self.b_h = np.ascontiguousarray(b, dtype=np.int32)
        self.delta_h = np.ascontiguousarray(delta, dtype=np.float32)
        self.basis_off_h = np.ascontiguousarray(basis_off, dtype=np.int64)
        n = self.r_h.size
        sizes = ((self.capacity + TILE - 1) // TILE) * 8 * self.r_h.astype(np.int64) * self.b_h
        self.code_off_h = np.zeros(n, dtype=np.int64)
        if n:
            self.code_off_h[1:] = np.cumsum(((sizes + 255) // 256) * 256)[:-1]
        total = int(self.code_off_h[-1] + sizes[-1]) if n else 0
        dev = torch.device(device)
        self.r = torch.as_tensor(self.r_h, device=dev)
        self.b = torch.as_tensor(self.b_h, device=dev)
        self.delta = torch.as_tensor(self.delta_h, device=dev)
        self.code_off = torch.as_tensor(self.code_off_h, device=dev)
        self.basis_off = torch.as_tensor(self.basis_off_h, device=dev)
        self.basis = torch.as_tensor(np.ascontiguousarray(basis_flat, dtype=np.uint16).view(np.int16), device=dev)
        self.codes = codes if codes is not None else torch.zeros(max(total, 16), dtype=torch.uint8, device=dev)
        assert self.codes.numel() >= total
        self.n_units = n
        self.desc = StreamDesc(
            n_units=n, d=HEAD_DIM, capacity=self.capacity, side=side,
            r_host=_np_ptr(self.r_h), b_host=_np_ptr(self.b_h), code_off_host=_np_ptr(self.code_off_h),
            basis_off_host=_np_ptr(self.basis_off_h), delta_host=_np_ptr(self.delta_h),
            r=self.r.data_ptr(), b=self.b.data_ptr(), code_off=self.code_off.data_ptr(),
            basis_off=self.basis_off.data_ptr(), delta=self.delta.data_ptr(),
            codes=self.codes.data_ptr(), codes_bytes=self.codes.numel(), basis=self.basis.data_ptr(),
            basis_elems=self.basis.numel())

    def stream_bytes(self, u: int, n_tok: int) -> int:
        return ((n_tok + TILE - 1) // TILE) * 8 * int(self.r_h[u]) * int(self.b_h[u])

    def unit_codes(self, u: int, n_tok: int):
        """Device view of unit u's stream bytes covering n_tok tokens."""
        off = int(self.code_off_h[u])
        return self.codes[off: off + self.stream_bytes(u, n_tok)]


class SideRange:
    """Units [u0, u0 + n) of a Side as a descriptor of their own: the per-unit tables are offset into
    the parent's, the code and basis arenas are shared (a layer of a cache, for per-layer calls)."""

    def __init__(self, parent: Side, u0: int, n: int):
        assert 0 <= u0 and n >= 0 and u0 + n <= parent.n_units
        self.parent = parent
        self.side, self.capacity, self.n_units = parent.side, parent.capacity, n
        self.r_h, self.b_h = parent.r_h[u0:u0 + n], parent.b_h[u0:u0 + n]
        self.delta_h, self.basis_off_h = parent.delta_h[u0:u0 + n], parent.basis_off_h[u0:u0 + n]
        self.code_off_h = parent.code_off_h[u0:u0 + n]
        self.codes, self.basis = parent.codes, parent.basis
        d = parent.desc
        self.desc = StreamDesc(
            n_units=n, d=d.d, capacity=d.capacity, side=d.side,
            r_host=_np_ptr(self.r_h), b_host=_np_ptr(self.b_h), code_off_host=_np_ptr(self.code_off_h),
            basis_off_host=_np_ptr(self.basis_off_h), delta_host=_np_ptr(self.delta_h),
            r=d.r + 4 * u0, b=d.b + 4 * u0, code_off=d.code_off + 8 * u0, basis_off=d.basis_off + 8 * u0,
            delta=d.delta + 4 * u0, codes=d.codes, codes_bytes=d.codes_bytes, basis=d.basis,
            basis_elems=d.basis_elems)

    def stream_bytes(self, u: int, n_tok: int) -> int:
        return ((n_tok + TILE - 1) // TILE) * 8 * int(self.r_h[u]) * int(self.b_h[u])


def _stream_ptr(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def kvc_encode(side: Side, x, t0: int, n_tok: int, stream=None):
    """x: fp16 tensor (n_units, >= n_tok, d) on the device."""
    import torch
    assert x.dtype == torch.float16 and x.is_contiguous() and x.dim() == 3
    assert x.shape[0] == side.n_units and x.shape[1] >= n_tok and x.shape[2] == HEAD_DIM
    assert x.device == side.codes.device
    _check(lib().kvc_encode(ctypes.byref(side.desc), ctypes.c_void_p(x.data_ptr()), int(x.stride(0)), int(t0),
                            int(n_tok), _stream_ptr(stream)))


def kvc_encode_kv(k: Side, v: Side, xk, xv, t0: int, n_tok: int, stream=None):
    """Keys and values of the same tokens: xk, xv fp16 tensors (n_units, >= n_tok, d) on the device."""
    import torch
    for side, x in ((k, xk), (v, xv)):
        assert x.dtype == torch.float16 and x.is_contiguous() and x.dim() == 3
        assert x.shape[0] == side.n_units and x.shape[1] >= n_tok and x.shape[2] == HEAD_DIM
        assert x.device == side.codes.device
    _check(lib().kvc_encode_kv(ctypes.byref(k.desc), ctypes.byref(v.desc), ctypes.c_void_p(xk.data_ptr()),
                               int(xk.stride(0)), ctypes.c_void_p(xv.data_ptr()), int(xv.stride(0)), int(t0),
                               int(n_tok), _stream_ptr(stream)))


def kvc_decode_attn_workspace(k: Side, v: Side, G: int, max_seq_len: int) -> int:
    n = lib().kvc_decode_attn_workspace(ctypes.byref(k.desc), ctypes.byref(v.desc), int(G), int(max_seq_len))
    if n == 0:
        _check(KVC_EINVAL if not lib().kvc_last_error() else KVC_EINVAL)
    return int(n)


def kvc_decode_attn(k: Side, v: Side, q, G: int, seq_len, max_seq_len: int, out, ws, stream=None):
    """q: fp16 (n_units, G, d); seq_len: int32 (n_units,); out: f32 (n_units, G, d); ws: uint8 workspace."""
    import torch
    U = k.n_units
    assert q.is_contiguous() and out.is_contiguous() and seq_len.is_contiguous()
    assert q.dtype == torch.float16 and q.numel() == U * G * HEAD_DIM
    assert out.dtype == torch.float32 and out.numel() == U * G * HEAD_DIM
    assert seq_len.dtype == torch.int32 and seq_len.numel() == U and v.n_units == U
    assert q.device == out.device == seq_len.device == ws.device == k.codes.device
    _check(lib().kvc_decode_attn(ctypes.byref(k.desc), ctypes.byref(v.desc), ctypes.c_void_p(q.data_ptr()), int(G),
                                 ctypes.c_void_p(seq_len.data_ptr()), int(max_seq_len),
                                 ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ws.data_ptr()), ws.numel(),
                                 _stream_ptr(stream)))


def kvc_decode_step(k: Side, v: Side, xk, xv, t_new: int, q, G: int, seq_len, max_seq_len: int, out, ws,
                    stream=None):
    """Append the new token (xk, xv: fp16 (n_units, >= 1, d)) at t_new to every unit, then decode attention."""
    import torch
    U = k.n_units
    for side, x in ((k, xk), (v, xv)):
        assert x.dtype == torch.float16 and x.is_contiguous() and x.dim() == 3
        assert x.shape[0] == side.n_units and x.shape[1] >= 1 and x.shape[2] == HEAD_DIM and x.device == side.codes.device
    assert q.is_contiguous() and out.is_contiguous() and seq_len.is_contiguous()
    assert q.dtype == torch.float16 and q.numel() == U * G * HEAD_DIM
    assert out.dtype == torch.float32 and out.numel() == U * G * HEAD_DIM
    assert seq_len.dtype == torch.int32 and seq_len.numel() == U and v.n_units == U
    assert q.device == out.device == seq_len.device == ws.device == k.codes.device
    _check(lib().kvc_decode_step(ctypes.byref(k.desc), ctypes.byref(v.desc), ctypes.c_void_p(xk.data_ptr()),
                                 int(xk.stride(0)), ctypes.c_void_p(xv.data_ptr()), int(xv.stride(0)), int(t_new),
                                 ctypes.c_void_p(q.data_ptr()), int(G), ctypes.c_void_p(seq_len.data_ptr()),
                                 int(max_seq_len), ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ws.data_ptr()),
                                 ws.numel(), _stream_ptr(stream)))


def kvc_decode_attn_rope(k: Side, v: Side, q, G: int, seq_len, max_seq_len: int, rope_base: float, out, ws,
                         stream=None):
    """Decode attention with RoPE: q fp16 (n_units, G, d) already rotated; keys rotated at their stream index."""
    import torch
    U = k.n_units
    assert q.is_contiguous() and out.is_contiguous() and seq_len.is_contiguous()
    assert q.dtype == torch.float16 and q.numel() == U * G * HEAD_DIM
    assert out.dtype == torch.float32 and out.numel() == U * G * HEAD_DIM
    assert seq_len.dtype == torch.int32 and seq_len.numel() == U and v.n_units == U
    assert q.device == out.device == seq_len.device == ws.device == k.codes.device
    _check(lib().kvc_decode_attn_rope(ctypes.byref(k.desc), ctypes.byref(v.desc), ctypes.c_void_p(q.data_ptr()), int(G),
                                      ctypes.c_void_p(seq_len.data_ptr()), int(max_seq_len), float(rope_base),
                                      ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ws.data_ptr()), ws.numel(),
                                      _stream_ptr(stream)))


def kvc_decode_attn_noalloc(k: Side, v: Side, q, G: int, seq_len, max_seq_len: int, out, stream=None):
    """kvc_decode_attn with the library's fixed workspace (no allocation; calls on one GPU must not overlap)."""
    import torch
    U = k.n_units
    assert q.is_contiguous() and out.is_contiguous() and seq_len.is_contiguous()
    assert q.dtype == torch.float16 and q.numel() == U * G * HEAD_DIM
    assert out.dtype == torch.float32 and out.numel() == U * G * HEAD_DIM
    assert seq_len.dtype == torch.int32 and seq_len.numel() == U and v.n_units == U
    assert q.device == out.device == seq_len.device == k.codes.device
    _check(lib().kvc_decode_attn_noalloc(ctypes.byref(k.desc), ctypes.byref(v.desc), ctypes.c_void_p(q.data_ptr()),
                                         int(G), ctypes.c_void_p(seq_len.data_ptr()), int(max_seq_len),
                                         ctypes.c_void_p(out.data_ptr()), _stream_ptr(stream)))


def kvc_reconstruct(side: Side, t0: int, n_tok: int, out, stream=None):
    import torch
    assert out.is_contiguous() and out.dtype == torch.float32 and out.numel() >= side.n_units * n_tok * HEAD_DIM
    assert out.device == side.codes.device
    _check(lib().kvc_reconstruct(ctypes.byref(side.desc), int(t0), int(n_tok), ctypes.c_void_p(out.data_ptr()),
                                 _stream_ptr(stream)))


def kvc_read_probe(buf, sink, stream=None):
    """Streaming read of a device buffer (uint8 tensor, 16-byte aligned, a multiple of 16 bytes); sink:
    a device int32/uint32 tensor of at least one element. Measures the achievable HBM read rate."""
    import torch
    assert buf.is_contiguous() and sink.is_contiguous() and sink.numel() >= 1
    assert sink.dtype in (torch.int32, torch.uint32) and buf.device == sink.device
    _check(lib().kvc_read_probe(ctypes.c_void_p(buf.data_ptr()), buf.numel() * buf.element_size(),
                                ctypes.c_void_p(sink.data_ptr()), _stream_ptr(stream)))


# ------------------------------------------------------------------ calibration (table step 1)

def kvc_covariance(x, n_tok: int, cov, centered: bool = True, stream=None):
    """x: fp16 (n_heads, >= n_tok, d) on the device; cov: f32 (n_heads, d, d)."""
    import torch
    assert x.dtype == torch.float16 and x.is_contiguous() and x.dim() == 3 and x.shape[2] == HEAD_DIM
    assert cov.dtype == torch.float32 and cov.is_contiguous() and cov.shape == (x.shape[0], HEAD_DIM, HEAD_DIM)
    assert x.shape[1] >= n_tok and x.device == cov.device
    _check(lib().kvc_covariance(ctypes.c_void_p(x.data_ptr()), int(x.stride(0)), int(x.shape[0]), int(n_tok),
                                int(bool(centered)), ctypes.c_void_p(cov.data_ptr()), _stream_ptr(stream)))


def kvc_eigh(S, lam, U, sweeps=None, stream=None):
    """S: f32 (n, d, d); lam: f32 (n, d); U: f32 (n, d, d); sweeps: int32 (n,) or None. All on the device."""
    import torch
    n = S.shape[0]
    for t in (S, U):
        assert t.dtype == torch.float32 and t.is_contiguous() and t.shape == (n, HEAD_DIM, HEAD_DIM)
    assert lam.dtype == torch.float32 and lam.is_contiguous() and lam.shape == (n, HEAD_DIM)
    assert sweeps is None or (sweeps.dtype == torch.int32 and sweeps.numel() == n)
    _check(lib().kvc_eigh(ctypes.c_void_p(S.data_ptr()), int(n), ctypes.c_void_p(lam.data_ptr()),
                          ctypes.c_void_p(U.data_ptr()), None if sweeps is None else ctypes.c_void_p(sweeps.data_ptr()),
                          _stream_ptr(stream)))


def kvc_query_variance(U, S_q, sig, stream=None):
    """U: f32 (n, d, d); S_q: f32 (n, G, d, d); sig: f32 (n, d). All on the device."""
    import torch
    n, G = S_q.shape[0], S_q.shape[1]
    assert U.dtype == S_q.dtype == sig.dtype == torch.float32
    assert U.is_contiguous() and S_q.is_contiguous() and sig.is_contiguous()
    assert U.shape == (n, HEAD_DIM, HEAD_DIM) and S_q.shape == (n, G, HEAD_DIM, HEAD_DIM) and sig.shape == (n, HEAD_DIM)
    _check(lib().kvc_query_variance(ctypes.c_void_p(U.data_ptr()), ctypes.c_void_p(S_q.data_ptr()), int(n), int(G),
                                    ctypes.c_void_p(sig.data_ptr()), _stream_ptr(stream)))


def kvc_measured_quant(x, n_tok: int, P_all, delta_all, row_w_all, quant, r_min: int = 2, r_step: int = 2,
                       stream=None):
    """x fp16 (n_heads, >= n_tok, d); P_all int16/uint16 (n_heads, sum r * d); delta_all f32 (n_heads, n_r, 8);
    row_w_all f32 (n_heads, sum r); quant f32 (n_heads, n_r, 8). All on the device."""
    import torch
    n = x.shape[0]
    assert x.dtype == torch.float16 and x.is_contiguous() and x.dim() == 3 and x.shape[2] == HEAD_DIM
    for t in (P_all, delta_all, row_w_all, quant):
        assert t.is_contiguous() and t.shape[0] == n and t.device == x.device
    assert delta_all.dtype == row_w_all.dtype == quant.dtype == torch.float32
    _check(lib().kvc_measured_quant(ctypes.c_void_p(x.data_ptr()), int(x.stride(0)), int(n), int(n_tok),
                                    ctypes.c_void_p(P_all.data_ptr()), int(P_all.stride(0)),
                                    ctypes.c_void_p(delta_all.data_ptr()), ctypes.c_void_p(row_w_all.data_ptr()),
                                    int(row_w_all.stride(0)), int(r_min), int(r_step),
                                    ctypes.c_void_p(quant.data_ptr()), _stream_ptr(stream)))
