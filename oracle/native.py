"""ctypes wrapper for oracle/kvc_oracle.c (exact encode, pack, unpack).

Test infrastructure only: nothing in the product path may import this module.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kvc_oracle.c")
_LIB = os.path.join(_HERE, "libkvc_oracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc (plain -O2, no FMA contraction, no fast-math; OpenMP over tokens)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared",
                               "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        u16p = ctypes.POINTER(ctypes.c_uint16)
        u8p = ctypes.POINTER(ctypes.c_uint8)
        lib.oracle_encode_codes.argtypes = [u16p, ctypes.c_int, ctypes.c_int, ctypes.c_float, ctypes.c_int,
                                            u16p, ctypes.c_int, u8p]
        lib.oracle_encode_codes.restype = ctypes.c_int
        lib.oracle_pack.argtypes = [u8p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, u8p]
        lib.oracle_pack.restype = None
        lib.oracle_unpack.argtypes = [u8p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, u8p]
        lib.oracle_unpack.restype = None
        f64p = ctypes.POINTER(ctypes.c_double)
        lib.oracle_jacobi_eigh.argtypes = [f64p, ctypes.c_int, ctypes.c_int, f64p, f64p, ctypes.POINTER(ctypes.c_int)]
        lib.oracle_jacobi_eigh.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray, ct):
    return a.ctypes.data_as(ctypes.POINTER(ct))


def encode_codes(P_bits: np.ndarray, step: float, b: int, x_bits: np.ndarray) -> np.ndarray:
    """Exact codes (n x r, uint8) of fp16 tokens x (n x d, raw bits) under fp16 basis P (r x d, raw bits)."""
    P_bits = np.ascontiguousarray(P_bits, dtype=np.uint16)
    x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
    r, d = P_bits.shape
    n = x_bits.shape[0]
    assert x_bits.shape[1] == d
    out = np.zeros((n, r), dtype=np.uint8)
    rc = _load().oracle_encode_codes(_ptr(P_bits, ctypes.c_uint16), r, d, float(np.float32(step)), int(b),
                                     _ptr(x_bits, ctypes.c_uint16), n, _ptr(out, ctypes.c_uint8))
    if rc != 0:
        raise ValueError("oracle encode: non-finite input or unsupported step")
    return out


def pack(codes: np.ndarray, r: int, b: int, side: int) -> np.ndarray:
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    n = codes.shape[0]
    out = np.zeros(((n + 63) // 64) * 8 * r * b, dtype=np.uint8)
    _load().oracle_pack(_ptr(codes, ctypes.c_uint8), n, r, b, side, _ptr(out, ctypes.c_uint8))
    return out


def unpack(stream: np.ndarray, n: int, r: int, b: int, side: int) -> np.ndarray:
    stream = np.ascontiguousarray(stream, dtype=np.uint8)
    assert stream.size >= ((n + 63) // 64) * 8 * r * b
    out = np.zeros((n, r), dtype=np.uint8)
    _load().oracle_unpack(_ptr(stream, ctypes.c_uint8), n, r, b, side, _ptr(out, ctypes.c_uint8))
    return out


def jacobi_eigh(S: np.ndarray):
    """Eigendecomposition of symmetric matrices S (n x d x d, or one d x d) by cyclic Jacobi in fp64:
    (eigenvalues descending, eigenvectors as columns with their largest entry positive, sweeps)."""
    S = np.ascontiguousarray(S, dtype=np.float64)
    one = S.ndim == 2
    if one:
        S = S[None]
    n, d, _ = S.shape
    lam = np.zeros((n, d))
    U = np.zeros((n, d, d))
    sw = np.zeros(n, dtype=np.int32)
    rc = _load().oracle_jacobi_eigh(_ptr(S, ctypes.c_double), n, d, _ptr(lam, ctypes.c_double),
                                    _ptr(U, ctypes.c_double), _ptr(sw, ctypes.c_int))
    if rc != 0:
        raise ValueError("oracle Jacobi: no convergence within 60 sweeps")
    return (lam[0], U[0], int(sw[0])) if one else (lam, U, sw)
