"""Fused Hadamard-rotated truncated basis of KV-COBRA, written plainly (oracle).

Test infrastructure only: nothing in the product path may import this module.

Passages followed
-----------------
* Section 3.4: the retained SVD coordinates are rotated by an r x r
  Walsh-Hadamard matrix with a fixed random sign flip drawn once at
  calibration; the rotation is folded into the projection so that encode is a
  single matrix-vector product.
* Calibration table, steps 5-6, and Appendix A (Lemma lem:head-dist):
  Y = H_r U_r^T X, i.e. the stored basis is P = H_r diag(s) U_r^T (r x d).
  (Step 5 of the table writes H_r V[:, :r], whose shapes do not multiply; the
  r x d reading above is the one consistent with the lemma.)
* Readings:
  - A Walsh-Hadamard matrix exists only for r = 2^k. For other even r the
    rotation is block-diagonal over the binary expansion of r (Sylvester
    blocks, largest first); the retained directions, in importance order, are
    dealt to the blocks by largest remainder so each block receives a share of
    the whole spectrum. For r = 2^k this is exactly the paper's H_r.
  - Entries of a block of size n are +-1/sqrt(n) (orthonormal rows).
  - The sign vector s (one +-1 per retained direction) is an input: it is the
    random draw the paper makes once at calibration.
"""
from __future__ import annotations

import math

import numpy as np

from .quant import head_step


def block_sizes(r: int) -> list[int]:
    """Binary expansion of r as powers of two, largest first."""
    out = []
    bit = 1 << (max(r, 1).bit_length() - 1)
    while bit:
        if r & bit:
            out.append(bit)
        bit >>= 1
    return out


def sylvester_entry(a: int, c: int) -> int:
    """Entry (a, c) of the unnormalised Sylvester-Hadamard matrix: (-1)^popcount(a & c)."""
    return -1 if bin(a & c).count("1") % 2 else 1


def sylvester(n: int) -> np.ndarray:
    return np.array([[sylvester_entry(a, c) for c in range(n)] for a in range(n)], dtype=np.int64)


def deal(r: int) -> list[tuple[int, int]]:
    """Assign importance positions 0..r-1 to (block, column within block).

    Position i goes to the block j maximising (i + 1) * n_j - r * count_j
    (its largest remaining quota); ties go to the larger block.
    """
    sizes = block_sizes(r)
    counts = [0] * len(sizes)
    out = []
    for i in range(r):
        best_j, best_v = -1, None
        for j, n in enumerate(sizes):
            if counts[j] >= n:
                continue
            v = (i + 1) * n - r * counts[j]
            if best_v is None or v > best_v:
                best_j, best_v = j, v
        out.append((best_j, counts[best_j]))
        counts[best_j] += 1
    return out


def rotation_matrix(r: int) -> np.ndarray:
    """The r x r integer (+-1 / 0) rotation H~ such that P = diag(1/sqrt(n_row)) H~ diag(s) U_r^T.

    Column i of H~ corresponds to importance position i.
    """
    sizes = block_sizes(r)
    row0 = np.cumsum([0] + sizes[:-1])
    H = np.zeros((r, r), dtype=np.int64)
    for i, (j, c) in enumerate(deal(r)):
        n = sizes[j]
        for a in range(n):
            H[row0[j] + a, i] = sylvester_entry(a, c)
    return H


def row_block_size(r: int) -> np.ndarray:
    sizes = block_sizes(r)
    return np.concatenate([np.full(n, n, dtype=np.int64) for n in sizes])


def fused_basis_f64(U: np.ndarray, order, r: int, sign) -> np.ndarray:
    """P = blockdiag(H_n / sqrt(n)) diag(s) U_r^T in fp64, r x d.

    Each row is accumulated over its block's columns in increasing column
    order, then multiplied by 1/sqrt(n) (both sides of the parity check use
    this order so the fp16 rounding agrees bit for bit).
    """
    U = np.asarray(U, dtype=np.float64)
    d = U.shape[0]
    sizes = block_sizes(r)
    row0 = np.cumsum([0] + sizes[:-1])
    members: list[list[int]] = [[] for _ in sizes]
    for i, (j, c) in enumerate(deal(r)):
        members[j].append(i)
    P = np.zeros((r, d), dtype=np.float64)
    for j, n in enumerate(sizes):
        H = sylvester(n)
        acc = np.zeros((n, d), dtype=np.float64)
        for c, i in enumerate(members[j]):
            col = float(sign[i]) * U[:, int(order[i])]
            acc = acc + H[:, c][:, None].astype(np.float64) * col[None, :]
        inv = 1.0 / math.sqrt(float(n))
        P[row0[j]:row0[j] + n, :] = acc * inv
    return P


def fp16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp64 to fp16 (round to nearest even) and return the raw bits."""
    return np.asarray(x, dtype=np.float64).astype(np.float16).view(np.uint16)


def make_basis(U: np.ndarray, order, lam, r: int, b: int, sign):
    """Table steps 5-6: the stored per-head record (P as fp16 bits, step as f32).

    U: d x d, column k is the k-th eigenvector; order: importance order of
    eigen indices (only the first r are used); lam: eigenvalues by eigen index;
    sign: r values in {-1, +1} by importance position.
    """
    P = fused_basis_f64(U, order, r, sign)
    lam_ret = [float(lam[int(order[i])]) for i in range(r)]
    return fp16_bits(P), head_step(lam_ret, b)
