"""Measured distortion tables for the exact DP (oracle, fp64).

Test infrastructure only: nothing in the product path may import this module.

Passages followed
-----------------
* Appendix D, "Exact DP over measured distortion": each head's calibration
  activations are quantized with the deployed quantizer once per candidate
  (r, b), and the exact DP runs on the measured distortions in place of the
  Bennett model D(r, b) = sum_{i>r} w_i + q(b) sum_{i<=r} w_i.
* Table steps 5-7 for the deployed quantizer: the fused fp16 basis P_r and
  step of each candidate (basis.make_basis), exact codes (kvc_oracle.c).

Reading (the paper gives no formula for the measured table)
-----------------------------------------------------------
The measured table keeps the model's split into a truncation and a
quantization term, both measured on the n calibration activations x_t:
  trunc(r)   = sum over dropped importance positions p >= r of
               wt_o[p] * mean_t (u_o[p] . x_t)^2
  quant(r,b) = mean_t sum_k c_k (z_tk - zhat_tk)^2,  z_t = P_r x_t,
               zhat_t the dequantized exact codes of z_t,
  D(r, b)    = trunc(r) + quant(r, b),
with wt the per-eigendirection weights (sigma^2_Q for the attention-KL
objective, 1 for MSE) and c_k = (sum of wt over the importance positions of
row k's Hadamard block) / (block size). Each column of a block has entries
+-1/sqrt(n), so c_k spreads the error of a rotated coordinate evenly over its
block's eigendirections: the expected weighted error when the errors of
different coordinates are uncorrelated. With wt = 1 every c_k = 1 and D is the
measured mean squared reconstruction error mean_t ||x_t - x_hat_t||^2 (up to
the fp16 rounding of P), which a test checks against direct reconstruction.
"""
from __future__ import annotations

import numpy as np

from .attention import dequantize, fp16_to_f64
from .basis import block_sizes, deal, make_basis
from .native import encode_codes


def row_weights(r: int, order, wt) -> np.ndarray:
    """c_k for the r rows of P_r: mean weight of the importance positions dealt to row k's block."""
    sizes = block_sizes(r)
    tot = [0.0] * len(sizes)
    for i, (j, _c) in enumerate(deal(r)):
        tot[j] += float(wt[int(order[i])])
    return np.concatenate([np.full(n, tot[j] / n) for j, n in enumerate(sizes)])


def sample_variances(x_bits: np.ndarray, U: np.ndarray) -> np.ndarray:
    """mean_t (u_i . x_t)^2 for every eigen index i (fp64, from the fp16 activations)."""
    y = fp16_to_f64(x_bits) @ np.asarray(U, dtype=np.float64)
    return np.mean(y * y, axis=0)


def truncation_terms(order, wt, lam_hat) -> np.ndarray:
    """T[r] = sum_{p >= r} wt_o[p] lam_hat_o[p] for r = 0..d, summed from the last position down."""
    d = len(order)
    T = [0.0] * (d + 1)
    for p in range(d - 1, -1, -1):
        i = int(order[p])
        T[p] = T[p + 1] + float(wt[i]) * float(lam_hat[i])
    return np.array(T)


def quant_table(x_bits, U, order, lam, sign, wt, ranks, widths) -> np.ndarray:
    """quant(r, b) for every rank in `ranks` and width in `widths` (rows, columns of the result)."""
    out = np.zeros((len(ranks), len(widths)))
    for ri, r in enumerate(ranks):
        c = row_weights(r, order, wt)
        for bi, b in enumerate(widths):
            P, step = make_basis(U, order, lam, r, b, sign)
            codes = encode_codes(P, step, b, x_bits)
            z = fp16_to_f64(x_bits) @ fp16_to_f64(P).T
            e = z - dequantize(codes, step, b)
            out[ri, bi] = float(np.mean(np.sum(c[None, :] * e * e, axis=1)))
    return out


def measured_table(x_bits, U, order, lam, sign, wt, ranks, widths):
    """D(r, b) = trunc(r) + quant(r, b) for the candidate grid (ranks x widths)."""
    T = truncation_terms(order, wt, sample_variances(x_bits, U))
    Q = quant_table(x_bits, U, order, lam, sign, wt, ranks, widths)
    return np.array([[T[r] + Q[ri, bi] for bi in range(len(widths))] for ri, r in enumerate(ranks)]), T, Q
