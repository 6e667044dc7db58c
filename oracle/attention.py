"""Decode attention over compressed KV and reconstruction, in fp64 (oracle).

Test infrastructure only: nothing in the product path may import this module.

Passages followed
-----------------
* Calibration/inference table, step 8: cached codes are dequantized when
  attention reads them.
* Appendix A (Lemma lem:head-dist): x_hat = U_r H_r^T Q(H_r U_r^T x), i.e.
  x_hat = P^T z_hat with z_hat the dequantized codes.
* Section 4: logits s_t = <q, k_t> / sqrt(d) with d the head dimension, and
  p = softmax(s).
* Appendix I, "Wall-clock at the primitive level": the decode primitive
  dequantizes and applies the inverse rotation in one pass. Since
  <q, P^T z> = <P q, z>, the logits are taken in the rank-r space here, and
  the value output is P_V^T (sum_t p_t z_V,t); both equal the dense
  computation on the reconstructed K and V (checked by a test).
"""
from __future__ import annotations

import math

import numpy as np

from .quant import dequant_level


def fp16_to_f64(bits: np.ndarray) -> np.ndarray:
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def dequantize(codes: np.ndarray, step: float, b: int) -> np.ndarray:
    """z_hat = (k - 2^(b-1) + 1/2) * step, element-wise."""
    return dequant_level(codes, float(step), b)


def reconstruct(codes: np.ndarray, P_bits: np.ndarray, step: float, b: int) -> np.ndarray:
    """x_hat_t = P^T z_hat_t for every token (n x d)."""
    return dequantize(codes, step, b) @ fp16_to_f64(P_bits)


def softmax(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def decode_logits(codes_k, Pk_bits, step_k, b_k, q_bits, seq_len):
    """Logits s[g, t] = (P_K q_g) . z_K,t / sqrt(d) of the first seq_len tokens (G x seq_len), in nats."""
    q = fp16_to_f64(q_bits)
    d = q.shape[1]
    zk = dequantize(codes_k[:seq_len], step_k, b_k)
    qt = q @ fp16_to_f64(Pk_bits).T                 # G x r_K
    return (qt @ zk.T) / math.sqrt(d)


def decode_attention(codes_k, codes_v, Pk_bits, Pv_bits, step_k, step_v, b_k, b_v, q_bits, seq_len):
    """One decode step for one unit: out[g] = P_V^T sum_t p_gt z_V,t with p = softmax((P_K q_g) . z_K,t / sqrt(d)).

    codes_*: (T x r) uint8, only the first seq_len tokens are attended; q_bits: (G x d) fp16 bits.
    """
    s = decode_logits(codes_k, Pk_bits, step_k, b_k, q_bits, seq_len)
    zv = dequantize(codes_v[:seq_len], step_v, b_v)
    p = softmax(s)
    zbar = p @ zv                                    # G x r_V
    return zbar @ fp16_to_f64(Pv_bits)               # G x d


def brute_force_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """softmax(q K^T / sqrt(d)) V in fp64 on dense K, V (T x d) and queries (G x d)."""
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    s = (q @ K.T) / math.sqrt(q.shape[1])
    return softmax(s) @ V
