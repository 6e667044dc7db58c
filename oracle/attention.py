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
* Section 5 ("Scope"): keys are compressed before the rotary position
  embedding. The attention of a model with RoPE then scores the query, rotated
  at its position, against each reconstructed key rotated at the key's
  position (decode_attention_rope); rank-space scoring no longer applies,
  because the rotation depends on the position.

Readings for RoPE (the paper does not restate it)
--------------------------------------------------
* The rotary embedding of the Llama family: coordinate pairs (j, j + d/2),
  j < d/2, rotated by the angle p theta_j with theta_j = base^(-2 j / d);
  the caller passes the query already rotated at its own position.
* The key of stream index t sits at position t.
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


def rope_rotate(X: np.ndarray, positions, base: float) -> np.ndarray:
    """Rows of X (n x d) rotated at their positions: pairs (j, j + d/2) by the angle p base^(-2j/d)."""
    X = np.asarray(X, dtype=np.float64)
    d = X.shape[1]
    h = d // 2
    theta = base ** (-2.0 * np.arange(h) / d)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * theta[None, :]
    c, s = np.cos(ang), np.sin(ang)
    a, b = X[:, :h], X[:, h:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=1)


def decode_attention_rope(codes_k, codes_v, Pk_bits, Pv_bits, step_k, step_v, b_k, b_v, q_rot_bits, seq_len, base):
    """One decode step with RoPE: out[g] = P_V^T sum_t p_gt z_V,t, p = softmax_t(q'_g . rope(k_hat_t, t) / sqrt(d)),
    k_hat_t = P_K^T z_K,t the reconstructed pre-RoPE key of stream index t and q'_g the rotated query (fp16 bits)."""
    q = fp16_to_f64(q_rot_bits)
    d = q.shape[1]
    K = reconstruct(codes_k[:seq_len], Pk_bits, step_k, b_k)
    s = (q @ rope_rotate(K, np.arange(seq_len), base).T) / math.sqrt(d)
    p = softmax(s)
    zv = dequantize(codes_v[:seq_len], step_v, b_v)
    return (p @ zv) @ fp16_to_f64(Pv_bits)
