"""Calibration statistics of one attention head (table step 1), in fp64 (oracle).

Test infrastructure only: nothing in the product path may import this module.

Passages followed
-----------------
* Table step 1: eigendecomposition of each head's key (and value) covariance,
  Sigma = U diag(lambda) U^T, and the query variance along each eigendirection.
* Section 2 (notation): sigma^2_Q,i is the variance of the query projected on
  the i-th key eigendirection, u_i^T Sigma_Q u_i.
* Proposition prop:kl-bound: the attention-KL weights w_i = sigma^2_Q,i lambda_i
  use these two quantities (the weights themselves are formed in alloc.py).

Readings
--------
* The eigendecomposition is the cyclic Jacobi method in fp64 (kvc_oracle.c,
  oracle_jacobi_eigh); eigenvalues descending, clamped at 0; each eigenvector's
  largest-magnitude entry positive (a fixed sign; the paper leaves it free).
* With G query heads sharing a KV head, sigma^2_Q,i is the mean over the G
  heads of u_i^T Sigma_Q,g u_i.
* The covariances are taken as given (the synthetic workloads know them
  exactly); from activations they would be the centred sample covariance.
"""
from __future__ import annotations

import numpy as np

from .native import jacobi_eigh


def query_variance(U: np.ndarray, S_q) -> np.ndarray:
    """sigma^2_Q,i = (1/G) sum_g u_i^T Sigma_Q,g u_i for the columns u_i of U."""
    U = np.asarray(U, dtype=np.float64)
    d = U.shape[1]
    out = np.zeros(d)
    for S in S_q:
        S = np.asarray(S, dtype=np.float64)
        for i in range(d):
            u = U[:, i]
            out[i] += u @ (S @ u)
    return out / len(S_q)


def sample_covariance(x: np.ndarray) -> np.ndarray:
    """Centred sample covariance (1/n) sum_t (x_t - mean)(x_t - mean)^T of activations x (n x d)."""
    x = np.asarray(x, dtype=np.float64)
    xc = x - x.mean(axis=0, keepdims=True)
    return (xc.T @ xc) / x.shape[0]


def head_calibration(S_k, S_v, S_q):
    """Per head: (lam_k, U_k, sigma2_q, lam_v, U_v) from the key, value and query-head covariances."""
    lam_k, U_k, _ = jacobi_eigh(S_k)
    lam_v, U_v, _ = jacobi_eigh(S_v)
    return lam_k, U_k, query_variance(U_k, S_q), lam_v, U_v


def calibrate_heads(S_k: np.ndarray, S_v: np.ndarray, S_q: np.ndarray):
    """Batched: S_k, S_v (n x d x d), S_q (n x G x d x d) -> dict of stacked lam_k, U_k, sigma2_q, lam_v, U_v."""
    lam_k, U_k, _ = jacobi_eigh(S_k)
    lam_v, U_v, _ = jacobi_eigh(S_v)
    sq = np.stack([query_variance(U_k[h], S_q[h]) for h in range(len(S_k))])
    return {"lam_k": lam_k, "U_k": U_k, "sigma2_q": sq, "lam_v": lam_v, "U_v": U_v}
