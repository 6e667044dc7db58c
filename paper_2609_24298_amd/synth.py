"""Seeded synthetic KV workloads (the only module both the oracle tests and the GPU path use).

This module draws inputs; it holds none of the compression method's
arithmetic. It stands in for the paper's models and calibration data, which
are not available: per (layer, KV head) the keys and values are drawn from
N(0, Sigma) with a power-law spectrum lambda_i = i^(-alpha), alpha ~ U[0.5, 2]
(the power-law spectra of Appendix F), a Haar-random eigenbasis and two
outlier channels whose standard deviation is multiplied by 8. Queries are
drawn the same way, one covariance per query head.

What a calibration pass would measure on real activations, the covariances,
is known exactly here (Sigma = F F^T for the generator's factor F) and is
handed out as such. Table step 1 (the eigendecomposition and the query
variance along each eigendirection) is not done here: the library computes it
on the device (kvc_eigh, kvc_query_variance) and the oracle on its own.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

D_HEAD = 128

KIND_K, KIND_V, KIND_Q, KIND_SIGN_K, KIND_SIGN_V, KIND_TOK, KIND_QVEC = range(7)


@dataclass(frozen=True)
class Workload:
    name: str
    layers: int
    kv_heads: int
    group: int          # query heads per KV head
    batch: int
    tokens: int
    bpd: float          # per side (K and V each)
    d: int = D_HEAD

    @property
    def n_heads(self) -> int:
        return self.layers * self.kv_heads

    @property
    def n_units(self) -> int:
        return self.layers * self.batch * self.kv_heads

    def unit(self, layer: int, batch: int, head: int) -> int:
        return (layer * self.batch + batch) * self.kv_heads + head

    def head_of_unit(self, u: int) -> int:
        layer = u // (self.batch * self.kv_heads)
        head = u % self.kv_heads
        return layer * self.kv_heads + head


WORKLOADS = {
    "small_l1_h8_t4k": Workload("small_l1_h8_t4k", 1, 8, 4, 1, 4096, 2.0),
    "llama8b_b8_t32k_2bpd": Workload("llama8b_b8_t32k_2bpd", 32, 8, 4, 8, 32768, 2.0),
    "llama8b_b1_t128k_0.5bpd": Workload("llama8b_b1_t128k_0.5bpd", 32, 8, 4, 1, 131072, 0.5),
    "llama8b_b16_t16k_sweep": Workload("llama8b_b16_t16k_sweep", 32, 8, 4, 16, 16384, 2.0),
    "llama70b_b4_t64k_1bpd": Workload("llama70b_b4_t64k_1bpd", 80, 8, 8, 4, 65536, 1.0),
}


def rng_for(seed: int, *key: int) -> np.random.Generator:
    return np.random.default_rng([int(seed)] + [int(k) for k in key])


def power_law_factor(rng: np.random.Generator, d: int = D_HEAD):
    """F with Sigma = F F^T = D U diag(lambda) U^T D; returns (F, Sigma, alpha)."""
    alpha = rng.uniform(0.5, 2.0)
    lam = np.arange(1, d + 1, dtype=np.float64) ** (-alpha)
    G = rng.standard_normal((d, d))
    Q, R = np.linalg.qr(G)
    Q = Q * np.sign(np.diag(R))[None, :]
    out = rng.choice(d, size=2, replace=False)
    Dg = np.ones(d)
    Dg[out] = 8.0
    F = (Dg[:, None] * Q) * np.sqrt(lam)[None, :]
    return F, F @ F.T, alpha


@dataclass
class HeadCov:
    """Exact covariances of one (layer, KV head) with the factors that generate its tokens."""
    S_k: np.ndarray          # key covariance (d x d)
    S_v: np.ndarray          # value covariance
    S_q: list                # one covariance per query head of the group
    F_k: np.ndarray          # S_k = F_k F_k^T
    F_v: np.ndarray
    F_q: list = field(default_factory=list)
    sign_k: np.ndarray | None = None  # +-1 per importance position (length d), the random sign flip
    sign_v: np.ndarray | None = None


def head_cov(seed: int, layer: int, head: int, group: int, d: int = D_HEAD) -> HeadCov:
    F_k, S_k, _ = power_law_factor(rng_for(seed, KIND_K, layer, head), d)
    F_v, S_v, _ = power_law_factor(rng_for(seed, KIND_V, layer, head), d)
    F_q, S_q = [], []
    for g in range(group):
        F, S, _ = power_law_factor(rng_for(seed, KIND_Q, layer, head, g), d)
        F_q.append(F)
        S_q.append(S)
    sk = rng_for(seed, KIND_SIGN_K, layer, head).integers(0, 2, size=d) * 2 - 1
    sv = rng_for(seed, KIND_SIGN_V, layer, head).integers(0, 2, size=d) * 2 - 1
    return HeadCov(S_k, S_v, S_q, F_k, F_v, F_q, sk.astype(np.int8), sv.astype(np.int8))


def workload_covs(w: Workload, seed: int = 0) -> list[HeadCov]:
    """Covariances of every (layer, KV head) of a workload, head index layer * kv_heads + head."""
    return [head_cov(seed, l, h, w.group, w.d) for l in range(w.layers) for h in range(w.kv_heads)]


def draw_tokens_np(F: np.ndarray, n: int, rng: np.random.Generator) -> np.ndarray:
    """n tokens x = F g (g ~ N(0, I)) rounded to fp16; returns float16 array (n x d)."""
    g = rng.standard_normal((n, F.shape[1]))
    return (g @ F.T).astype(np.float16)


def draw_tokens_torch(F: np.ndarray, n: int, seed_key, device, chunk: int = 1 << 16):
    """Same distribution, drawn with a seeded torch generator on `device` (fp16 tensor n x d)."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(np.random.SeedSequence(list(seed_key)).generate_state(1)[0]))
    Ft = torch.as_tensor(F, dtype=torch.float32, device=device)
    out = torch.empty((n, F.shape[0]), dtype=torch.float16, device=device)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        g = torch.randn((e - s, F.shape[1]), generator=gen, device=device, dtype=torch.float32)
        out[s:e] = (g @ Ft.T).to(torch.float16)
    return out
