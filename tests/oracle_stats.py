"""The oracle's calibration of a synthetic workload (table step 1 from the exact covariances, in fp64),
packed as the pipeline's per-head records, so that a cache built from it and the oracle's own tables
start from the same eigenvalues, eigenvectors and query variances. Test helper (not collected)."""
import functools

import numpy as np

from oracle import calib
from paper_2609_24298_amd import pipeline, synth


def stats_from_covs(covs):
    S_k = np.stack([c.S_k for c in covs])
    S_v = np.stack([c.S_v for c in covs])
    S_q = np.stack([np.stack(c.S_q) for c in covs])
    cal = calib.calibrate_heads(S_k, S_v, S_q)
    return [pipeline.HeadStats(c, cal["lam_k"][h], cal["U_k"][h], cal["sigma2_q"][h], cal["lam_v"][h], cal["U_v"][h])
            for h, c in enumerate(covs)]


@functools.lru_cache(maxsize=8)
def _cached(layers, kv_heads, group, d, seed):
    w = synth.Workload("calib", layers, kv_heads, group, 1, 1, 1.0, d)
    return tuple(stats_from_covs(synth.workload_covs(w, seed)))


def oracle_stats(w, seed=0):
    """Oracle calibration of every (layer, KV head) of workload w (depends only on its head shape)."""
    return list(_cached(w.layers, w.kv_heads, w.group, w.d, seed))
