"""Seeded synthetic inputs for the learner step.

This module holds only random-number recipes; none of the method's arithmetic
lives here.  Tests feed the same arrays to the HIP library and to the CPU
oracle, and the benchmark uses the same recipes.

The paper trains on SWB-300/SWB-2000 (Section 5.2), which are not available;
these arrays stand in for them with the paper's shapes: 260-dimensional fused
features, 21-frame chunks, 32000 context-dependent state labels.

Seeds: parameters 0, features 1, labels 2, peer 3, replica r -> 10 + r.
"""

from __future__ import annotations

import numpy as np

SEED_PARAMS = 0
SEED_FEATURES = 1
SEED_LABELS = 2
SEED_PEER = 3
SEED_REPLICA0 = 10
SEED_HIDDEN = 20
SEED_DY = 21


def params(n: int, seed: int = SEED_PARAMS, bound: float = 0.1) -> np.ndarray:
    """Flat float32 weights, U(-bound, bound)."""
    rng = np.random.default_rng(seed)
    return rng.uniform(-bound, bound, size=n).astype(np.float32)


def features(T: int, B: int, D: int, seed: int = SEED_FEATURES) -> np.ndarray:
    """Features [T, B, D] float32, N(0, 1)."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal((T, B, D), dtype=np.float32)


def labels(T: int, B: int, K: int, seed: int = SEED_LABELS, dist: str = "uniform",
           zipf_s: float = 1.1) -> np.ndarray:
    """Frame labels [T, B] int32 in [0, K).

    dist="uniform": uniform integers.
    dist="zipf": truncated Zipf, P(rank r) proportional to (r+1)^-zipf_s for
    r < K, drawn by inverse CDF; ranks are mapped to classes through a seeded
    permutation so that frequent classes are spread over the class range."""
    rng = np.random.default_rng(seed)
    if dist == "uniform":
        return rng.integers(0, K, size=(T, B), dtype=np.int64).astype(np.int32)
    if dist == "zipf":
        w = (np.arange(K, dtype=np.float64) + 1.0) ** (-zipf_s)
        cdf = np.cumsum(w)
        cdf /= cdf[-1]
        u = rng.random(size=(T, B))
        rank = np.minimum(np.searchsorted(cdf, u, side="right"), K - 1)
        perm = rng.permutation(K)
        return perm[rank].astype(np.int32)
    raise ValueError(dist)


def peer(theta: np.ndarray, seed: int = SEED_PEER, bound: float = 0.05) -> np.ndarray:
    """A neighbour's weights: theta plus U(-bound, bound) noise, float32."""
    rng = np.random.default_rng(seed)
    return (np.asarray(theta, dtype=np.float32)
            + rng.uniform(-bound, bound, size=theta.shape).astype(np.float32)).astype(np.float32)


def replica_grads(n: int, R: int, seed0: int = SEED_REPLICA0, std: float = 1e-3) -> list:
    """R replica gradient buffers, each n float32 values N(0, std^2)."""
    out = []
    for r in range(R):
        rng = np.random.default_rng(seed0 + r)
        out.append((rng.standard_normal(n, dtype=np.float32) * np.float32(std)).astype(np.float32))
    return out


def hidden_states(T: int, B: int, width: int, seed: int = SEED_HIDDEN) -> np.ndarray:
    """Stand-in top-layer outputs [T, B, width] float32, U(-1, 1) like h = o*tanh(c)."""
    rng = np.random.default_rng(seed)
    return rng.uniform(-1.0, 1.0, size=(T, B, width)).astype(np.float32)


def output_grads(T: int, B: int, width: int, seed: int = SEED_DY, std: float = 1e-3) -> np.ndarray:
    """Stand-in loss gradients w.r.t. the top layer [T, B, width] float32."""
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((T, B, width), dtype=np.float32) * np.float32(std)).astype(np.float32)


# The five workloads: a tiny float32 step, the full model at batch 128, the
# large-batch regime at 512, the update alone on the full parameter vector,
# and a long-chunk stress step.
CONFIGS = {
    "tiny": dict(L=1, D=40, H=64, P=32, K=100, T=21, B=8, precision="fp32",
                 label_dist="uniform", lr=0.1),
    "full_b128": dict(L=6, D=260, H=512, P=256, K=32000, T=21, B=128, precision="bf16",
                      label_dist="zipf", lr=0.05),
    "full_b512": dict(L=6, D=260, H=512, P=256, K=32000, T=21, B=512, precision="bf16",
                      label_dist="zipf", lr=0.05),
    "update_r8": dict(L=6, D=260, H=512, P=256, K=32000, T=21, B=128, precision="fp32",
                      label_dist="zipf", lr=0.05, R=8),
    "stress_t64_b1024": dict(L=6, D=260, H=512, P=256, K=32000, T=64, B=1024, precision="bf16",
                             label_dist="zipf", lr=0.05),
    # two super-learners of two replicas each in the ring of eq. 7
    "ring_s2_n2": dict(L=6, D=260, H=512, P=256, K=32000, T=21, B=128, precision="bf16",
                       label_dist="zipf", lr=0.05, S=2, N=2),
}
