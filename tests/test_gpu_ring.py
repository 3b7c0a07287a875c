"""GPU: the ring of learners (eq. 7 over several learners, super-learners
of Section 4) against the oracle's ring on the same seeded inputs."""

import numpy as np
import pytest
import torch

from oracle import blstm_ref as ref
from paper_1907_05701_amd import inputs

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def run_ring(shape, precision, S, N, rounds, staleness, lr, tol, seed=40):
    from paper_1907_05701_amd.ring import LearnerRing
    say(f"[ring] shape={shape} {precision} S={S} N={N} rounds={rounds} staleness={staleness}")
    dims = ref.Dims(**shape)
    n = ref.param_count(dims)
    thetas = [inputs.params(n, seed=seed + s) for s in range(S)]
    batches = [[(inputs.features(dims.T, dims.B, dims.D, seed=seed + 100 + 10 * s + r),
                 inputs.labels(dims.T, dims.B, dims.K, seed=seed + 200 + 10 * s + r))
                for r in range(N)] for s in range(S)]
    ring = LearnerRing(shape, S, N, precision=precision, staleness=staleness)
    ring.load(thetas, batches)
    for _ in range(rounds):
        ring.round(lr)
    torch.cuda.synchronize()
    ring.check_recurrence()
    got = [ring.theta(s).cpu().numpy() for s in range(S)]
    # the oracle's ring on the same batches
    th = [t.astype(np.float64) for t in thetas]
    prev = th
    for k in range(rounds):
        grads = []
        for s in range(S):
            gs = [ref.learner_gradient(th[s], dims, *batches[s][r])["grad"] for r in range(N)]
            grads.append(ref.replica_grad_reduce(gs, 1.0 / N))
        new = ref.ring_round(th, grads, lr, k, peers=None if staleness == 0 else prev)
        prev, th = th, new
    errs = [rel(got[s], th[s]) for s in range(S)]
    say(f"[ring] worst learner rel err {max(errs):.3e}")
    assert max(errs) <= tol, errs
    return got


@pytest.mark.parametrize("staleness", [0, 1])
def test_ring_fp32_tiny(gpu_lib, staleness):
    run_ring(dict(L=1, D=40, H=64, P=32, K=100, T=21, B=8), "fp32", S=4, N=2, rounds=3,
             staleness=staleness, lr=0.1, tol=1e-4)


def test_ring_bf16_two_layers(gpu_lib):
    run_ring(dict(L=2, D=40, H=128, P=32, K=300, T=11, B=16), "bf16", S=2, N=2, rounds=2,
             staleness=0, lr=0.1, tol=2e-2)


def test_ring_averaging_alone_keeps_the_sum_and_reaches_consensus(gpu_lib):
    """lr = 0: only the doubly stochastic averaging acts; the learners' sum
    stays (float32 rounding aside) and they approach their mean."""
    from paper_1907_05701_amd.ring import LearnerRing
    shape = dict(L=1, D=40, H=64, P=32, K=100, T=21, B=8)
    dims = ref.Dims(**shape)
    n = ref.param_count(dims)
    S = 4
    thetas = [inputs.params(n, seed=60 + s) for s in range(S)]
    batches = [[(inputs.features(dims.T, dims.B, dims.D, seed=70 + s),
                 inputs.labels(dims.T, dims.B, dims.K, seed=80 + s))] for s in range(S)]
    ring = LearnerRing(shape, S, 1, precision="fp32")
    ring.load(thetas, batches)
    total = np.sum([t.astype(np.float64) for t in thetas], axis=0)
    mean = total / S
    spread0 = max(np.abs(t - mean).max() for t in thetas)
    for _ in range(40):
        ring.round(0.0)
    torch.cuda.synchronize()
    got = [ring.theta(s).cpu().numpy().astype(np.float64) for s in range(S)]
    assert np.abs(np.sum(got, axis=0) - total).max() < 1e-5
    spread = max(np.abs(t - mean).max() for t in got)
    say(f"[ring] consensus spread {spread0:.3e} -> {spread:.3e}")
    assert spread < 1e-6
