"""Pins of the oracle's ring of learners (eq. 7 with several columns;
Section 3's consensus argument; Section 4's super-learners)."""

import numpy as np
import pytest

from oracle import blstm_ref as ref


@pytest.mark.parametrize("n", [2, 4, 6, 8])
def test_pairing_matrix_is_the_papers_t_k(n):
    """T_k: symmetric, doubly stochastic, two 0.5s per row and column, the
    off-diagonal one at a ring neighbour (Section 2, after eq. 7)."""
    for k in range(4):
        T = ref.ring_matrix(k, n)
        np.testing.assert_array_equal(T, T.T)
        np.testing.assert_array_equal(T.sum(axis=0), np.ones(n))
        for s in range(n):
            nz = np.flatnonzero(T[s])
            if n == 2:
                np.testing.assert_array_equal(T[s], [0.5, 0.5])
                continue
            assert len(nz) == 2 and T[s, s] == 0.5
            other = [j for j in nz if j != s][0]
            assert (other - s) % n in (1, n - 1)


def test_rounds_alternate_between_left_and_right_neighbours():
    n = 6
    for s in range(n):
        a, b = ref.ring_partner(s, 0, n), ref.ring_partner(s, 1, n)
        assert {a, b} == {(s + 1) % n, (s - 1) % n}
    with pytest.raises(ValueError):
        ref.ring_partner(0, 0, 5)


def test_round_is_theta_times_t_minus_step():
    """Column form against the matrix product of eq. 7."""
    rng = np.random.default_rng(5)
    n, d, lr = 6, 37, 0.3
    th = rng.standard_normal((n, d))
    g = rng.standard_normal((n, d))
    for k in range(3):
        got = np.stack(ref.ring_round(list(th), list(g), lr, k))
        want = (th.T @ ref.ring_matrix(k, n)).T - lr * g
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-14)


def test_averaging_preserves_the_sum_and_reaches_consensus():
    """With no local step the doubly stochastic averaging keeps the sum of
    the learners' weights and drives every learner to their mean (the
    argument that ADPSGD contains synchronous SGD as a special case)."""
    rng = np.random.default_rng(7)
    for n in (4, 8):
        th = list(rng.standard_normal((n, 11)))
        total = np.sum(th, axis=0)
        mean = total / n
        zero = [np.zeros(11)] * n
        for k in range(200):
            th = ref.ring_round(th, zero, 0.0, k)
            np.testing.assert_allclose(np.sum(th, axis=0), total, rtol=0, atol=1e-12)
        assert max(np.abs(t - mean).max() for t in th) < 1e-9


def test_stale_peer_copies():
    """peers=None reads the round-start weights; passing those same weights
    as the peer copies changes nothing, and an older copy enters only
    through the partner's half."""
    rng = np.random.default_rng(9)
    n = 4
    th = list(rng.standard_normal((n, 5)))
    old = list(rng.standard_normal((n, 5)))
    g = list(rng.standard_normal((n, 5)))
    a = ref.ring_round(th, g, 0.1, 1)
    b = ref.ring_round(th, g, 0.1, 1, peers=th)
    np.testing.assert_array_equal(np.stack(a), np.stack(b))
    c = ref.ring_round(th, g, 0.1, 1, peers=old)
    for s in range(n):
        p = ref.ring_partner(s, 1, n)
        np.testing.assert_allclose(c[s] - a[s], 0.5 * (old[p] - th[p]), rtol=0, atol=1e-14)


def test_super_learner_gradient_is_the_replica_mean():
    """Section 4: a super-learner of N replicas steps with the mean of their
    gradients (eq. 6 with scale 1/N); N replicas of equal batches give the
    replica gradient itself."""
    rng = np.random.default_rng(11)
    g = rng.standard_normal(13)
    np.testing.assert_allclose(ref.replica_grad_reduce([g, g, g], 1.0 / 3), g, rtol=0, atol=1e-15)
