"""Pins for the oracle's super-learner reduction and ADPSGD update
(Section 2, eqs. 3, 6, 7; Section 3's consensus argument), against closed
forms, exact dyadic arithmetic and the properties of the mixing matrix T_k."""

import numpy as np
import pytest

from oracle import blstm_ref as ref
from paper_1907_05701_amd import inputs


def _dyadic(n, seed, scale=2.0**-10):
    """Values k * 2^-10 with |k| < 2^12: sums, halvings and products with
    power-of-two learning rates of these are exact in binary32 and binary64."""
    rng = np.random.default_rng(seed)
    return (rng.integers(-4096, 4096, size=n) * scale).astype(np.float32)


def test_sgd_closed_form():
    """eq. 3 (read theta_{k+1} = theta_k - alpha g): with theta_peer = theta
    the eq. 7 order is exactly SGD."""
    th, g = _dyadic(1000, 1), _dyadic(1000, 2)
    lr = 0.25
    out = ref.adpsgd_update(th, th, g, lr, order="eq7")
    np.testing.assert_array_equal(out, th.astype(np.float64) - lr * g.astype(np.float64))


def test_averaging_preserves_pair_sum():
    """T_k is doubly stochastic: averaging both columns leaves their sum
    unchanged, so after SGD-then-average the pair sum drops by exactly lr*g."""
    th, pe, g = _dyadic(1000, 3), _dyadic(1000, 4), _dyadic(1000, 5)
    lr = 0.5
    new = ref.adpsgd_update(th, pe, g, lr)
    before = th.astype(np.float64) + pe.astype(np.float64)
    np.testing.assert_array_equal(new + new, before - lr * g.astype(np.float64))
    new_eq7 = ref.adpsgd_update(th, pe, np.zeros_like(g), 0.3, order="eq7")
    np.testing.assert_array_equal(new_eq7 + new_eq7, before)


def test_orders_differ_by_half_the_gradient_step():
    rng = np.random.default_rng(0)
    th, pe, g = (rng.standard_normal(100) for _ in range(3))
    lr = 0.05
    a = ref.adpsgd_update(th, pe, g, lr)
    b = ref.adpsgd_update(th, pe, g, lr, order="eq7")
    np.testing.assert_allclose(a - b, 0.5 * lr * g, rtol=1e-12, atol=1e-15)


def test_zero_learning_rate_is_pure_averaging():
    th, pe = _dyadic(500, 6), _dyadic(500, 7)
    for order in ("sgd_then_avg", "eq7"):
        out = ref.adpsgd_update(th, pe, _dyadic(500, 8), 0.0, order=order)
        np.testing.assert_array_equal(out, (th.astype(np.float64) + pe) / 2)


def test_repeated_ring_averaging_reaches_the_mean():
    """Section 3: with no local updates, repeated averaging through T_k drives
    every learner to (1/n) sum_i theta^i; alternating left/right pairings on a
    ring of 8 learners."""
    lam, n = 8, 64
    rng = np.random.default_rng(1)
    thetas = [rng.standard_normal(n) for _ in range(lam)]
    mean = np.mean(thetas, axis=0)
    total = np.sum(thetas, axis=0)
    for k in range(400):
        shift = k % 2                     # pair (0,1),(2,3).. then (1,2),(3,4)..,(7,0)
        for a in range(shift, lam + shift, 2):
            i, j = a % lam, (a + 1) % lam
            avg = ref.adpsgd_update(thetas[i], thetas[j], np.zeros(n), 0.0)
            thetas[i], thetas[j] = avg, avg.copy()
        np.testing.assert_allclose(np.sum(thetas, axis=0), total, rtol=0, atol=1e-12)
    for th in thetas:
        np.testing.assert_allclose(th, mean, rtol=0, atol=1e-10)


def test_replica_reduce_is_the_scaled_sum():
    grads = inputs.replica_grads(1000, 8)
    out = ref.replica_grad_reduce(grads, 1.0 / 8)
    np.testing.assert_allclose(out, np.mean(np.stack(grads).astype(np.float64), axis=0), rtol=1e-15)
    # super-learner + update equals SSGD on the averaged gradient (eq. 6)
    th = inputs.params(1000)
    np.testing.assert_allclose(ref.adpsgd_update(th, th, out, 0.05, order="eq7"),
                               th.astype(np.float64) - 0.05 * out, rtol=1e-15, atol=1e-18)


@pytest.mark.parametrize("order", ["sgd_then_avg", "eq7"])
def test_fp32_order_is_exact_on_dyadic_inputs(order):
    th, pe = _dyadic(2000, 9), _dyadic(2000, 10)
    grads = [_dyadic(2000, 11 + r) for r in range(4)]
    got = ref.adpsgd_update_fp32(th, pe, grads, 0.25, 0.5, order)
    want = ref.adpsgd_update(th, pe, ref.replica_grad_reduce(grads, 0.25), 0.5, order)
    np.testing.assert_array_equal(got.astype(np.float64), want)


@pytest.mark.parametrize("order", ["sgd_then_avg", "eq7"])
def test_fp32_order_is_within_rounding_of_fp64(order):
    n, R = 20000, 8
    th = inputs.params(n)
    pe = inputs.peer(th)
    grads = inputs.replica_grads(n, R)
    got = ref.adpsgd_update_fp32(th, pe, grads, 1.0 / R, 0.05, order).astype(np.float64)
    want = ref.adpsgd_update(th, pe, ref.replica_grad_reduce(grads, 1.0 / R), 0.05, order)
    # a handful of roundings of values below 0.2 in magnitude
    assert np.max(np.abs(got - want)) < 8 * 2.0**-24 * 0.2


def test_fp32_reduce_order_is_left_to_right():
    """(a + b) + c differs from a + (b + c) here; the oracle fixes the former."""
    a = np.array([1.0], np.float32)
    b = np.array([2.0**-24], np.float32)
    c = np.array([2.0**-24], np.float32)
    out = ref.replica_grad_reduce_fp32([a, b, c], 1.0)
    assert out[0] == np.float32(1.0)                    # each tiny add rounds away
    assert (a + (b + c))[0] == np.float32(1.0 + 2.0**-23)


def test_training_loop_rate_matches_the_oracle_recipe():
    """The training loop's learning-rate function against the oracle's
    recipe (itself pinned to Section 3's worked example above), over the
    warm-up, the annealing and other batch ratios."""
    from paper_1907_05701_amd import train
    for base_lr, base_batch, batch, warm in ((0.1, 256, 2560, 10), (0.05, 128, 512, 10), (1.0, 8, 8, 3)):
        for e in range(1, 20):
            want = ref.lr_schedule(e, base_lr, base_batch, batch, warm)
            assert abs(train.lr_schedule(e, base_lr, base_batch, batch, warm) - want) <= 1e-15 * max(1.0, want)
