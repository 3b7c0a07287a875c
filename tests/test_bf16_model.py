"""CPU checks of the float64 model of the bf16 path's rounding points
(tests/bf16_path_model.py), which the GPU tests use as the error bound
where the 2e-2 bar cannot hold for any path with bf16 operands.

With no rounding point switched on the model must be the oracle's learner
step; each rounding point must change something; its rounding must be the
oracle's round-to-nearest-even; and the one regime where the bound replaces
the bar (saturated cells) is shown to be ill-conditioned by the oracle alone:
the exact gradient at the bf16 copy of the weights is far from the exact
gradient at theta."""

import os
import sys

import numpy as np
import pytest

from oracle import blstm_ref as ref
from paper_1907_05701_amd import inputs

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import bf16_path_model as bm  # noqa: E402

SMALL = dict(L=2, D=12, H=32, P=8, K=20, T=5, B=3)


def _inputs(shape, seed=0):
    dims = ref.Dims(**shape)
    theta = inputs.params(ref.param_count(dims), seed=seed, bound=0.3)
    x = inputs.features(dims.T, dims.B, dims.D, seed=seed + 1)
    lab = inputs.labels(dims.T, dims.B, dims.K, seed=seed + 2)
    return dims, theta, x, lab


def _rel(a, b):
    return float(np.linalg.norm(np.asarray(a) - np.asarray(b)) / np.linalg.norm(b))


def test_without_rounding_it_is_the_oracle():
    dims, theta, x, lab = _inputs(SMALL)
    want = ref.learner_gradient(theta, dims, x, lab)
    for mu in (8, 32):
        got = bm.learner_gradient(theta, SMALL, x, lab, points=(), member_units=mu)
        assert abs(got["loss"] - want["loss"]) <= 1e-12 * abs(want["loss"])
        assert _rel(got["grad"], want["grad"]) <= 1e-12
        assert _rel(got["y_top"], want["y_top"]) <= 1e-12
        assert _rel(got["dy_top"], want["dy_top"]) <= 1e-12


def test_head_without_rounding_is_the_oracle():
    shape = dict(L=1, D=4, H=16, P=8, K=50, T=3, B=4)
    dims = ref.Dims(**shape)
    theta = inputs.params(ref.param_count(dims), seed=7)
    y = inputs.hidden_states(dims.T, dims.B, 2 * dims.H, seed=8)
    lab = inputs.labels(dims.T, dims.B, dims.K, seed=9)
    loss, _, dy, g = ref.head_forward_backward(theta, dims, y, lab)
    l2, g2, dy2 = bm.head_gradient(theta, shape, y, lab, points=())
    assert abs(l2 - loss) <= 1e-12 * loss
    assert _rel(dy2, dy) <= 1e-12
    for k in g:
        assert _rel(g2[k], g[k]) <= 1e-12, k


@pytest.mark.parametrize("point", bm.ALL_POINTS)
def test_each_rounding_point_changes_the_step(point):
    dims, theta, x, lab = _inputs(SMALL, seed=3)
    exact = bm.learner_gradient(theta, SMALL, x, lab, points=(), member_units=8)
    one = bm.learner_gradient(theta, SMALL, x, lab, points=(point,), member_units=8)
    # bf16 keeps 8 significant bits: a rounding point moves the step by
    # about 2^-9 relative, never by nothing and never by more than a little
    e = max(abs(one["loss"] - exact["loss"]) / abs(exact["loss"]), _rel(one["grad"], exact["grad"]))
    assert 1e-8 < e < 5e-2, (point, e)


def test_rounding_is_round_to_nearest_even():
    rng = np.random.default_rng(4)
    v = np.concatenate([(rng.standard_normal(10000) * 10.0 ** rng.integers(-20, 20, 10000)).astype(np.float32),
                        np.array([1.00390625, 1.01171875, -1.00390625, 0.0, -0.0], np.float32)])
    np.testing.assert_array_equal(bm.bf(v), ref.bf16_to_float(ref.bf16_round(v)).astype(np.float64))


def test_path_points_exclude_the_float32_logits():
    assert set(bm.PATH_POINTS) == set(bm.ALL_POINTS) - {"s"}


def test_saturated_cells_make_the_gradient_ill_conditioned():
    """Gate biases i, f: +6, g: +2, o: +7 (the saturated-cell GPU test at a
    smaller width): rounding only the weight matrices to bf16 moves the
    exact (oracle) gradient by more than the bf16 bar in some block, so the
    bar cannot hold there for any path that multiplies bf16 weights."""
    shape = dict(L=2, D=40, H=128, P=32, K=100, T=21, B=16)
    dims = ref.Dims(**shape)
    blocks, n = ref.param_layout(dims)
    H = dims.H
    theta = inputs.params(n, seed=31).copy()
    for key, (off, shp) in blocks.items():
        if key[0] == "b_ih":
            b = theta[off:off + int(np.prod(shp))]
            b[0:2 * H] = 6.0
            b[2 * H:3 * H] = 2.0
            b[3 * H:] = 7.0
    x = inputs.features(dims.T, dims.B, dims.D, seed=32)
    lab = inputs.labels(dims.T, dims.B, dims.K, seed=33)
    g0 = ref.learner_gradient(theta, dims, x, lab)["grad"]
    tw = theta.copy()
    for key, (off, shp) in blocks.items():
        if (key if isinstance(key, str) else key[0]).startswith("W"):
            sl = slice(off, off + int(np.prod(shp)))
            tw[sl] = ref.bf16_to_float(ref.bf16_round(theta[sl]))
    g1 = ref.learner_gradient(tw, dims, x, lab)["grad"]
    worst = max(_rel(g1[o:o + int(np.prod(s))], g0[o:o + int(np.prod(s))]) for o, s in blocks.values())
    assert worst > 2e-2, worst
    # the same weight rounding at ordinary (unsaturated) biases stays far below the bar
    plain = inputs.params(n, seed=31)
    g0p = ref.learner_gradient(plain, dims, x, lab)["grad"]
    twp = plain.copy()
    for key, (off, shp) in blocks.items():
        if (key if isinstance(key, str) else key[0]).startswith("W"):
            sl = slice(off, off + int(np.prod(shp)))
            twp[sl] = ref.bf16_to_float(ref.bf16_round(plain[sl]))
    g1p = ref.learner_gradient(twp, dims, x, lab)["grad"]
    worst_plain = max(_rel(g1p[o:o + int(np.prod(s))], g0p[o:o + int(np.prod(s))]) for o, s in blocks.values())
    assert worst_plain < 5e-3, worst_plain
