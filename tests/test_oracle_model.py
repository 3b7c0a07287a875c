"""Pins for the oracle's model arithmetic (BLSTM forward/BPTT and the
softmax cross-entropy head), each against something other than the oracle:
the paper's printed model size, central finite differences, PyTorch's own
nn.LSTM/cross_entropy (float64, CPU), closed forms and invariances."""

import math
import os

import numpy as np
import pytest
import torch

from oracle import blstm_ref as ref
from paper_1907_05701_amd import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

MICRO = ref.Dims(L=2, D=3, H=4, P=3, K=5, T=4, B=2)
TINY = ref.Dims(L=1, D=40, H=64, P=32, K=100, T=21, B=8)
FULL = ref.Dims(L=6, D=260, H=512, P=256, K=32000, T=21, B=128)


def _read_golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.strip()
            if line and not line.startswith("#"):
                k, v = line.split()
                vals[k] = float(v)
    return vals


def _step_inputs(dims, seed=0, dist="uniform"):
    n = ref.param_count(dims)
    theta = inputs.params(n, seed=seed).astype(np.float64)
    x = inputs.features(dims.T, dims.B, dims.D, seed=seed + 1).astype(np.float64)
    lab = inputs.labels(dims.T, dims.B, dims.K, seed=seed + 2, dist=dist)
    return theta, x, lab


def _loss(theta, dims, x, lab):
    y, _ = ref.blstm_forward(theta, dims, x)
    return ref.head_forward_backward(theta, dims, y, lab)[0]


# ---------------------------------------------------------------- layout ---

def test_param_count_matches_paper_model_size():
    g = _read_golden("model_size.txt")
    dims = ref.Dims(L=int(g["layers"]), D=int(g["input_dim"]), H=int(g["cells_per_direction"]),
                    P=int(g["bottleneck"]), K=int(g["classes"]), T=int(g["unroll"]), B=1)
    n = ref.param_count(dims)
    assert n == 43_154_944
    assert n > g["min_params"]
    mb = n * 4 / 2**20
    assert abs(mb - g["approx_megabytes"]) < 1.0      # 164.6 MiB is "about 165MB"
    assert ref.param_count(TINY) == 61_700


def test_layout_is_torch_nn_lstm_order():
    dims = MICRO
    lstm = torch.nn.LSTM(dims.D, dims.H, num_layers=dims.L, bidirectional=True)
    blocks, total = ref.param_layout(dims)
    expect = []
    for layer in range(dims.L):
        for d in range(2):
            suf = "_reverse" if d else ""
            for name in ("weight_ih", "weight_hh", "bias_ih", "bias_hh"):
                expect.append(f"{name}_l{layer}{suf}")
    assert [n for n, _ in lstm.named_parameters()] == expect
    sizes = [p.numel() for p in lstm.parameters()]
    lstm_keys = [k for k in blocks if isinstance(k, tuple)]
    assert [int(np.prod(blocks[k][1])) for k in lstm_keys] == sizes
    offs = [blocks[k][0] for k in lstm_keys] + [blocks[k][0] for k in ("W_l", "b_l", "W_s", "b_s")]
    assert offs == sorted(offs) and offs[0] == 0


# ------------------------------------------------- torch float64 cross-check ---

def _torch_step(theta, dims, x, lab, loss_scale=None):
    """The same step through PyTorch's own modules (float64, CPU)."""
    torch.manual_seed(0)
    lstm = torch.nn.LSTM(dims.D, dims.H, num_layers=dims.L, bidirectional=True).double()
    lin = torch.nn.Linear(2 * dims.H, dims.P).double()
    out = torch.nn.Linear(dims.P, dims.K).double()
    params = list(lstm.parameters()) + [lin.weight, lin.bias, out.weight, out.bias]
    flat = torch.tensor(theta, dtype=torch.float64)
    off = 0
    with torch.no_grad():
        for p in params:
            p.copy_(flat[off:off + p.numel()].view_as(p))
            off += p.numel()
    assert off == flat.numel()
    xt = torch.tensor(x, dtype=torch.float64)
    y, _ = lstm(xt)
    logits = out(lin(y.reshape(-1, 2 * dims.H)))
    scale = 1.0 / (dims.B * dims.T) if loss_scale is None else loss_scale
    loss = torch.nn.functional.cross_entropy(
        logits, torch.tensor(lab.reshape(-1), dtype=torch.long), reduction="sum") * scale
    loss.backward()
    grad = torch.cat([p.grad.reshape(-1) for p in params]).numpy()
    return float(loss.detach()), y.detach().numpy(), grad


@pytest.mark.parametrize("dims", [MICRO, TINY, ref.Dims(L=3, D=10, H=16, P=8, K=50, T=5, B=3)],
                         ids=["micro", "tiny", "3layer"])
def test_matches_torch_float64(dims):
    theta, x, lab = _step_inputs(dims)
    got = ref.learner_gradient(theta, dims, x, lab)
    loss_t, y_t, grad_t = _torch_step(theta, dims, x, lab)
    assert abs(got["loss"] - loss_t) <= 1e-12 * abs(loss_t)
    np.testing.assert_allclose(got["y_top"], y_t, rtol=0, atol=1e-13)
    blocks, _ = ref.param_layout(dims)
    for key, (off, shape) in blocks.items():
        sl = slice(off, off + int(np.prod(shape)))
        a, b = got["grad"][sl], grad_t[sl]
        assert np.linalg.norm(a - b) <= 1e-11 * max(np.linalg.norm(b), 1e-30), key


def test_matches_torch_at_full_layer_dims_small_batch():
    """Full layer widths (260 -> 6 x 2 x 512 -> 256 -> 32000) with B=2, T=3."""
    dims = ref.Dims(L=6, D=260, H=512, P=256, K=32000, T=3, B=2)
    theta, x, lab = _step_inputs(dims, dist="zipf")
    got = ref.learner_gradient(theta, dims, x, lab)
    loss_t, y_t, grad_t = _torch_step(theta, dims, x, lab)
    assert abs(got["loss"] - loss_t) <= 1e-12 * abs(loss_t)
    np.testing.assert_allclose(got["y_top"], y_t, rtol=0, atol=1e-12)
    assert np.linalg.norm(got["grad"] - grad_t) <= 1e-10 * np.linalg.norm(grad_t)


# ------------------------------------------------------- finite differences ---

def test_gradient_matches_central_differences():
    dims = MICRO
    theta, x, lab = _step_inputs(dims, seed=5)
    # larger weights so that every gate sits away from saturation-free linearity
    theta = theta * 10.0
    g = ref.learner_gradient(theta, dims, x, lab)["grad"]
    eps = 1e-6
    fd = np.zeros_like(theta)
    for k in range(theta.size):
        tp = theta.copy(); tp[k] += eps
        tm = theta.copy(); tm[k] -= eps
        fd[k] = (_loss(tp, dims, x, lab) - _loss(tm, dims, x, lab)) / (2 * eps)
    blocks, _ = ref.param_layout(dims)
    for key, (off, shape) in blocks.items():
        sl = slice(off, off + int(np.prod(shape)))
        err = np.linalg.norm(g[sl] - fd[sl]) / max(np.linalg.norm(fd[sl]), 1e-30)
        assert err < 1e-6, (key, err)


# ------------------------------------------------------------ closed forms ---

def test_zero_head_gives_log_k_and_uniform_softmax():
    for dims in (TINY, ref.Dims(L=1, D=3, H=4, P=4, K=32000, T=2, B=3)):
        n = ref.param_count(dims)
        theta = inputs.params(n).astype(np.float64)
        blocks, _ = ref.param_layout(dims)
        for key in ("W_s", "b_s"):
            off, shape = blocks[key]
            theta[off:off + int(np.prod(shape))] = 0.0
        x = inputs.features(dims.T, dims.B, dims.D).astype(np.float64)
        lab = inputs.labels(dims.T, dims.B, dims.K)
        y, _ = ref.blstm_forward(theta, dims, x)
        loss, ell, dy, grads = ref.head_forward_backward(theta, dims, y, lab)
        assert abs(loss - math.log(dims.K)) < 1e-12
        np.testing.assert_allclose(ell, math.log(dims.K), rtol=0, atol=1e-12)
        np.testing.assert_array_equal(dy, 0.0)               # dz = ds W_s = 0
        M = dims.T * dims.B
        counts = np.bincount(lab.reshape(-1), minlength=dims.K)
        np.testing.assert_allclose(grads["b_s"], (M / dims.K - counts) / M, rtol=0, atol=1e-15)
    assert abs(math.log(32000) - 10.373491181781864) < 1e-15


def test_bias_only_cell_follows_geometric_recurrence():
    """With W_ih = W_hh = 0 every step sees the same gates, so
    c_n = i*g*(1 - f^n)/(1 - f) after n steps and h_n = o*tanh(c_n)."""
    dims = ref.Dims(L=1, D=5, H=6, P=2, K=3, T=7, B=2)
    n = ref.param_count(dims)
    theta = np.zeros(n)
    blocks, _ = ref.param_layout(dims)
    rng = np.random.default_rng(7)
    for d in range(2):
        for name in ("b_ih", "b_hh"):
            off, shape = blocks[(name, 0, d)]
            theta[off:off + shape[0]] = rng.uniform(-1, 1, size=shape[0])
    x = rng.standard_normal((dims.T, dims.B, dims.D))
    y, _ = ref.blstm_forward(theta, dims, x)
    H = dims.H
    for d in range(2):
        a = sum(theta[blocks[(nm, 0, d)][0]:blocks[(nm, 0, d)][0] + 4 * H] for nm in ("b_ih", "b_hh"))
        sg = lambda v: 1.0 / (1.0 + np.exp(-v))
        i, f, g, o = sg(a[:H]), sg(a[H:2 * H]), np.tanh(a[2 * H:3 * H]), sg(a[3 * H:])
        for t in range(dims.T):
            steps = t + 1 if d == 0 else dims.T - t
            c = i * g * (1 - f ** steps) / (1 - f)
            np.testing.assert_allclose(y[t, :, d * H:(d + 1) * H], np.broadcast_to(o * np.tanh(c), (dims.B, H)),
                                       rtol=0, atol=1e-14)


# -------------------------------------------------------------- invariances ---

def test_batch_permutation_permutes_outputs_and_keeps_gradient():
    dims = ref.Dims(L=2, D=6, H=8, P=5, K=7, T=5, B=4)
    theta, x, lab = _step_inputs(dims, seed=3)
    perm = np.array([2, 0, 3, 1])
    a = ref.learner_gradient(theta, dims, x, lab)
    b = ref.learner_gradient(theta, dims, x[:, perm], lab[:, perm])
    np.testing.assert_allclose(b["y_top"], a["y_top"][:, perm], rtol=0, atol=1e-14)
    np.testing.assert_allclose(b["grad"], a["grad"], rtol=1e-12, atol=1e-16)


def test_batch_gradient_is_mean_of_sequence_gradients():
    dims = ref.Dims(L=2, D=6, H=8, P=5, K=7, T=5, B=3)
    theta, x, lab = _step_inputs(dims, seed=4)
    full = ref.learner_gradient(theta, dims, x, lab)
    one = ref.Dims(L=2, D=6, H=8, P=5, K=7, T=5, B=1)
    per = [ref.learner_gradient(theta, one, x[:, b:b + 1], lab[:, b:b + 1]) for b in range(dims.B)]
    np.testing.assert_allclose(full["grad"], np.mean([p["grad"] for p in per], axis=0),
                               rtol=1e-11, atol=1e-16)
    np.testing.assert_allclose(full["loss"], np.mean([p["loss"] for p in per]), rtol=1e-13)


def test_time_reversal_swaps_directions():
    """Reversing the chunk in time and swapping the two directions' weights
    reverses the output in time and swaps its halves (one layer)."""
    dims = ref.Dims(L=1, D=6, H=8, P=5, K=7, T=6, B=2)
    theta, x, _ = _step_inputs(dims, seed=6)
    blocks, _ = ref.param_layout(dims)
    swapped = theta.copy()
    for name in ("W_ih", "W_hh", "b_ih", "b_hh"):
        o0, s0 = blocks[(name, 0, 0)]
        o1, _ = blocks[(name, 0, 1)]
        size = int(np.prod(s0))
        swapped[o0:o0 + size], swapped[o1:o1 + size] = theta[o1:o1 + size], theta[o0:o0 + size]
    y, _ = ref.blstm_forward(theta, dims, x)
    yr, _ = ref.blstm_forward(swapped, dims, x[::-1])
    H = dims.H
    np.testing.assert_allclose(yr[::-1, :, :H], y[:, :, H:], rtol=0, atol=1e-14)
    np.testing.assert_allclose(yr[::-1, :, H:], y[:, :, :H], rtol=0, atol=1e-14)


# ---------------------------------------------- planted mistakes are caught ---

def _fd_error(dims, theta, x, lab):
    g = ref.learner_gradient(theta, dims, x, lab)["grad"]
    eps = 1e-6
    rng = np.random.default_rng(11)
    idx = rng.choice(theta.size, size=60, replace=False)
    fd = []
    for k in idx:
        tp = theta.copy(); tp[k] += eps
        tm = theta.copy(); tm[k] -= eps
        fd.append((_loss(tp, dims, x, lab) - _loss(tm, dims, x, lab)) / (2 * eps))
    fd = np.array(fd)
    return np.linalg.norm(g[idx] - fd) / np.linalg.norm(fd)


MUTATIONS = {
    "drop_dc_next": ("dc = dh * o * (1.0 - tc * tc) + dc_next", "dc = dh * o * (1.0 - tc * tc)"),
    "sign_in_da_g": ("dc * i * (1.0 - g * g)", "dc * i * (1.0 + g * g)"),
    "c_prev_index": ("c_prev = cs[t_prev] if inside", "c_prev = cs[t] if inside"),
    "transposed_w_hh": ("dh_rec = da @ W_hh", "dh_rec = da @ W_hh.reshape(4, -1, W_hh.shape[1]).transpose(0, 2, 1).reshape(W_hh.shape)"),
    "wrong_step_order": ("t_prev = t + 1 if reverse else t - 1", "t_prev = t - 1 if reverse else t + 1"),
}


def _mutant(kind):
    """Recompile the oracle's BPTT with one planted mistake."""
    import inspect
    import textwrap
    src = textwrap.dedent(inspect.getsource(ref.lstm_direction_backward))
    old, new = MUTATIONS[kind]
    assert src.count(old) == 1, kind
    ns = {}
    exec(compile(src.replace(old, new), "<mutant>", "exec"), vars(ref), ns)
    return ns["lstm_direction_backward"]


@pytest.mark.parametrize("kind", sorted(MUTATIONS))
def test_planted_backward_mistakes_fail_the_fd_pin(monkeypatch, kind):
    dims = ref.Dims(L=1, D=3, H=4, P=3, K=5, T=4, B=2)
    theta, x, lab = _step_inputs(dims, seed=9)
    theta = theta * 10.0
    assert _fd_error(dims, theta, x, lab) < 1e-6
    monkeypatch.setattr(ref, "lstm_direction_backward", _mutant(kind))
    assert _fd_error(dims, theta, x, lab) > 1e-3


def test_planted_gate_order_mistake_fails_the_torch_pin(monkeypatch):
    dims = MICRO
    theta, x, lab = _step_inputs(dims, seed=2)
    orig = ref.lstm_direction_forward

    def swapped_gates(x_, W_ih, W_hh, b_ih, b_hh, reverse):
        H = W_hh.shape[1]
        perm = np.r_[H:2 * H, 0:H, 2 * H:4 * H]          # read i and f in the wrong order
        return orig(x_, W_ih[perm], W_hh[perm], b_ih[perm], b_hh[perm], reverse)

    monkeypatch.setattr(ref, "lstm_direction_forward", swapped_gates)
    got = ref.learner_gradient(theta, dims, x, lab)
    loss_t, y_t, _ = _torch_step(theta, dims, x, lab)
    assert np.abs(got["y_top"] - y_t).max() > 1e-4


# ----------------------------------------------------------- bf16 rounding ---

def test_bf16_round_matches_torch_and_special_values():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(10000).astype(np.float32) * 10.0,
                        np.array([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, 3.4e38, 1e-40, -1e-40,
                                  1.00390625, 1.01171875], dtype=np.float32)])
    ours = ref.bf16_round(x)
    theirs = torch.tensor(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, theirs)
    # ties go to even: 1 + 2^-8 is halfway between 1 and 1 + 2^-7
    assert ref.bf16_round(np.float32(1.00390625)) == 0x3F80
    assert ref.bf16_round(np.float32(1.01171875)) == 0x3F82
    assert ref.bf16_round(np.float32(np.nan)) == 0x7FC0


# ----------------------------------------------------------- the LR recipe ---

def test_lr_recipe_worked_example():
    rows = []
    with open(os.path.join(GOLDEN, "lr_recipe.txt")) as fh:
        for line in fh:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([float(v) for v in line.split()])
    base_lr, base_batch, batch = rows[0]
    for epoch, lr in rows[1:]:
        assert abs(ref.lr_schedule(int(epoch), base_lr, base_batch, batch) - lr) < 1e-12
