"""Oracle for one learner step of the H-ADPSGD acoustic-model training loop.

TEST INFRASTRUCTURE ONLY.  This module is the plain, slow and obviously
correct CPU definition that the HIP library is checked against.  Only the
test-suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it; the product path never does, and this module
imports nothing from the product package.

Everything is computed in float64 from float32 inputs, except the functions
whose name ends in ``_fp32``: those spell out one exact float32 operation
order for the parameter update so that a kernel following the same order can
be compared bit for bit.

What is computed, and where it comes from in the paper
(arXiv 1907.05701, "A Highly Efficient Distributed Deep Learning System for
Automatic Speech Recognition"):

* Model (Section 5.2, "DL Models and Dataset"): 6 bidirectional LSTM layers
  with 512 cells per direction, unrolled over 21 frames on non-overlapping
  chunks, a linear projection to 256 units, and a softmax over 32000
  context-dependent HMM states.  The paper names the framework (PyTorch,
  Section 5.1) but prints no cell equations; the cell is read as PyTorch's
  ``nn.LSTM`` (gate order i, f, g, o; no peepholes; separate input and
  recurrent biases), which reproduces the paper's "over 43 million
  parameters, about 165MB" (43,154,944 float32 values = 164.6 MiB).
* Objective (Section 2, eqs. 1-2): the frame cross-entropy, averaged over the
  B*T frames of the mini-batch (the 1/m of eq. 4 with m counted in frames;
  exposed as ``loss_scale``).
* Gradient (Section 2, eq. 4): the exact gradient of that loss, by
  back-propagation through time.
* Super-learner reduction (Section 2, eq. 6; Section 4): the learner-gradient
  average (1/lambda) * sum_i g_i, with the scale left as an argument.
* Local update (Section 2, eq. 7, one column): plain SGD (eq. 3, read as
  theta_{k+1} = theta_k - alpha_k g because the printed form applies F to both
  sides) combined with averaging against one ring neighbour with weights
  0.5/0.5 (the doubly stochastic T_k).  Two orders are offered: the default
  takes the SGD step first and then averages with the peer; ``order="eq7"``
  averages the pre-update weights and subtracts the full gradient step, as
  eq. 7 is printed.

Parity pins for every function live in ``tests/test_oracle_*.py``.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np


# --------------------------------------------------------------------------
# Shapes and the flat parameter layout (Section 5.2).
# --------------------------------------------------------------------------

@dataclass(frozen=True)
class Dims:
    """L layers, D input features, H cells per direction, P bottleneck units,
    K output classes, T unrolled frames, B sequences per mini-batch."""
    L: int
    D: int
    H: int
    P: int
    K: int
    T: int
    B: int


def layer_input_dim(dims: Dims, layer: int) -> int:
    """Layer 0 reads the features; every later layer reads both directions'
    hidden states of the layer below."""
    return dims.D if layer == 0 else 2 * dims.H


def param_layout(dims: Dims):
    """Return ({name: (offset, shape)}, total) for the flat float32 vector.

    Order follows PyTorch's ``nn.LSTM`` parameter list: for each layer, the
    forward direction then the reverse direction, each holding W_ih [4H, D_l],
    W_hh [4H, H], b_ih [4H], b_hh [4H] with gate row blocks i, f, g, o.  Then
    the bottleneck W_l [P, 2H], b_l [P] and the softmax layer W_s [K, P],
    b_s [K].  LSTM keys are (name, layer, direction)."""
    H = dims.H
    off = 0
    blocks = {}
    for layer in range(dims.L):
        dl = layer_input_dim(dims, layer)
        for direction in range(2):
            for name, shape in (("W_ih", (4 * H, dl)), ("W_hh", (4 * H, H)),
                                ("b_ih", (4 * H,)), ("b_hh", (4 * H,))):
                blocks[(name, layer, direction)] = (off, shape)
                off += int(np.prod(shape))
    for name, shape in (("W_l", (dims.P, 2 * H)), ("b_l", (dims.P,)),
                        ("W_s", (dims.K, dims.P)), ("b_s", (dims.K,))):
        blocks[name] = (off, shape)
        off += int(np.prod(shape))
    return blocks, off


def param_count(dims: Dims) -> int:
    return param_layout(dims)[1]


def unflatten(theta: np.ndarray, dims: Dims) -> dict:
    """Views of the flat vector, converted to float64 copies."""
    blocks, total = param_layout(dims)
    assert theta.shape == (total,), (theta.shape, total)
    out = {}
    for key, (off, shape) in blocks.items():
        size = int(np.prod(shape))
        out[key] = np.asarray(theta[off:off + size], dtype=np.float64).reshape(shape)
    return out


def flatten(parts: dict, dims: Dims) -> np.ndarray:
    """Inverse of ``unflatten`` (float64)."""
    blocks, total = param_layout(dims)
    flat = np.zeros(total, dtype=np.float64)
    for key, (off, shape) in blocks.items():
        flat[off:off + int(np.prod(shape))] = np.asarray(parts[key], dtype=np.float64).reshape(-1)
    return flat


# --------------------------------------------------------------------------
# The LSTM cell and the bidirectional stack (Section 5.2; cell as nn.LSTM).
# --------------------------------------------------------------------------

def sigmoid(a):
    # 1/(1+exp(-a)) written through tanh, which never overflows.
    return 0.5 * (np.tanh(0.5 * a) + 1.0)


def lstm_direction_forward(x, W_ih, W_hh, b_ih, b_hh, reverse):
    """One direction of one layer over a chunk.

    x: [T, B, D_l].  Processing order is t = 0..T-1 (forward direction) or
    t = T-1..0 (reverse direction); each chunk starts from h = c = 0 (the
    chunks are independent, non-overlapping subsequences).

    For each step, a = W_ih x_t + b_ih + W_hh h_prev + b_hh is split into
    gate blocks, i = sigmoid(a_i), f = sigmoid(a_f), g = tanh(a_g),
    o = sigmoid(a_o), then c_t = f*c_prev + i*g and h_t = o*tanh(c_t).

    Returns h [T, B, H] and a cache holding i, f, g, o, c per time index."""
    T, B, _ = x.shape
    H = W_hh.shape[1]
    h_prev = np.zeros((B, H))
    c_prev = np.zeros((B, H))
    hs = np.zeros((T, B, H))
    cs = np.zeros((T, B, H))
    gates = np.zeros((T, B, 4, H))
    steps = range(T - 1, -1, -1) if reverse else range(T)
    for t in steps:
        a = x[t] @ W_ih.T + b_ih + h_prev @ W_hh.T + b_hh
        i = sigmoid(a[:, 0:H])
        f = sigmoid(a[:, H:2 * H])
        g = np.tanh(a[:, 2 * H:3 * H])
        o = sigmoid(a[:, 3 * H:4 * H])
        c = f * c_prev + i * g
        h = o * np.tanh(c)
        hs[t], cs[t] = h, c
        gates[t, :, 0], gates[t, :, 1], gates[t, :, 2], gates[t, :, 3] = i, f, g, o
        h_prev, c_prev = h, c
    return hs, {"c": cs, "gates": gates}


def lstm_direction_backward(dh_out, x, hs, cache, W_ih, W_hh, reverse):
    """Back-propagation through time for one direction of one layer.

    dh_out: [T, B, H], the loss gradient reaching h_t from above.  Steps run
    in the opposite order of the forward pass.  With tc = tanh(c_t):
        dh   = dh_out[t] + dh_rec
        dc   = dh*o*(1 - tc^2) + dc_next
        da_o = dh*tc*o*(1-o);   da_i = dc*g*i*(1-i)
        da_g = dc*i*(1-g^2);    da_f = dc*c_prev*f*(1-f)
        dc_next = dc*f;         dh_rec = W_hh^T da
    and the parameter gradients accumulate da x_t^T, da h_prev^T and da (the
    same da feeds both biases).  Returns (dW_ih, dW_hh, db, dx)."""
    T, B, H = hs.shape
    cs, gates = cache["c"], cache["gates"]
    dW_ih = np.zeros_like(W_ih)
    dW_hh = np.zeros_like(W_hh)
    db = np.zeros(4 * H)
    dx = np.zeros(x.shape)
    dh_rec = np.zeros((B, H))
    dc_next = np.zeros((B, H))
    steps = range(T) if reverse else range(T - 1, -1, -1)
    for t in steps:
        t_prev = t + 1 if reverse else t - 1        # the step before t in the forward pass
        inside = 0 <= t_prev < T
        h_prev = hs[t_prev] if inside else np.zeros((B, H))
        c_prev = cs[t_prev] if inside else np.zeros((B, H))
        i, f, g, o = (gates[t, :, k] for k in range(4))
        tc = np.tanh(cs[t])
        dh = dh_out[t] + dh_rec
        dc = dh * o * (1.0 - tc * tc) + dc_next
        da = np.concatenate([dc * g * i * (1.0 - i),
                             dc * c_prev * f * (1.0 - f),
                             dc * i * (1.0 - g * g),
                             dh * tc * o * (1.0 - o)], axis=1)
        dW_ih += da.T @ x[t]
        dW_hh += da.T @ h_prev
        db += da.sum(axis=0)
        dx[t] += da @ W_ih
        dh_rec = da @ W_hh
        dc_next = dc * f
    return dW_ih, dW_hh, db, dx


def blstm_forward(theta, dims: Dims, x):
    """The bidirectional stack.  x: [T, B, D] float32/64.  Returns the top
    layer's output y [T, B, 2H] (forward half first) and the per-layer caches
    needed by ``blstm_backward``."""
    p = unflatten(theta, dims)
    inp = np.asarray(x, dtype=np.float64)
    caches = []
    for layer in range(dims.L):
        halves, per_dir = [], []
        for d in range(2):
            hs, cache = lstm_direction_forward(
                inp, p[("W_ih", layer, d)], p[("W_hh", layer, d)],
                p[("b_ih", layer, d)], p[("b_hh", layer, d)], reverse=(d == 1))
            halves.append(hs)
            per_dir.append((hs, cache))
        caches.append((inp, per_dir))
        inp = np.concatenate(halves, axis=2)
    return inp, caches


def blstm_backward(theta, dims: Dims, caches, dy_top):
    """Gradient of the LSTM parameters given dL/dy_top [T, B, 2H].  Returns a
    dict keyed like ``param_layout`` (LSTM entries only)."""
    p = unflatten(theta, dims)
    H = dims.H
    grads = {}
    dy = np.asarray(dy_top, dtype=np.float64)
    for layer in range(dims.L - 1, -1, -1):
        inp, per_dir = caches[layer]
        dx_total = np.zeros(inp.shape)
        for d in range(2):
            hs, cache = per_dir[d]
            dW_ih, dW_hh, db, dx = lstm_direction_backward(
                dy[:, :, d * H:(d + 1) * H], inp, hs, cache,
                p[("W_ih", layer, d)], p[("W_hh", layer, d)], reverse=(d == 1))
            grads[("W_ih", layer, d)] = dW_ih
            grads[("W_hh", layer, d)] = dW_hh
            grads[("b_ih", layer, d)] = db
            grads[("b_hh", layer, d)] = db.copy()
            dx_total += dx
        dy = dx_total
    return grads


# --------------------------------------------------------------------------
# Bottleneck, softmax and frame cross-entropy (Section 5.2; eqs. 1-2, 4).
# --------------------------------------------------------------------------

def head_forward_backward(theta, dims: Dims, y_top, labels, loss_scale=None):
    """z = W_l y + b_l (linear, no nonlinearity), s = W_s z + b_s,
    per-frame loss l = logsumexp(s) - s[label], L = loss_scale * sum l with
    loss_scale = 1/(B*T) by default.  Returns (L, per-frame losses [T, B],
    dL/dy_top [T, B, 2H], dict of head gradients)."""
    p = unflatten(theta, dims)
    T, B = dims.T, dims.B
    scale = 1.0 / (B * T) if loss_scale is None else float(loss_scale)
    y = np.asarray(y_top, dtype=np.float64).reshape(T * B, 2 * dims.H)
    lab = np.asarray(labels).reshape(T * B).astype(np.int64)
    z = y @ p["W_l"].T + p["b_l"]
    s = z @ p["W_s"].T + p["b_s"]
    smax = s.max(axis=1, keepdims=True)
    lse = smax[:, 0] + np.log(np.exp(s - smax).sum(axis=1))
    rows = np.arange(T * B)
    ell = lse - s[rows, lab]
    loss = scale * ell.sum()
    ds = np.exp(s - lse[:, None])
    ds[rows, lab] -= 1.0
    ds *= scale
    grads = {"W_s": ds.T @ z, "b_s": ds.sum(axis=0)}
    dz = ds @ p["W_s"]
    grads["W_l"] = dz.T @ y
    grads["b_l"] = dz.sum(axis=0)
    dy = dz @ p["W_l"]
    return loss, ell.reshape(T, B), dy.reshape(T, B, 2 * dims.H), grads


def learner_gradient(theta, dims: Dims, x, labels, loss_scale=None):
    """Loss and g(theta, xi) (eq. 4) for one mini-batch, as a flat float64
    vector in the ``param_layout`` order.  Also returns y_top and dy_top."""
    y_top, caches = blstm_forward(theta, dims, x)
    loss, ell, dy_top, head = head_forward_backward(theta, dims, y_top, labels, loss_scale)
    lstm = blstm_backward(theta, dims, caches, dy_top)
    grads = dict(lstm)
    grads.update(head)
    return {"loss": loss, "frame_loss": ell, "grad": flatten(grads, dims),
            "y_top": y_top, "dy_top": dy_top}


# --------------------------------------------------------------------------
# Super-learner reduction and the ADPSGD local update (eqs. 3, 6, 7).
# --------------------------------------------------------------------------

def replica_grad_reduce(grads, scale):
    """scale * sum_r g_r in float64 (eq. 6's bracket with scale = 1/lambda)."""
    acc = np.zeros(np.asarray(grads[0]).shape, dtype=np.float64)
    for g in grads:
        acc += np.asarray(g, dtype=np.float64)
    return scale * acc


def adpsgd_update(theta, theta_peer, g, lr, order="sgd_then_avg"):
    """One column of eq. 7 with T_k pairing this learner and one neighbour at
    weights 0.5/0.5.  Returns the new weights (the peer receives the same
    value when the pair is updated together).

    order="sgd_then_avg":  0.5 * ((theta - lr*g) + theta_peer)
    order="eq7":           0.5 * (theta + theta_peer) - lr*g"""
    th = np.asarray(theta, dtype=np.float64)
    pe = np.asarray(theta_peer, dtype=np.float64)
    gg = np.asarray(g, dtype=np.float64)
    if order == "sgd_then_avg":
        return 0.5 * ((th - lr * gg) + pe)
    if order == "eq7":
        return 0.5 * (th + pe) - lr * gg
    raise ValueError(order)


def replica_grad_reduce_fp32(grads, scale):
    """float32 order: s = g_0; s = s + g_r for r = 1..R-1; out = s * scale.
    Each operation is one IEEE-754 binary32 operation, rounded to nearest
    even, with no fused multiply-add."""
    s = np.array(grads[0], dtype=np.float32, copy=True)
    for g in grads[1:]:
        s = (s + np.asarray(g, dtype=np.float32)).astype(np.float32)
    return (s * np.float32(scale)).astype(np.float32)


def adpsgd_update_fp32(theta, theta_peer, grads, scale, lr, order="sgd_then_avg"):
    """The fused reduce + update in one fixed float32 operation order:
    g = reduce_fp32(grads, scale); t = lr*g; then
    sgd_then_avg: u = theta - t; v = u + peer; new = v*0.5
    eq7:          v = theta + peer; a = v*0.5; new = a - t"""
    g = replica_grad_reduce_fp32(grads, scale)
    th = np.asarray(theta, dtype=np.float32)
    pe = np.asarray(theta_peer, dtype=np.float32)
    t = (np.float32(lr) * g).astype(np.float32)
    if order == "sgd_then_avg":
        u = (th - t).astype(np.float32)
        v = (u + pe).astype(np.float32)
        return (v * np.float32(0.5)).astype(np.float32)
    if order == "eq7":
        v = (th + pe).astype(np.float32)
        a = (v * np.float32(0.5)).astype(np.float32)
        return (a - t).astype(np.float32)
    raise ValueError(order)


def bf16_round(x):
    """float32 -> bfloat16 by round-to-nearest-even on the upper 16 bits,
    returned as uint16 bit patterns.  NaN maps to a quiet NaN."""
    xf = np.atleast_1d(np.asarray(x, dtype=np.float32))
    u = xf.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    out = rounded.astype(np.uint16)
    out[np.isnan(xf)] = 0x7FC0
    return out.reshape(np.shape(x))


def bf16_to_float(bits):
    """uint16 bfloat16 patterns -> float32 values."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------
# Learning-rate recipe (Section 3): linear scaling, warm-up, annealing.
# --------------------------------------------------------------------------

def lr_schedule(epoch, base_lr, base_batch, batch, warmup_epochs=10):
    """Learning rate for 1-based ``epoch``: the target rate is base_lr scaled
    by batch/base_batch; it is reached linearly over the first
    ``warmup_epochs`` epochs and then divided by sqrt(2) per further epoch."""
    target = base_lr * batch / base_batch
    if epoch <= warmup_epochs:
        return target * epoch / warmup_epochs
    return target * math.sqrt(0.5) ** (epoch - warmup_epochs)


# --------------------------------------------------------------------------
# The ring of learners (Section 2, eq. 7; Section 4): several learners'
# columns of Theta, each super-learner's gradient the mean of its replicas.
# --------------------------------------------------------------------------

def ring_partner(s, k, n):
    """The neighbour learner s averages with in round k of an n-learner ring:
    T_k pairs every learner with one ring neighbour, the right one when
    s + k is even and the left one otherwise, so that consecutive rounds
    alternate between the two neighbours and every round is a perfect
    matching (n must be even)."""
    if n < 2 or n % 2:
        raise ValueError("the ring pairing needs an even number of learners")
    return (s + 1) % n if (s + k) % 2 == 0 else (s - 1) % n


def ring_matrix(k, n):
    """T_k of eq. 7 for round k: 0.5 on the diagonal and at each learner's
    partner (symmetric, rows and columns summing to 1)."""
    T = np.zeros((n, n))
    for s in range(n):
        T[s, s] += 0.5
        T[ring_partner(s, k, n), s] += 0.5
    return T


def ring_round(thetas, grads, lr, k, peers=None):
    """One round of eq. 7 for n learners: Theta_{k+1} = W T_k - lr * G, where
    column s of G is learner s's gradient and W holds the weights the
    averaging reads: the round-start weights themselves (peers=None), or an
    earlier round's weights (a learner reading stale peer copies, as in the
    asynchronous variant).  The learner's own column of W is its current
    weight vector in either case.  Returns the list of new weight vectors.

    With super-learners (Section 4), grads[s] is already the mean of the
    replica gradients (replica_grad_reduce with scale 1/N, eq. 6)."""
    n = len(thetas)
    cur = [np.asarray(t, dtype=np.float64) for t in thetas]
    src = cur if peers is None else [np.asarray(t, dtype=np.float64) for t in peers]
    out = []
    for s in range(n):
        p = ring_partner(s, k, n)
        out.append(0.5 * cur[s] + 0.5 * src[p] - lr * np.asarray(grads[s], dtype=np.float64))
    return out
