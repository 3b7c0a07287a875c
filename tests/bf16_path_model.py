"""Float64 model of where the library's bf16 path rounds (test infrastructure).

The oracle defines what the learner step computes; this module does the same
arithmetic in float64 but rounds to bfloat16 (round to nearest even) at the
points where the HIP path stores or feeds an MFMA with a bf16 value.  Each
rounding point can be switched on or off, so a test can tell which of them
moves a result and by how much: with every point off this is the exact
step, with every point on it is the bf16 path up to float32 accumulation
order (relative 1e-6 or so, far below the bf16 effects it measures).

Nothing here is part of the product, and nothing here is shared with the HIP
code; it follows the cell of PyTorch's nn.LSTM (Section 5.2 of the paper)
and the frame cross-entropy of eqs. 1-2 and 4, written out again with the
rounding points inserted.

Rounding points (names used in ``points``):
  x      features as the MFMA operand of the layer-0 input projection
  w      every weight matrix as an MFMA operand (W_ih, W_hh, W_l, W_s)
  gx     the stored input projection X W_ih^T + b_ih + b_hh
  hrec   h of the previous step as the operand of the recurrent product
  y      layer outputs (next layer's input, dW_hh and head operands)
  pre    the saved gate pre-activations the backward evaluates sigma/tanh from
  z      the bottleneck output z
  s      the stored logits
  ds     ds = scale (softmax - onehot) as the operand of dW_s, dz and db_s
  dz     dz as the operand of dW_l and dy
  da     the gate-gradient da as the operand of dW_ih, dW_hh, dX, db and of
         the recurrent partial product
  part   each recurrent workgroup's partial sum of dh_rec (from the gate
         rows of its member_units hidden units) rounded before the partials
         are added

``PATH_POINTS`` is the set the library rounds at (all but "s": its logits
are float32).
"""

from __future__ import annotations

import numpy as np

ALL_POINTS = ("x", "w", "gx", "hrec", "y", "pre", "z", "s", "ds", "dz", "da", "part")
# the points where the library's bf16 path rounds (its logits are float32)
PATH_POINTS = tuple(p for p in ALL_POINTS if p != "s")
MEMBER_UNITS = 64   # hidden units whose gate rows one recurrent workgroup owns


def bf(v):
    """float64 -> the float64 value of its bfloat16 (via float32, round to
    nearest even on the upper 16 bits)."""
    f = np.asarray(v, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000).astype(np.uint32)
    return u.view(np.float32).astype(np.float64)


def _sig(a):
    return 0.5 * (np.tanh(0.5 * a) + 1.0)


def _layout(L, D, H, P, K):
    off, blocks = 0, {}
    for l in range(L):
        dl = D if l == 0 else 2 * H
        for d in range(2):
            for name, shape in (("W_ih", (4 * H, dl)), ("W_hh", (4 * H, H)), ("b_ih", (4 * H,)), ("b_hh", (4 * H,))):
                blocks[(name, l, d)] = (off, shape)
                off += int(np.prod(shape))
    for name, shape in (("W_l", (P, 2 * H)), ("b_l", (P,)), ("W_s", (K, P)), ("b_s", (K,))):
        blocks[name] = (off, shape)
        off += int(np.prod(shape))
    return blocks, off


def _rounders(points):
    on = set(points)
    unknown = on - set(ALL_POINTS)
    if unknown:
        raise ValueError(f"unknown rounding points {sorted(unknown)}")
    return {p: (bf if p in on else (lambda v: np.asarray(v, dtype=np.float64))) for p in ALL_POINTS}


def _params(theta, shape, r):
    L, D, H, P, K = (shape[k] for k in "LDHPK")
    blocks, n = _layout(L, D, H, P, K)
    th = np.asarray(theta, dtype=np.float64)
    p = {k: th[o:o + int(np.prod(s))].reshape(s) for k, (o, s) in blocks.items()}
    is_w = lambda k: (k if isinstance(k, str) else k[0]).startswith("W")
    wq = {k: (r["w"](v) if is_w(k) else v) for k, v in p.items()}
    return blocks, n, p, wq


def _head(p, wq, yf, labels, r, scale):
    """Bottleneck, logits, frame cross-entropy and their backward for the
    frames yf [M, 2H] (already in the precision the products read)."""
    M = yf.shape[0]
    z = r["z"](yf @ wq["W_l"].T + p["b_l"])
    s = r["s"](z @ wq["W_s"].T + p["b_s"])
    lab = np.asarray(labels).reshape(M).astype(np.int64)
    mx = s.max(axis=1, keepdims=True)
    lse = mx[:, 0] + np.log(np.exp(s - mx).sum(axis=1))
    rows = np.arange(M)
    loss = scale * (lse - s[rows, lab]).sum()
    ds = np.exp(s - lse[:, None])
    ds[rows, lab] -= 1.0
    ds = r["ds"](scale * ds)
    grads = {"W_s": ds.T @ z, "b_s": ds.sum(axis=0)}
    dz = ds @ wq["W_s"]
    grads["b_l"] = dz.sum(axis=0)
    dzq = r["dz"](dz)
    grads["W_l"] = dzq.T @ yf
    return loss, grads, dzq @ wq["W_l"]


def head_gradient(theta, shape, y_top, labels, points=PATH_POINTS, loss_scale=None):
    """The head alone on given top-layer outputs y_top [T, B, 2H]: loss,
    dict of head gradients (W_l, b_l, W_s, b_s) and dy_top."""
    r = _rounders(points)
    T, B, H = shape["T"], shape["B"], shape["H"]
    M = T * B
    _, _, p, wq = _params(theta, shape, r)
    scale = 1.0 / M if loss_scale is None else float(loss_scale)
    yf = r["y"](np.asarray(y_top, dtype=np.float64).reshape(M, 2 * H))
    loss, grads, dy = _head(p, wq, yf, labels, r, scale)
    return loss, grads, dy.reshape(T, B, 2 * H)


def learner_gradient(theta, shape, x, labels, points=PATH_POINTS, loss_scale=None, member_units=MEMBER_UNITS):
    """Loss, flat gradient, y_top and dy_top of one learner step with the
    chosen rounding points.  shape: dict with L, D, H, P, K, T, B."""
    r = _rounders(points)
    L, D, H, P, K, T, B = (shape[k] for k in "LDHPKTB")
    blocks, n, p, wq = _params(theta, shape, r)
    M = T * B
    scale = 1.0 / M if loss_scale is None else float(loss_scale)

    # ---- forward
    inp = r["x"](np.asarray(x, dtype=np.float64))
    saved = []
    for l in range(L):
        outs, per = [], []
        for d in range(2):
            Wih, Whh = wq[("W_ih", l, d)], wq[("W_hh", l, d)]
            gx = r["gx"](inp.reshape(M, -1) @ Wih.T + p[("b_ih", l, d)] + p[("b_hh", l, d)]).reshape(T, B, 4 * H)
            h = np.zeros((B, H))
            c = np.zeros((B, H))
            hs, cs, pre = np.zeros((T, B, H)), np.zeros((T, B, H)), np.zeros((T, B, 4 * H))
            for t in (range(T - 1, -1, -1) if d else range(T)):
                a = gx[t] + r["hrec"](h) @ Whh.T
                pre[t] = a
                i, f, g, o = _sig(a[:, :H]), _sig(a[:, H:2 * H]), np.tanh(a[:, 2 * H:3 * H]), _sig(a[:, 3 * H:])
                c = f * c + i * g
                h = o * np.tanh(c)
                hs[t], cs[t] = h, c
            outs.append(hs)
            per.append((hs, cs, r["pre"](pre)))
        saved.append((inp, per))
        inp = r["y"](np.concatenate(outs, axis=2))
    y_top = inp

    # ---- head
    loss, hgrads, dy = _head(p, wq, y_top.reshape(M, 2 * H), labels, r, scale)
    grads = dict(hgrads)
    dy = dy.reshape(T, B, 2 * H)
    dy_top = dy.copy()

    # ---- BPTT
    mu = min(member_units, H)
    own = [np.concatenate([np.arange(q * H + m * mu, q * H + (m + 1) * mu) for q in range(4)])
           for m in range(H // mu)]
    for l in range(L - 1, -1, -1):
        inp, per = saved[l]
        dx = np.zeros(inp.shape)
        for d in range(2):
            hs, cs, pre = per[d]
            hq = r["y"](hs)
            Wih, Whh = wq[("W_ih", l, d)], wq[("W_hh", l, d)]
            dWih, dWhh, db = np.zeros(Wih.shape), np.zeros(Whh.shape), np.zeros(4 * H)
            dh_rec, dc_next = np.zeros((B, H)), np.zeros((B, H))
            for t in (range(T) if d else range(T - 1, -1, -1)):
                tp = t + 1 if d else t - 1
                inside = 0 <= tp < T
                h_prev = hq[tp] if inside else np.zeros((B, H))
                c_prev = cs[tp] if inside else np.zeros((B, H))
                a = pre[t]
                i, f, g, o = _sig(a[:, :H]), _sig(a[:, H:2 * H]), np.tanh(a[:, 2 * H:3 * H]), _sig(a[:, 3 * H:])
                tc = np.tanh(cs[t])
                dh = dy[t, :, d * H:(d + 1) * H] + dh_rec
                dc = dh * o * (1.0 - tc * tc) + dc_next
                da = r["da"](np.concatenate([dc * g * i * (1.0 - i), dc * c_prev * f * (1.0 - f),
                                             dc * i * (1.0 - g * g), dh * tc * o * (1.0 - o)], axis=1))
                dWih += da.T @ inp[t]
                dWhh += da.T @ h_prev
                db += da.sum(axis=0)
                dx[t] += da @ Wih
                dh_rec = sum(r["part"](da[:, rows_m] @ Whh[rows_m]) for rows_m in own)
                dc_next = dc * f
            grads[("W_ih", l, d)], grads[("W_hh", l, d)] = dWih, dWhh
            grads[("b_ih", l, d)], grads[("b_hh", l, d)] = db, db.copy()
        dy = dx
    flat = np.zeros(n)
    for k, (o, s_) in blocks.items():
        flat[o:o + int(np.prod(s_))] = np.asarray(grads[k]).reshape(-1)
    return {"loss": loss, "grad": flat, "y_top": y_top, "dy_top": dy_top, "blocks": blocks}
