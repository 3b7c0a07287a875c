"""One learner step on the GPU through the C ABI.

``LearnerStep`` owns the device buffers of one learner (torch allocations:
memory only) and runs, per step, the five library calls in order:
blstm_fwd -> softmax_ce_fwd_bwd -> blstm_bwd -> adpsgd_step (which also
refreshes the bf16 operand copy for the next step).  Nothing here computes
anything; it only marshals arguments."""

from __future__ import annotations

import numpy as np
import torch

from . import binding as bd


class LearnerStep:
    def __init__(self, L, D, H, P, K, T, B, precision="bf16", device="cuda:0"):
        self.dims = bd.make_dims(L, D, H, P, K, T, B, precision)
        self.shape = dict(L=L, D=D, H=H, P=P, K=K, T=T, B=B)
        self.precision = precision
        self.device = torch.device(device)
        self.n = bd.blstm_param_count(self.dims)
        sizes = bd.blstm_workspace_bytes(self.dims)
        self.sizes = sizes
        dev = self.device
        act_dtype = torch.bfloat16 if precision == "bf16" else torch.float32
        self.act_dtype = act_dtype
        self.theta = torch.empty(self.n, dtype=torch.float32, device=dev)
        self.peer = torch.empty(self.n, dtype=torch.float32, device=dev)
        self.grad = torch.empty(self.n, dtype=torch.float32, device=dev)
        self.theta_lp = (torch.empty(self.n, dtype=torch.bfloat16, device=dev)
                         if precision == "bf16" else None)
        self.x = torch.empty((T, B, D), dtype=torch.float32, device=dev)
        self.labels = torch.empty((T, B), dtype=torch.int32, device=dev)
        self.y_top = torch.empty((T, B, 2 * H), dtype=act_dtype, device=dev)
        self.dy_top = torch.empty((T, B, 2 * H), dtype=torch.float32, device=dev)
        self.loss = torch.zeros(1, dtype=torch.float32, device=dev)
        self.act_ws = torch.empty(max(sizes["act_ws"], 1), dtype=torch.uint8, device=dev)
        self.head_ws = torch.empty(max(sizes["head_ws"], 1), dtype=torch.uint8, device=dev)
        self.loss_scale = 1.0 / (T * B)

    # ---------------------------------------------------------------- data ---
    def load(self, theta, x, labels, peer=None):
        self.theta.copy_(torch.from_numpy(np.ascontiguousarray(theta, dtype=np.float32)))
        self.x.copy_(torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)))
        self.labels.copy_(torch.from_numpy(np.ascontiguousarray(labels, dtype=np.int32)))
        if peer is not None:
            self.peer.copy_(torch.from_numpy(np.ascontiguousarray(peer, dtype=np.float32)))
        self.pack()

    def pack(self):
        if self.theta_lp is not None:
            bd.blstm_pack_params(self.dims, self.theta, self.theta_lp)

    # ---------------------------------------------------------- the calls ---
    def forward(self):
        bd.blstm_fwd(self.dims, self.theta, self.theta_lp, self.x, self.act_ws, self.y_top)

    def head(self, y_top=None):
        bd.softmax_ce_fwd_bwd(self.dims, self.theta, self.theta_lp,
                              self.y_top if y_top is None else y_top, self.labels,
                              self.loss_scale, self.loss, self.dy_top, self.grad, self.head_ws)

    def backward(self, dy_top=None):
        bd.blstm_bwd(self.dims, self.theta, self.theta_lp, self.act_ws, self.y_top,
                     self.dy_top if dy_top is None else dy_top, self.grad)

    def gradient(self):
        self.forward()
        self.head()
        self.backward()

    def check_recurrence(self):
        """Raises if a recurrent exchange wait gave up since the last forward
        call (synchronises the current stream)."""
        bd.blstm_recurrence_ok(self.dims, self.act_ws)

    def update(self, lr, flags=0, grads=None, scale=1.0):
        bd.adpsgd_step(self.theta, self.peer, [self.grad] if grads is None else grads, scale, lr,
                       flags, self.theta_lp)

    def step(self, lr, flags=0):
        """The whole learner step: gradient, then the fused update."""
        self.gradient()
        self.update(lr, flags)

    def capture(self, lr, steps=1, flags=0):
        """Record `steps` learner steps into a HIP graph (replaying it runs
        them again on the current buffers, i.e. continues training)."""
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(steps):
                self.step(lr, flags)
        return graph
