"""A ring of learners on one GPU (Section 2, eq. 7; Section 4).

``LearnerRing`` holds S super-learners of N replicas each.  A round runs, for
every super-learner, the N replica gradients at its weights (each replica
its own mini-batch) and then one column of eq. 7 through ``adpsgd_step``
(order eq. 7: the replica gradients summed with scale 1/N as in eq. 6, the
weights averaged 0.5/0.5 with the ring partner of this round, the bf16
operand copy refreshed).  The partner alternates between the right and the
left neighbour from round to round, so every round pairs the learners off
(S must be even).

The averaging reads a copy of the partner's weights taken at the start of
the round (``staleness=0``: every pair averages the same two vectors, the
sum over learners is kept) or at the start of the previous round
(``staleness=1``: the stale reads of the asynchronous variant, on a fixed
schedule).

Overlap: the gradient calls of all learners run in order on the current
stream (two persistent recurrent launches must never run at the same time,
each needs every CU); a learner's update, which only streams HBM, runs on a
second stream while the next learner computes its gradients.  The
exchange between learners on different GPUs, and real asynchrony, are not
part of this library.
"""

from __future__ import annotations

import numpy as np
import torch

from . import binding as bd
from .step import LearnerStep


def partner(s: int, k: int, n: int) -> int:
    """Ring neighbour of learner s in round k: right when s + k is even,
    left otherwise."""
    if n < 2 or n % 2:
        raise ValueError("the ring needs an even number of super-learners")
    return (s + 1) % n if (s + k) % 2 == 0 else (s - 1) % n


class LearnerRing:
    def __init__(self, shape: dict, n_super: int, n_replicas: int = 1, precision: str = "bf16",
                 staleness: int = 0, overlap: bool = True, device: str = "cuda:0"):
        if staleness not in (0, 1):
            raise ValueError("staleness is 0 or 1 rounds")
        partner(0, 0, n_super)   # validates n_super
        self.S, self.N, self.staleness = n_super, n_replicas, staleness
        self.steps = [[LearnerStep(**shape, precision=precision, device=device) for _ in range(n_replicas)]
                      for _ in range(n_super)]
        # the replicas of a super-learner compute at its weights: they share
        # replica 0's weight vector and bf16 copy
        for reps in self.steps:
            for r in range(1, n_replicas):
                reps[r].theta = reps[0].theta
                reps[r].theta_lp = reps[0].theta_lp
        self.snap = [[torch.empty_like(reps[0].theta) for _ in range(2)] for reps in self.steps]
        self.side = torch.cuda.Stream(device=device) if overlap else None
        self.k = 0
        self.frames_per_round = n_super * n_replicas * shape["T"] * shape["B"]

    def theta(self, s: int) -> torch.Tensor:
        return self.steps[s][0].theta

    def load(self, thetas, batches):
        """thetas[s]: float32 weights of super-learner s; batches[s][r]:
        (features [T][B][D], labels [T][B]) of replica r."""
        for s, reps in enumerate(self.steps):
            for r, st in enumerate(reps):
                x, lab = batches[s][r]
                if r == 0:
                    st.load(thetas[s], x, lab)
                else:
                    st.x.copy_(torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)))
                    st.labels.copy_(torch.from_numpy(np.ascontiguousarray(lab, dtype=np.int32)))
        for s in range(self.S):
            self.snap[s][1].copy_(self.theta(s))   # "previous round" copy for the first stale round
        self.k = 0

    def round(self, lr: float):
        k, S = self.k, self.S
        main = torch.cuda.current_stream()
        # round-start copies (what the partners' averaging reads)
        for s in range(S):
            self.snap[s][k % 2].copy_(self.theta(s))
        for s in range(S):
            for st in self.steps[s]:
                st.gradient()
            p = partner(s, k, S)
            peer = self.snap[p][k % 2] if self.staleness == 0 else self.snap[p][(k + 1) % 2]
            grads = [st.grad for st in self.steps[s]]
            lead = self.steps[s][0]
            if self.side is None:
                bd.adpsgd_step(lead.theta, peer, grads, 1.0 / self.N, lr, bd.ADPSGD_ORDER_EQ7, lead.theta_lp)
            else:
                # the update streams HBM while the next learner computes
                self.side.wait_stream(main)
                bd.adpsgd_step(lead.theta, peer, grads, 1.0 / self.N, lr, bd.ADPSGD_ORDER_EQ7, lead.theta_lp,
                               stream=self.side)
        if self.side is not None:
            main.wait_stream(self.side)
        self.k += 1

    def check_recurrence(self):
        for reps in self.steps:
            for st in reps:
                st.check_recurrence()
