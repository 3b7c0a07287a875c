"""Training loop with the paper's learning-rate recipe (Section 3).

The rate for a total batch B is the baseline rate scaled by B / B_base
(linear scaling); it is reached linearly over the first ``warmup_epochs``
epochs (epoch e of the warm-up uses e / warmup_epochs of it) and divided by
sqrt(2) for every epoch after the warm-up.  Section 3's worked example: a
baseline of 0.1 at batch 256 and a total batch of 2560 give 0.1, 0.2, ...,
1.0 over epochs 1-10.

``Trainer`` runs a ``LearnerStep`` over a fixed set of device-resident
mini-batches, one learner step (gradient + fused update) per batch, with the
rate of the current epoch, and records the mean loss of each epoch.
"""

from __future__ import annotations

import math

import numpy as np
import torch


def lr_schedule(epoch: int, base_lr: float, base_batch: int, batch: int, warmup_epochs: int = 10) -> float:
    """Learning rate of 1-based ``epoch``."""
    if epoch < 1:
        raise ValueError("epochs count from 1")
    peak = base_lr * batch / base_batch
    if epoch <= warmup_epochs:
        return peak * epoch / warmup_epochs
    return peak / math.sqrt(2.0) ** (epoch - warmup_epochs)


class Trainer:
    def __init__(self, step, batches, base_lr: float, base_batch: int, warmup_epochs: int = 10, flags: int = 0):
        """step: a LearnerStep with its weights (and peer) loaded; batches:
        list of (features [T][B][D], labels [T][B]) numpy arrays, kept on the
        device.  The batch size of the recipe is the step's B (sequences).
        flags: the update's flags (ADPSGD_WRITE_PEER keeps the peer equal to
        the learner, which makes the update plain SGD at half the rate)."""
        self.step = step
        dev = step.device
        self.x = [torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(dev) for x, _ in batches]
        self.lab = [torch.from_numpy(np.ascontiguousarray(y, dtype=np.int32)).to(dev) for _, y in batches]
        self.base_lr, self.base_batch, self.warmup = base_lr, base_batch, warmup_epochs
        self.batch = step.shape["B"]
        self.flags = flags

    def run(self, epochs: int):
        """Returns [(epoch, lr, mean loss of the epoch's steps)]."""
        hist = []
        acc = torch.zeros(1, dtype=torch.float32, device=self.step.device)
        for e in range(1, epochs + 1):
            lr = lr_schedule(e, self.base_lr, self.base_batch, self.batch, self.warmup)
            acc.zero_()
            for x, y in zip(self.x, self.lab):
                self.step.x.copy_(x)
                self.step.labels.copy_(y)
                self.step.step(lr, self.flags)
                acc += self.step.loss
            torch.cuda.synchronize()
            self.step.check_recurrence()
            hist.append((e, lr, float(acc.cpu()[0]) / len(self.x)))
        return hist
