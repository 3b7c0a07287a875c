"""GPU: the training loop with the learning-rate recipe lowers the loss on
a fixed synthetic data set (random labels, memorised)."""

import numpy as np
import pytest

from oracle import blstm_ref as ref
from paper_1907_05701_amd import inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("precision", ["fp32", "bf16"])
def test_loss_decreases_over_epochs(gpu_lib, precision):
    from paper_1907_05701_amd.step import LearnerStep
    from paper_1907_05701_amd.train import Trainer
    shape = dict(L=1, D=40, H=64, P=32, K=100, T=21, B=8)
    dims = ref.Dims(**shape)
    theta = inputs.params(ref.param_count(dims), seed=90)
    batches = [(inputs.features(dims.T, dims.B, dims.D, seed=91 + i), inputs.labels(dims.T, dims.B, dims.K, seed=95 + i))
               for i in range(2)]
    st = LearnerStep(**shape, precision=precision)
    st.load(theta, *batches[0], inputs.peer(theta))
    from paper_1907_05701_amd import binding as bd
    st.peer.copy_(st.theta)   # the peer follows the learner: plain SGD at half the rate
    # 16 steps per epoch (the two batches 8 times), the recipe's 10-epoch
    # warm-up to 4.0 (measured: fp32 and bf16 both fall from ln 100 = 4.6 to
    # below 0.1 by epoch 12; a peak of 10 diverges in bf16)
    hist = Trainer(st, batches * 8, base_lr=4.0, base_batch=8, warmup_epochs=10,
                   flags=bd.ADPSGD_WRITE_PEER).run(12)
    print("[train]", [(e, round(lr, 4), round(l, 4)) for e, lr, l in hist], flush=True)
    losses = [l for _, _, l in hist]
    assert np.isfinite(losses).all()
    assert losses[-1] < 0.1 * losses[0], losses
    assert losses[-1] < losses[-2] < losses[-3], losses
