"""GPU: the allocation-free head entry point (softmax_ce_fwd_bwd_static,
whose workspace is a static device array) against softmax_ce_fwd_bwd with a
caller workspace, through the C ABI: two calls in a row, the second with a
smaller input, each bit for bit equal to the workspace variant; dims whose
head workspace exceeds the static array are rejected before any launch."""

import numpy as np
import pytest
import torch

from oracle import blstm_ref as ref
from paper_1907_05701_amd import inputs

pytestmark = pytest.mark.gpu


def _compare(shape, precision, seed):
    from paper_1907_05701_amd import binding as bd
    from paper_1907_05701_amd.step import LearnerStep
    dims = ref.Dims(**shape)
    n = ref.param_count(dims)
    print(f"[static head] shape={shape} precision={precision} seed={seed}", flush=True)
    st = LearnerStep(**shape, precision=precision)
    assert st.sizes["head_ws"] <= bd.HEAD_STATIC_SCRATCH_BYTES
    theta = inputs.params(n, seed=seed)
    st.load(theta, np.zeros((dims.T, dims.B, dims.D), np.float32),
            inputs.labels(dims.T, dims.B, dims.K, seed=seed + 1, dist="zipf"))
    y = inputs.hidden_states(dims.T, dims.B, 2 * dims.H, seed=seed + 2)
    st.y_top.copy_(torch.from_numpy(y).to(st.act_dtype))
    st.grad.fill_(0.0)
    st.head()
    loss2 = torch.full_like(st.loss, float("nan"))
    dy2 = torch.full_like(st.dy_top, float("nan"))
    grad2 = torch.zeros_like(st.grad)
    bd.softmax_ce_fwd_bwd_static(st.dims, st.theta, st.theta_lp, st.y_top, st.labels, st.loss_scale, loss2, dy2,
                                 grad2)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(loss2.cpu().numpy(), st.loss.cpu().numpy())
    np.testing.assert_array_equal(dy2.cpu().numpy(), st.dy_top.cpu().numpy())
    np.testing.assert_array_equal(grad2.cpu().numpy(), st.grad.cpu().numpy())
    assert np.isfinite(loss2.cpu().numpy()).all()


def test_static_head_matches_workspace_head_twice(gpu_lib):
    _compare(dict(L=1, D=8, H=512, P=256, K=32000, T=21, B=16), "bf16", 70)
    _compare(dict(L=1, D=8, H=128, P=64, K=1000, T=7, B=8), "bf16", 75)
    _compare(dict(L=1, D=8, H=64, P=32, K=100, T=5, B=4), "fp32", 78)


def test_static_head_rejects_dims_above_its_array(gpu_lib):
    from paper_1907_05701_amd import binding as bd
    dims = bd.make_dims(1, 8, 512, 256, 32000, 21, 128, "bf16")
    assert bd.blstm_workspace_bytes(dims)["head_ws"] > bd.HEAD_STATIC_SCRATCH_BYTES
    dev = torch.device("cuda:0")
    one = torch.zeros(8, dtype=torch.float32, device=dev)
    with pytest.raises(bd.BlstmError) as ei:
        bd.softmax_ce_fwd_bwd_static(dims, one, one, one, one.view(torch.int32), 1.0, one, one, one)
    assert ei.value.code == bd.BLSTM_EUNSUPPORTED
