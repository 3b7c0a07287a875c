"""GPU parity: the HIP library (through its C ABI) against the CPU oracle on
the same seeded inputs.

Tolerances: float32 path <= 1e-4 and bf16-MFMA path <= 2e-2, as norm-wise
relative errors ||gpu - ref|| / ||ref|| per parameter block, for y_top and
dy_top, and |dL|/|L| for the loss; the oracle runs in float64 on the
unrounded float32 inputs.  Row by row as well (each row of a parameter
matrix, 16-element pieces of a vector, each frame of y_top and dy_top):
relative row errors <= 1e-4 (float32) and <= 0.2 (bf16), where a single
wrong row scores about 1 (tests/parity_measures.py).  The update kernels follow the oracle's float32
operation order exactly and are compared bit for bit; the bf16 operand copy
is compared bit for bit with round-to-nearest-even."""

import os
import sys

import numpy as np
import pytest
import torch

from oracle import blstm_ref as ref
from paper_1907_05701_amd import inputs

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from parity_measures import block_row_errors, row_errors  # noqa: E402

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-4
BF16_TOL = 2e-2
# bound on the largest relative row error of a block (see row_errors in
# parity_measures.py): a single wrong row scores about 1
# (measured: at most 3.4e-6 on the float32 path and 7e-2 on the bf16 path)
ROW_TOL = {"fp32": 1e-4, "bf16": 0.2}


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def block_errors(g_gpu, g_ref, dims):
    blocks, _ = ref.param_layout(dims)
    out = {}
    for key, (off, shape) in blocks.items():
        sl = slice(off, off + int(np.prod(shape)))
        out[key] = rel(g_gpu[sl], g_ref[sl])
    return out


def check_rows(errs, precision):
    worst = max(errs.items(), key=lambda kv: kv[1])
    say(f"[parity] worst row error {worst[0]}={worst[1]:.3e} (bound {ROW_TOL[precision]:.0e})")
    bad = {k: v for k, v in errs.items() if not v <= ROW_TOL[precision]}
    assert not bad, bad


def run_step_and_compare(shape, precision, tol, dist="uniform", seed=0, check_update=True, edit_theta=None,
                         check=None, row_check=True):
    from paper_1907_05701_amd.step import LearnerStep
    say(f"[parity] shape={shape} precision={precision} seed={seed}")
    dims = ref.Dims(**shape)
    n = ref.param_count(dims)
    theta = inputs.params(n, seed=seed)
    if edit_theta is not None:
        theta = edit_theta(theta.copy(), dims)
    x = inputs.features(dims.T, dims.B, dims.D, seed=seed + 1)
    lab = inputs.labels(dims.T, dims.B, dims.K, seed=seed + 2, dist=dist)
    peer = inputs.peer(theta, seed=seed + 3)
    st = LearnerStep(**shape, precision=precision)
    assert st.n == n
    st.load(theta, x, lab, peer)
    st.gradient()
    torch.cuda.synchronize()
    st.check_recurrence()
    want = ref.learner_gradient(theta, dims, x, lab)
    loss = float(st.loss.cpu()[0])
    errs = {"loss": abs(loss - want["loss"]) / abs(want["loss"]),
            "y_top": rel(st.y_top.float().cpu().numpy(), want["y_top"]),
            "dy_top": rel(st.dy_top.cpu().numpy(), want["dy_top"])}
    grad = st.grad.cpu().numpy()
    errs.update({str(k): v for k, v in block_errors(grad, want["grad"], dims).items()})
    errs["grad"] = rel(grad, want["grad"])
    if check is not None:
        check(st)
    worst = max(errs.items(), key=lambda kv: kv[1])
    say(f"[parity] loss gpu={loss:.7f} ref={want['loss']:.7f}; worst {worst[0]}={worst[1]:.3e}")
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, bad
    if row_check:
        T, B = dims.T, dims.B
        rows = block_row_errors(grad, want["grad"], dims, param_layout=ref.param_layout)
        rows = {str(k): v for k, v in rows.items()}
        rows["y_top"] = row_errors(st.y_top.float().cpu().numpy(), want["y_top"], T * B)
        rows["dy_top"] = row_errors(st.dy_top.cpu().numpy(), want["dy_top"], T * B)
        check_rows(rows, precision)
    if check_update:
        lr = 0.1
        st.update(lr)
        torch.cuda.synchronize()
        new_ref = ref.adpsgd_update(theta, peer, want["grad"], lr)
        e = rel(st.theta.cpu().numpy(), new_ref)
        say(f"[parity] updated theta rel err {e:.3e}")
        assert e <= tol
        if st.theta_lp is not None:
            lp = st.theta_lp.view(torch.int16).cpu().numpy().view(np.uint16)
            np.testing.assert_array_equal(lp, ref.bf16_round(st.theta.cpu().numpy()))
    return errs


def test_tiny_step_fp32(gpu_lib):
    run_step_and_compare(dict(L=1, D=40, H=64, P=32, K=100, T=21, B=8), "fp32", FP32_TOL)


def test_two_layer_fp32_ragged(gpu_lib):
    run_step_and_compare(dict(L=2, D=44, H=48, P=24, K=37, T=5, B=19), "fp32", FP32_TOL, seed=5)


def test_tiny_shape_bf16(gpu_lib):
    run_step_and_compare(dict(L=1, D=40, H=64, P=32, K=100, T=21, B=8), "bf16", BF16_TOL)


def test_ragged_bf16(gpu_lib):
    run_step_and_compare(dict(L=2, D=44, H=96, P=24, K=133, T=5, B=19), "bf16", BF16_TOL, seed=7)


@pytest.mark.parametrize("prec,tol", [("fp32", FP32_TOL), ("bf16", BF16_TOL)])
def test_single_frame_and_single_sequence(gpu_lib, prec, tol):
    run_step_and_compare(dict(L=2, D=8, H=32, P=8, K=10, T=1, B=1), prec, tol, seed=3)
    run_step_and_compare(dict(L=1, D=8, H=32, P=8, K=10, T=3, B=1), prec, tol, seed=4)


def test_full_model_dims_bf16_b16(gpu_lib):
    run_step_and_compare(dict(L=6, D=260, H=512, P=256, K=32000, T=21, B=16), "bf16", BF16_TOL,
                         dist="zipf")


def test_full_model_bf16_b128(gpu_lib):
    """The full workload the benchmark times (6 x 2 x 512, T=21, B=128)."""
    run_step_and_compare(dict(L=6, D=260, H=512, P=256, K=32000, T=21, B=128), "bf16", BF16_TOL,
                         dist="zipf", check_update=False)


def test_full_model_dims_fp32_b8(gpu_lib):
    run_step_and_compare(dict(L=6, D=260, H=512, P=256, K=32000, T=21, B=8), "fp32", FP32_TOL,
                         dist="zipf", check_update=False)


def run_replicated_and_compare(shape, reps, tol, seed=11):
    """The step at a large batch built from `reps` copies of a small seeded
    batch of shape["B"] sequences.  Sequences are independent in the model
    and the loss is a mean over frames, so the loss and the gradient equal
    those of the small batch and every copy's y_top equals the small batch's:
    the oracle runs on the small batch only, while the GPU runs the full
    batch in the launch configuration of the large workload."""
    from paper_1907_05701_amd.step import LearnerStep
    dims = ref.Dims(**shape)
    B0, T = dims.B, dims.T
    big = dict(shape, B=B0 * reps)
    say(f"[parity] replicated batch {B0} x {reps}: shape={big}")
    n = ref.param_count(dims)
    theta = inputs.params(n, seed=seed)
    x = inputs.features(T, B0, dims.D, seed=seed + 1)
    lab = inputs.labels(T, B0, dims.K, seed=seed + 2, dist="zipf")
    xb = np.ascontiguousarray(np.tile(x, (1, reps, 1)))
    lb = np.ascontiguousarray(np.tile(lab, (1, reps)))
    st = LearnerStep(**big, precision="bf16")
    st.load(theta, xb, lb, inputs.peer(theta, seed=seed + 3))
    st.gradient()
    torch.cuda.synchronize()
    st.check_recurrence()
    want = ref.learner_gradient(theta, dims, x, lab)
    loss = float(st.loss.cpu()[0])
    y = st.y_top.float().cpu().numpy().reshape(T, reps, B0, -1)
    errs = {"loss": abs(loss - want["loss"]) / abs(want["loss"])}
    for c in sorted({0, reps // 2, reps - 1}):
        errs[f"y_top copy {c}"] = rel(y[:, c], want["y_top"])
    grad = st.grad.cpu().numpy()
    errs.update({str(k): v for k, v in block_errors(grad, want["grad"], dims).items()})
    worst = max(errs.items(), key=lambda kv: kv[1])
    say(f"[parity] loss gpu={loss:.7f} ref={want['loss']:.7f}; worst {worst[0]}={worst[1]:.3e}")
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, bad
    rows = block_row_errors(grad, want["grad"], dims, param_layout=ref.param_layout)
    rows = {str(k): v for k, v in rows.items()}
    for c in range(reps):   # every copy, frame by frame
        rows[f"y_top copy {c}"] = row_errors(y[:, c], want["y_top"], T * B0)
    check_rows(rows, "bf16")


def test_full_model_b512_replicated(gpu_lib):
    """The large-batch workload (B = 512, T = 21) as 32 copies of 16 sequences."""
    run_replicated_and_compare(dict(L=6, D=260, H=512, P=256, K=32000, T=21, B=16), 32, BF16_TOL)


def test_stress_t64_b1024_replicated(gpu_lib):
    """The stress workload (T = 64, B = 1024) as 64 copies of 16 sequences."""
    run_replicated_and_compare(dict(L=6, D=260, H=512, P=256, K=32000, T=64, B=16), 64, BF16_TOL, seed=21)


def _bf16_model():
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import bf16_path_model
    return bf16_path_model


def _blockwise(g, want, blocks):
    return {str(k): rel(g[o:o + int(np.prod(s))], want[o:o + int(np.prod(s))]) for k, (o, s) in blocks.items()}


def test_saturated_cells_bf16(gpu_lib):
    """Cells driven into saturation so that most outputs h are +-1.0 in bf16
    (gate biases i, f: +6, g: +2, o: +7: the cells charge by about one per
    step and o tanh c rounds to 1): the recurrent exchange packs h with a tag
    in bit 14 of each bf16, which is free for |h| <= 1.

    At this point the gradient is badly conditioned: the exact gradient at
    the bf16 copy of the weights is several per cent from the one at theta
    (pinned on the CPU in test_bf16_model.py), so no path with bf16 operands
    meets the 2e-2 bar here.  Every block is compared instead with the bound
    that the bf16 rounding points themselves give: a float64 model of the
    path's rounding points (tests/bf16_path_model.py) is E from the oracle
    per block; the GPU must be within max(2e-2, 1.25 E) of the oracle in
    every block, and closer to that model than the model is to the oracle
    (so what remains is the rounding the model names, not a defect)."""
    bm = _bf16_model()
    shape = dict(L=2, D=40, H=512, P=32, K=100, T=21, B=16)
    dims = ref.Dims(**shape)
    H = dims.H

    def edit(theta, dims):
        blocks, _ = ref.param_layout(dims)
        for key, (off, shp) in blocks.items():
            if key[0] == "b_ih":   # gates i, f, g, o
                b = theta[off:off + int(np.prod(shp))]
                b[0:2 * H] = 6.0
                b[2 * H:3 * H] = 2.0
                b[3 * H:4 * H] = 7.0
        return theta

    got = {}

    def keep(st):
        frac = float((st.y_top.float().abs() == 1.0).float().mean())
        say(f"[parity] fraction of top-layer h equal to +-1: {frac:.3f}")
        assert frac > 0.3
        got["grad"] = st.grad.cpu().numpy()
        got["loss"] = float(st.loss.cpu()[0])

    errs = run_step_and_compare(shape, "bf16", 1e9, seed=31, edit_theta=edit, check=keep, check_update=False,
                                row_check=False)
    theta = edit(inputs.params(ref.param_count(dims), seed=31).copy(), dims)
    x = inputs.features(dims.T, dims.B, dims.D, seed=32)
    lab = inputs.labels(dims.T, dims.B, dims.K, seed=33)
    want = ref.learner_gradient(theta, dims, x, lab)
    model = bm.learner_gradient(theta, shape, x, lab)
    blocks, _ = ref.param_layout(dims)
    e_model = _blockwise(model["grad"], want["grad"], blocks)
    e_gpu_model = _blockwise(got["grad"], model["grad"], blocks)
    bad = {}
    for k, e in e_model.items():
        bound = max(BF16_TOL, 1.25 * e)
        say(f"[parity] {k}: gpu {errs[k]:.2e} model {e:.2e} gpu-model {e_gpu_model[k]:.2e} bound {bound:.2e}")
        if not (errs[k] <= bound and (e_gpu_model[k] <= BF16_TOL or e_gpu_model[k] < e)):
            bad[k] = (errs[k], e, e_gpu_model[k])
    assert not bad, bad
    assert errs["loss"] <= BF16_TOL and errs["y_top"] <= BF16_TOL, errs
    # row by row against the model, which carries the rounding the oracle
    # does not (against the oracle a row can be as far off as its block)
    rows = {str(k): v for k, v in block_row_errors(got["grad"], model["grad"], dims,
                                                    param_layout=ref.param_layout).items()}
    check_rows(rows, "bf16")


def _peaked_head(gamma, seed=60):
    """Head-alone inputs at the paper's head size whose softmax is peaked as
    in a trained model: W_s scaled by gamma, each frame labelled with the
    class of its largest exact logit (the loss is then far below ln K)."""
    shape = dict(L=1, D=8, H=512, P=256, K=32000, T=21, B=16)
    dims = ref.Dims(**shape)
    n = ref.param_count(dims)
    blocks, _ = ref.param_layout(dims)
    theta = inputs.params(n, seed=seed).copy()
    off, shp = blocks["W_s"]
    theta[off:off + int(np.prod(shp))] *= np.float32(gamma)
    y = inputs.hidden_states(dims.T, dims.B, 2 * dims.H, seed=seed + 1)
    p = ref.unflatten(theta, dims)
    logits = (y.reshape(-1, 2 * dims.H).astype(np.float64) @ p["W_l"].T + p["b_l"]) @ p["W_s"].T + p["b_s"]
    lab = logits.argmax(axis=1).reshape(dims.T, dims.B).astype(np.int32)
    return shape, dims, theta, y, lab


def _head_on_gpu(shape, theta, y, lab):
    from paper_1907_05701_amd.step import LearnerStep
    dims = ref.Dims(**shape)
    st = LearnerStep(**shape, precision="bf16")
    st.load(theta, np.zeros((dims.T, dims.B, dims.D), np.float32), lab)
    st.y_top.copy_(torch.from_numpy(y).to(st.act_dtype))
    st.head()
    torch.cuda.synchronize()
    blocks, _ = ref.param_layout(dims)
    g = st.grad.cpu().numpy()
    out = {k: g[blocks[k][0]:blocks[k][0] + int(np.prod(blocks[k][1]))].reshape(blocks[k][1])
           for k in ("W_l", "b_l", "W_s", "b_s")}
    return float(st.loss.cpu()[0]), out, st.dy_top.cpu().numpy()


def test_peaked_softmax_head_bf16(gpu_lib):
    """The bf16 head where the model is confident (W_s scaled by 8, labels at
    each frame's largest logit: loss about 0.64 against ln K = 10.4): the
    logits are kept in float32, so the loss and every head gradient meet the
    2e-2 bar (with bf16 logits the float64 model of the path gives 3.3e-2)."""
    shape, dims, theta, y, lab = _peaked_head(8.0)
    loss_ref, _, dy_ref, g_ref = ref.head_forward_backward(theta, dims, y, lab)
    assert loss_ref < 0.1 * np.log(dims.K)
    loss, g, dy = _head_on_gpu(shape, theta, y, lab)
    errs = {"loss": abs(loss - loss_ref) / loss_ref, "dy_top": rel(dy, dy_ref)}
    errs.update({k: rel(g[k], g_ref[k]) for k in g})
    say(f"[peaked] loss gpu={loss:.6f} ref={loss_ref:.6f}; " + " ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    bad = {k: v for k, v in errs.items() if not v <= BF16_TOL}
    assert not bad, bad


def test_very_peaked_softmax_head_bf16(gpu_lib):
    """W_s scaled by 16 (loss about 0.28, logits up to about 80): here the
    bf16 operands themselves (weights, z, y) move the head gradients by
    about 3.7e-2 in the float64 model of the path, so each block is held to
    max(2e-2, 1.25 x that model's error), and the GPU must be closer to the
    model than the model is to the oracle."""
    bm = _bf16_model()
    shape, dims, theta, y, lab = _peaked_head(16.0)
    loss_ref, _, dy_ref, g_ref = ref.head_forward_backward(theta, dims, y, lab)
    loss_m, g_m, dy_m = bm.head_gradient(theta, shape, y, lab)
    loss, g, dy = _head_on_gpu(shape, theta, y, lab)
    pairs = {"loss": ((loss, loss_m), loss_ref), "dy_top": ((dy, dy_m), dy_ref)}
    pairs.update({k: ((g[k], g_m[k]), g_ref[k]) for k in g})
    bad = {}
    for k, ((gpu, mod), exact) in pairs.items():
        if k == "loss":
            e_gpu, e_mod, e_gm = abs(gpu - exact) / exact, abs(mod - exact) / exact, abs(gpu - mod) / abs(mod)
        else:
            e_gpu, e_mod, e_gm = rel(gpu, exact), rel(mod, exact), rel(gpu, mod)
        bound = max(BF16_TOL, 1.25 * e_mod)
        say(f"[very peaked] {k}: gpu {e_gpu:.2e} model {e_mod:.2e} gpu-model {e_gm:.2e} bound {bound:.2e}")
        if not (e_gpu <= bound and (e_gm <= BF16_TOL or e_gm < e_mod)):
            bad[k] = (e_gpu, e_mod, e_gm)
    assert not bad, bad


def test_long_sequence_bf16(gpu_lib):
    """T = 300 on the persistent kernels: the exchange tag carries only bit 1
    of the step number, so the sequence length is not bounded by it."""
    run_step_and_compare(dict(L=2, D=24, H=64, P=16, K=30, T=300, B=8), "bf16", BF16_TOL, seed=41,
                         check_update=False)


def test_non_finite_gradients_keep_the_exchange_going(gpu_lib):
    """dy_top with a NaN row, a row of +-1e30 and a row of +-inf: the BPTT's
    exchanged partial sums saturate instead of carrying a non-finite value
    into the tag bits, so no member waits in vain (the recurrence status
    stays clear) and the non-finite rows reach the gradient as non-finite
    values while the exchange of every other row goes on."""
    from paper_1907_05701_amd.step import LearnerStep
    shape = dict(L=2, D=24, H=128, P=16, K=30, T=5, B=8)
    say(f"[non-finite] shape={shape}")
    dims = ref.Dims(**shape)
    theta = inputs.params(ref.param_count(dims), seed=5)
    st = LearnerStep(**shape, precision="bf16")
    st.load(theta, inputs.features(5, 8, 24, seed=6), inputs.labels(5, 8, 30, seed=7))
    st.forward()
    st.check_recurrence()
    dy = torch.from_numpy(np.random.default_rng(8).standard_normal((5, 8, 256)).astype(np.float32))
    dy[:, 0, :] = float("nan")
    dy[:, 1, ::2], dy[:, 1, 1::2] = 1e30, -1e30
    dy[:, 2, ::2], dy[:, 2, 1::2] = float("inf"), float("-inf")
    st.backward(dy_top=dy.to(st.device))
    torch.cuda.synchronize()
    st.check_recurrence()
    assert not torch.isfinite(st.grad).all().item()


@pytest.mark.parametrize("H", [192, 320, 448], ids=["3_members", "5_members", "7_members"])
def test_recurrence_member_counts_bf16(gpu_lib, H):
    """Groups of 3, 5 and 7 members (H = 64 x members): the BPTT's gathering
    threads split the members into two parts of unequal size, and the
    forward's gathered words per row (H / 4) are not a power of two."""
    from paper_1907_05701_amd import binding as bd
    bd.blstm_timing_begin("lstm_rec")
    run_step_and_compare(dict(L=2, D=40, H=H, P=32, K=50, T=5, B=24), "bf16", BF16_TOL, seed=13,
                         check_update=False)
    got = bd.blstm_timing_end()
    if os.environ.get("ADPSGD_BLSTM_NO_PERSIST") != "1":   # the persistent kernels ran, one launch per layer
        assert got["lstm_rec_fwd_persist"][0] == 2 and got["lstm_rec_bwd_persist"][0] == 2, got


@pytest.mark.parametrize("B", [200, 300, 1100], ids=["ragged_slices", "two_chunks", "five_chunks"])
def test_recurrence_batch_regimes_bf16(gpu_lib, B):
    """Batches whose last 16-row slice is ragged (B=200: 13 slices), that
    need two launches per layer (B=300: 256 + 44 rows) and five (B=1100).
    Two layers, so that exchange words left by the previous layer's
    launches (forward bottom-up, backward top-down) are met and must not
    match."""
    run_step_and_compare(dict(L=2, D=40, H=512, P=32, K=50, T=3, B=B), "bf16", BF16_TOL, seed=11,
                         check_update=False)


def test_cooperative_and_plain_persistent_launches_agree(gpu_lib, monkeypatch):
    """The persistent kernels as plain launches (default when the grid fits)
    and as cooperative launches give bit-identical results; both report
    that every exchange wait completed."""
    from paper_1907_05701_amd.step import LearnerStep
    shape = dict(L=2, D=260, H=512, P=256, K=1000, T=21, B=128)
    dims = ref.Dims(**shape)
    theta = inputs.params(ref.param_count(dims), seed=31)
    x = inputs.features(dims.T, dims.B, dims.D, seed=32)
    lab = inputs.labels(dims.T, dims.B, dims.K, seed=33, dist="zipf")
    grads = []
    for coop in ("0", "1"):
        monkeypatch.setenv("ADPSGD_BLSTM_COOPERATIVE", coop)
        say(f"[launch] cooperative={coop}")
        st = LearnerStep(**shape, precision="bf16")
        st.load(theta, x, lab, inputs.peer(theta))
        st.gradient()
        torch.cuda.synchronize()
        st.check_recurrence()
        grads.append(st.grad.cpu().numpy())
    np.testing.assert_array_equal(grads[0].view(np.uint32), grads[1].view(np.uint32))


def test_per_step_recurrence_path_bf16(gpu_lib, monkeypatch):
    """The per-step recurrent kernels (used when the persistent ones do not
    apply) on the full layer widths."""
    monkeypatch.setenv("ADPSGD_BLSTM_NO_PERSIST", "1")
    run_step_and_compare(dict(L=2, D=260, H=512, P=256, K=1000, T=6, B=24), "bf16", BF16_TOL, seed=12,
                         check_update=False)


# ------------------------------------------------------------ the update ---

@pytest.mark.parametrize("flags", [0, 1, 2, 3])
def test_update_bitwise_full_vector_r8(gpu_lib, flags):
    """The update-only workload: 43,154,944 parameters, 8 resident replica
    gradients N(0, 1e-3^2), lr 0.05, seeded peer; bit-exact."""
    from paper_1907_05701_amd import binding as bd
    n, R, lr = 43_154_944, 8, 0.05
    say(f"[update] n={n} R={R} flags={flags}")
    theta = inputs.params(n)
    peer = inputs.peer(theta)
    grads = inputs.replica_grads(n, R)
    dev = torch.device("cuda:0")
    th = torch.from_numpy(theta).to(dev)
    pe = torch.from_numpy(peer).to(dev)
    gs = [torch.from_numpy(g).to(dev) for g in grads]
    lp = torch.empty(n, dtype=torch.bfloat16, device=dev)
    bd.adpsgd_step(th, pe, gs, 1.0 / R, lr, flags, lp)
    torch.cuda.synchronize()
    order = "eq7" if flags & 1 else "sgd_then_avg"
    want = ref.adpsgd_update_fp32(theta, peer, grads, 1.0 / R, lr, order)
    got = th.cpu().numpy()
    np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32))
    np.testing.assert_array_equal(lp.view(torch.int16).cpu().numpy().view(np.uint16), ref.bf16_round(want))
    if flags & 2:
        np.testing.assert_array_equal(pe.cpu().numpy().view(np.uint32), want.view(np.uint32))
    else:
        np.testing.assert_array_equal(pe.cpu().numpy(), peer)


@pytest.mark.parametrize("n", [1, 3, 4, 1001, 1 << 20])
def test_update_and_reduce_bitwise_odd_sizes(gpu_lib, n):
    from paper_1907_05701_amd import binding as bd
    R = 3
    theta = inputs.params(n, seed=40)
    peer = inputs.peer(theta, seed=41)
    grads = inputs.replica_grads(n, R, seed0=42)
    dev = torch.device("cuda:0")
    gs = [torch.from_numpy(g).to(dev) for g in grads]
    out = torch.empty(n, dtype=torch.float32, device=dev)
    bd.replica_grad_reduce(gs, 0.25, out)
    th = torch.from_numpy(theta).to(dev)
    pe = torch.from_numpy(peer).to(dev)
    bd.adpsgd_step(th, pe, gs, 0.25, 0.05, 0, None)
    # misaligned views take the scalar path
    big = torch.from_numpy(np.concatenate([[0.0], theta]).astype(np.float32)).to(dev)
    thm = big[1:]
    bd.adpsgd_step(thm, pe.clone(), gs, 0.25, 0.05, 0, None)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out.cpu().numpy().view(np.uint32),
                                  ref.replica_grad_reduce_fp32(grads, 0.25).view(np.uint32))
    want = ref.adpsgd_update_fp32(theta, peer, grads, 0.25, 0.05)
    np.testing.assert_array_equal(th.cpu().numpy().view(np.uint32), want.view(np.uint32))
    np.testing.assert_array_equal(thm.cpu().numpy().view(np.uint32), want.view(np.uint32))


def test_reduce_in_place_into_first_buffer(gpu_lib):
    from paper_1907_05701_amd import binding as bd
    n, R = 100_003, 8
    grads = inputs.replica_grads(n, R)
    dev = torch.device("cuda:0")
    gs = [torch.from_numpy(g).to(dev) for g in grads]
    bd.replica_grad_reduce(gs, 1.0 / R, gs[0])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gs[0].cpu().numpy().view(np.uint32),
                                  ref.replica_grad_reduce_fp32(grads, 1.0 / R).view(np.uint32))


def test_pack_is_round_to_nearest_even(gpu_lib):
    from paper_1907_05701_amd import binding as bd
    dims = bd.make_dims(1, 40, 64, 32, 100, 21, 8, "bf16")
    n = bd.blstm_param_count(dims)
    rng = np.random.default_rng(0)
    theta = (rng.standard_normal(n) * 3.0).astype(np.float32)
    theta[:6] = [0.0, -0.0, 1.00390625, 1.01171875, 3.4e38, -1e-40]
    th = torch.from_numpy(theta).cuda()
    lp = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    bd.blstm_pack_params(dims, th, lp)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(lp.view(torch.int16).cpu().numpy().view(np.uint16), ref.bf16_round(theta))


# ---------------------------------------------- entry points on their own ---

@pytest.mark.parametrize("prec,tol", [("fp32", FP32_TOL), ("bf16", BF16_TOL)])
def test_head_alone_on_given_hidden_states(gpu_lib, prec, tol):
    from paper_1907_05701_amd.step import LearnerStep
    shape = dict(L=1, D=8, H=64, P=64, K=1000, T=7, B=24)
    dims = ref.Dims(**shape)
    n = ref.param_count(dims)
    theta = inputs.params(n, seed=50)
    y = inputs.hidden_states(dims.T, dims.B, 2 * dims.H, seed=51)
    lab = inputs.labels(dims.T, dims.B, dims.K, seed=52, dist="zipf")
    st = LearnerStep(**shape, precision=prec)
    st.load(theta, np.zeros((dims.T, dims.B, dims.D), np.float32), lab)
    st.y_top.copy_(torch.from_numpy(y).to(st.act_dtype))
    st.head()
    torch.cuda.synchronize()
    loss, _, dy, grads = ref.head_forward_backward(theta, dims, y, lab)
    assert abs(float(st.loss.cpu()[0]) - loss) / loss <= tol
    assert rel(st.dy_top.cpu().numpy(), dy) <= tol
    g = st.grad.cpu().numpy()
    blocks, _ = ref.param_layout(dims)
    for key in ("W_l", "b_l", "W_s", "b_s"):
        off, shp = blocks[key]
        assert rel(g[off:off + int(np.prod(shp))], grads[key].reshape(-1)) <= tol, key


@pytest.mark.parametrize("sign", [1.0, -1.0], ids=["scale_pos", "scale_neg"])
@pytest.mark.parametrize("shape", [
    dict(L=1, D=8, H=64, P=64, K=1000, T=7, B=24),   # 8 class blocks, the last one partial; 3 frame chunks, ragged
    dict(L=1, D=8, H=32, P=24, K=50, T=1, B=5),      # one partial class block, one partial frame chunk
], ids=["blocks", "one_block"])
@pytest.mark.parametrize("blk", ["1", "0"], ids=["class_block", "tiled"])
def test_logits_forms_on_given_hidden_states(gpu_lib, monkeypatch, blk, shape, sign):
    """Both forms of the two logits products (the class-block kernels, and
    the tiled products with the statistics and softmax epilogues) give the
    head's loss and gradients.  A negative loss scale takes the form that
    multiplies by the scale after the exponential (log2 of the scale cannot
    be folded into the exponent); loss and gradients change sign."""
    from paper_1907_05701_amd.step import LearnerStep
    monkeypatch.setenv("ADPSGD_LOGITS_BLOCK", blk)
    dims = ref.Dims(**shape)
    n = ref.param_count(dims)
    theta = inputs.params(n, seed=60)
    y = inputs.hidden_states(dims.T, dims.B, 2 * dims.H, seed=61)
    lab = inputs.labels(dims.T, dims.B, dims.K, seed=62, dist="zipf")
    st = LearnerStep(**shape, precision="bf16")
    st.load(theta, np.zeros((dims.T, dims.B, dims.D), np.float32), lab)
    st.loss_scale = sign / (dims.T * dims.B)
    st.y_top.copy_(torch.from_numpy(y).to(st.act_dtype))
    st.head()
    torch.cuda.synchronize()
    loss, _, dy, grads = ref.head_forward_backward(theta, dims, y, lab)
    assert abs(float(st.loss.cpu()[0]) - sign * loss) / loss <= BF16_TOL
    assert rel(st.dy_top.cpu().numpy(), sign * dy) <= BF16_TOL
    g = st.grad.cpu().numpy()
    blocks, _ = ref.param_layout(dims)
    for key in ("W_l", "b_l", "W_s", "b_s"):
        off, shp = blocks[key]
        assert rel(g[off:off + int(np.prod(shp))], sign * grads[key].reshape(-1)) <= BF16_TOL, key


@pytest.mark.parametrize("blk", ["1", "0"], ids=["class_block", "tiled"])
def test_logits_forms_zero_loss_scale(gpu_lib, monkeypatch, blk):
    """A zero loss scale (no log2 of it to fold into the exponent) gives a
    zero loss and exactly zero head gradients and dy_top in both forms of
    the logits products; 128 frames, two whole 64-frame chunks."""
    from paper_1907_05701_amd.step import LearnerStep
    monkeypatch.setenv("ADPSGD_LOGITS_BLOCK", blk)
    shape = dict(L=1, D=8, H=64, P=64, K=1000, T=8, B=16)
    dims = ref.Dims(**shape)
    n = ref.param_count(dims)
    theta = inputs.params(n, seed=63)
    y = inputs.hidden_states(dims.T, dims.B, 2 * dims.H, seed=64)
    lab = inputs.labels(dims.T, dims.B, dims.K, seed=65, dist="zipf")
    st = LearnerStep(**shape, precision="bf16")
    st.load(theta, np.zeros((dims.T, dims.B, dims.D), np.float32), lab)
    st.loss_scale = 0.0
    st.y_top.copy_(torch.from_numpy(y).to(st.act_dtype))
    st.grad.fill_(1.0)
    st.head()
    torch.cuda.synchronize()
    assert float(st.loss.cpu()[0]) == 0.0
    assert not st.dy_top.abs().max().item()
    g = st.grad.cpu().numpy()
    blocks, _ = ref.param_layout(dims)
    for key in ("W_l", "b_l", "W_s", "b_s"):
        off, shp = blocks[key]
        assert not np.abs(g[off:off + int(np.prod(shp))]).max(), key


def test_deterministic_across_runs(gpu_lib):
    from paper_1907_05701_amd.step import LearnerStep
    shape = dict(L=2, D=260, H=128, P=64, K=3000, T=9, B=40)
    dims = ref.Dims(**shape)
    n = ref.param_count(dims)
    theta = inputs.params(n)
    x = inputs.features(dims.T, dims.B, dims.D)
    lab = inputs.labels(dims.T, dims.B, dims.K, dist="zipf")
    outs = []
    for _ in range(2):
        st = LearnerStep(**shape, precision="bf16")
        st.load(theta, x, lab, theta)
        st.gradient()
        torch.cuda.synchronize()
        outs.append((st.loss.cpu().numpy().copy(), st.grad.cpu().numpy().copy(),
                     st.y_top.float().cpu().numpy().copy()))
    for a, b in zip(outs[0], outs[1]):
        np.testing.assert_array_equal(a, b)


def test_timing_hooks_report_kernels(gpu_lib):
    from paper_1907_05701_amd import binding as bd
    from paper_1907_05701_amd.step import LearnerStep
    shape = dict(L=1, D=40, H=64, P=32, K=100, T=4, B=8)
    n = ref.param_count(ref.Dims(**shape))
    st = LearnerStep(**shape, precision="bf16")
    st.load(inputs.params(n), inputs.features(4, 8, 40), inputs.labels(4, 8, 100), inputs.params(n, seed=9))
    bd.blstm_timing_begin("lstm_rec")
    st.gradient()
    got = bd.blstm_timing_end()
    if os.environ.get("ADPSGD_BLSTM_NO_PERSIST") == "1":
        assert set(got) == {"lstm_rec_fwd", "lstm_rec_bwd"}
        assert got["lstm_rec_fwd"][0] == 4 and got["lstm_rec_bwd"][0] == 4
    else:
        assert set(got) == {"lstm_rec_fwd_persist", "lstm_rec_bwd_persist"}
        assert got["lstm_rec_fwd_persist"][0] == 1 and got["lstm_rec_bwd_persist"][0] == 1
    assert all(v[1] > 0 for v in got.values())


def test_graph_replays_match_eager_steps(gpu_lib, monkeypatch):
    """A captured learner step replayed several times, with eager work and
    synchronisation in between, gives bit-identical results to the same
    number of eagerly launched steps (both on the per-step recurrent kernels,
    which is what a captured step uses)."""
    from paper_1907_05701_amd.step import LearnerStep
    monkeypatch.setenv("ADPSGD_BLSTM_NO_PERSIST", "1")
    shape = dict(L=2, D=260, H=128, P=64, K=3000, T=7, B=40)
    dims = ref.Dims(**shape)
    n = ref.param_count(dims)
    theta = inputs.params(n)
    x = inputs.features(dims.T, dims.B, dims.D)
    lab = inputs.labels(dims.T, dims.B, dims.K, dist="zipf")
    peer = inputs.peer(theta)
    eager = LearnerStep(**shape, precision="bf16")
    eager.load(theta, x, lab, peer)
    replayed = LearnerStep(**shape, precision="bf16")
    replayed.load(theta, x, lab, peer)
    graph = replayed.capture(0.05)
    torch.cuda.synchronize()
    replayed.load(theta, x, lab, peer)          # capture ran nothing; start from the same state
    for i in range(3):
        eager.step(0.05)
        graph.replay()
        torch.cuda.synchronize()
        _ = (eager.theta * 2.0).sum().item()       # unrelated eager work between replays
        np.testing.assert_array_equal(replayed.theta.cpu().numpy(), eager.theta.cpu().numpy())
        np.testing.assert_array_equal(replayed.loss.cpu().numpy(), eager.loss.cpu().numpy())
        np.testing.assert_array_equal(replayed.grad.cpu().numpy(), eager.grad.cpu().numpy())
        say(f"[graph] replay {i} matches, loss {float(eager.loss.cpu()[0]):.6f}")


def test_graph_replays_with_persistent_forward(gpu_lib, monkeypatch):
    """Same as above with the persistent forward kernel recorded into the
    graph as a cooperative node (bit-identical to eager persistent steps)."""
    from paper_1907_05701_amd.step import LearnerStep
    monkeypatch.delenv("ADPSGD_BLSTM_NO_PERSIST", raising=False)
    monkeypatch.setenv("ADPSGD_BLSTM_RECURRENCE", "auto")
    monkeypatch.setenv("ADPSGD_BLSTM_GRAPH_PERSIST", "1")
    shape = dict(L=2, D=260, H=512, P=64, K=3000, T=7, B=40)
    dims = ref.Dims(**shape)
    n = ref.param_count(dims)
    theta = inputs.params(n)
    x = inputs.features(dims.T, dims.B, dims.D)
    lab = inputs.labels(dims.T, dims.B, dims.K, dist="zipf")
    peer = inputs.peer(theta)
    eager = LearnerStep(**shape, precision="bf16")
    eager.load(theta, x, lab, peer)
    replayed = LearnerStep(**shape, precision="bf16")
    replayed.load(theta, x, lab, peer)
    graph = replayed.capture(0.05)
    torch.cuda.synchronize()
    replayed.load(theta, x, lab, peer)
    for i in range(3):
        eager.step(0.05)
        graph.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(replayed.theta.cpu().numpy(), eager.theta.cpu().numpy())
        np.testing.assert_array_equal(replayed.y_top.float().cpu().numpy(), eager.y_top.float().cpu().numpy())
        say(f"[graph+persistent] replay {i} matches, loss {float(eager.loss.cpu()[0]):.6f}")


def test_recurrence_status_is_sticky_until_queried(gpu_lib):
    """The give-up flag (the int32 at act_ws_bytes - 256) set from the host
    survives the next forward and backward calls, so the query after them
    fails; the query clears it, and the next query succeeds."""
    from paper_1907_05701_amd import binding as bd
    from paper_1907_05701_amd.step import LearnerStep
    shape = dict(L=2, D=40, H=512, P=32, K=100, T=5, B=16)
    n = ref.param_count(ref.Dims(**shape))
    st = LearnerStep(**shape, precision="bf16")
    theta = inputs.params(n)
    st.load(theta, inputs.features(5, 16, 40), inputs.labels(5, 16, 100), theta)
    st.step(0.05)
    st.check_recurrence()
    flag = st.act_ws[st.act_ws.numel() - 256:st.act_ws.numel() - 252].view(torch.int32)
    flag.fill_(1)
    st.step(0.05)
    st.step(0.05)
    torch.cuda.synchronize()
    with pytest.raises(bd.BlstmError) as ei:
        st.check_recurrence()
    assert "gave up" in str(ei.value)
    assert int(flag.cpu()[0]) == 0
    st.check_recurrence()
    st.step(0.05)
    st.check_recurrence()


def test_graph_replays_at_benchmark_shape(gpu_lib):
    """The benchmark's configuration: the full model at B = 128 captured
    into one HIP graph (the persistent kernels recorded as plain launches)
    and replayed three times, with eager work and synchronisation between
    the replays; each replay must equal the same number of eager steps bit
    for bit, and the sticky recurrence flag must show no give-up over all
    replays."""
    from paper_1907_05701_amd.step import LearnerStep
    shape = dict(L=6, D=260, H=512, P=256, K=32000, T=21, B=128)
    dims = ref.Dims(**shape)
    n = ref.param_count(dims)
    theta = inputs.params(n)
    x = inputs.features(dims.T, dims.B, dims.D)
    lab = inputs.labels(dims.T, dims.B, dims.K, dist="zipf")
    peer = inputs.peer(theta)
    eager = LearnerStep(**shape, precision="bf16")
    eager.load(theta, x, lab, peer)
    replayed = LearnerStep(**shape, precision="bf16")
    replayed.load(theta, x, lab, peer)
    graph = replayed.capture(0.05, steps=2)
    torch.cuda.synchronize()
    replayed.load(theta, x, lab, peer)
    for i in range(3):
        eager.step(0.05)
        eager.step(0.05)
        graph.replay()
        torch.cuda.synchronize()
        _ = (eager.theta * 2.0).sum().item()
        for name in ("theta", "loss", "grad", "y_top"):
            a = getattr(replayed, name).float().cpu().numpy()
            b = getattr(eager, name).float().cpu().numpy()
            np.testing.assert_array_equal(a, b, err_msg=f"replay {i}: {name}")
        say(f"[graph bench shape] replay {i} matches, loss {float(eager.loss.cpu()[0]):.6f}")
    replayed.check_recurrence()
    eager.check_recurrence()


@pytest.mark.parametrize("shape", [
    dict(L=6, D=260, H=512, P=256, K=32000, T=21, B=128),   # the benchmark's step
    dict(L=2, D=260, H=256, P=64, K=3000, T=25, B=44),      # two row passes, a 4-row last slice
    dict(L=2, D=64, H=512, P=64, K=500, T=11, B=200),       # 16-row slices, unpadded layer-0 W_ih
], ids=["b128", "ragged", "rows16"])
def test_fused_products_match_the_separate_launches(gpu_lib, monkeypatch, shape):
    """The persistent forward computing each workgroup's slice of the input
    projection itself, and the persistent BPTT adding the split-K partial
    sums of dX itself (with every layer's bias sums in one reduction after
    the last BPTT), give the same step, bit for bit, as the separate product
    and reduction launches (same k order, summation order and rounding)."""
    from paper_1907_05701_amd.step import LearnerStep
    dims = ref.Dims(**shape)
    n = ref.param_count(dims)
    theta = inputs.params(n, seed=5)
    x = inputs.features(dims.T, dims.B, dims.D, seed=6)
    lab = inputs.labels(dims.T, dims.B, dims.K, seed=7, dist="zipf")
    out = {}
    for fuse in ("1", "0"):
        monkeypatch.setenv("ADPSGD_BLSTM_FUSE_GX", fuse)
        monkeypatch.setenv("ADPSGD_BLSTM_FUSE_DY", fuse)
        st = LearnerStep(**shape, precision="bf16")
        st.load(theta, x, lab, theta)
        st.gradient()
        torch.cuda.synchronize()
        st.check_recurrence()
        out[fuse] = {k: getattr(st, k).float().cpu().numpy() for k in ("y_top", "loss", "grad")}
        del st
    for k in ("y_top", "loss", "grad"):
        np.testing.assert_array_equal(out["1"][k], out["0"][k], err_msg=k)
    say(f"[fused] {shape} bit-identical, loss {float(out['1']['loss'][0]):.6f}")
