"""Host-side checks of the C ABI that need no GPU: the library loads, it
exports every function the public header declares, and its host logic
(parameter count, workspace sizes, argument validation) is right.  No
kernel is launched here."""

import ctypes
import os
import re

import pytest

from oracle import blstm_ref as ref

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "adpsgd_blstm.h")


def _lib():
    from paper_1907_05701_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        pytest.fail("libadpsgd_blstm.so is not built; run __graft_entry__.build()")
    return binding


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\**\s*([a-z_][a-z0-9_]*)\s*\(",
                       text, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_five_calls():
    names = _declared_functions()
    for fn in ("blstm_fwd", "blstm_bwd", "softmax_ce_fwd_bwd", "replica_grad_reduce", "adpsgd_step"):
        assert fn in names


def test_library_exports_every_declared_symbol():
    bd = _lib()
    cdll = ctypes.CDLL(bd.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(cdll, name), name
    assert set(bd.EXPORTED) == set(_declared_functions())


@pytest.mark.parametrize("shape", [
    dict(L=1, D=40, H=64, P=32, K=100, T=21, B=8),
    dict(L=6, D=260, H=512, P=256, K=32000, T=21, B=128),
    dict(L=2, D=12, H=32, P=8, K=7, T=3, B=5),
])
def test_param_count_agrees_with_oracle(shape):
    bd = _lib()
    for prec in ("fp32", "bf16"):
        dims = bd.make_dims(**shape, precision=prec)
        assert bd.blstm_param_count(dims) == ref.param_count(ref.Dims(**shape))


def test_workspace_sizes_scale_with_batch():
    bd = _lib()
    a = bd.blstm_workspace_bytes(bd.make_dims(6, 260, 512, 256, 32000, 21, 128, "bf16"))
    b = bd.blstm_workspace_bytes(bd.make_dims(6, 260, 512, 256, 32000, 21, 256, "bf16"))
    assert a["theta_lp"] == 2 * 43_154_944
    assert a["y_top"] == 21 * 128 * 1024 * 2
    # the activations kept for backpropagation grow with the frame count:
    # per frame and layer the gates (8H bf16) and cell states (2H fp32), and
    # the outputs (2H bf16) of every layer but the top one
    H, L, extra_frames = 512, 6, 21 * 128
    assert b["act_ws"] - a["act_ws"] >= extra_frames * (L * (8 * H * 2 + 2 * H * 4) + (L - 1) * 2 * H * 2)
    assert b["head_ws"] > a["head_ws"]
    f = bd.blstm_workspace_bytes(bd.make_dims(1, 40, 64, 32, 100, 21, 8, "fp32"))
    assert f["theta_lp"] == 0 and f["y_top"] == 21 * 8 * 128 * 4


@pytest.mark.parametrize("bad,code", [
    (dict(L=0), -1), (dict(B=0), -1), (dict(precision=7), -1),
    (dict(H=40), -2), (dict(P=12), -2), (dict(D=6), -2), (dict(L=17), -2),
])
def test_invalid_dims_are_rejected_with_a_message(bad, code):
    bd = _lib()
    shape = dict(L=2, D=40, H=64, P=32, K=100, T=4, B=8, precision=bd.BLSTM_BF16)
    shape.update(bad)
    dims = bd.Dims(*[shape[k] for k in ("L", "D", "H", "P", "K", "T", "B", "precision")])
    with pytest.raises(bd.BlstmError) as ei:
        bd.blstm_param_count(dims)
    assert ei.value.code == code
    assert len(str(ei.value)) > 20


def test_null_pointers_are_rejected_before_any_launch():
    bd = _lib()
    L = bd.lib()
    dims = bd.make_dims(1, 40, 64, 32, 100, 21, 8, "fp32")
    assert L.blstm_fwd(ctypes.byref(dims), None, None, None, None, None, None) == bd.BLSTM_EINVAL
    assert b"NULL" in L.blstm_last_error()
    assert L.blstm_bwd(ctypes.byref(dims), None, None, None, None, None, None, None) == bd.BLSTM_EINVAL
    assert L.softmax_ce_fwd_bwd(ctypes.byref(dims), None, None, None, None, ctypes.c_float(1.0),
                                None, None, None, None, None) == bd.BLSTM_EINVAL
    assert L.adpsgd_step(None, None, None, 1, ctypes.c_float(1.0), 10, ctypes.c_float(0.1), 0,
                         None, None) == bd.BLSTM_EINVAL
    assert L.replica_grad_reduce(None, 1, 10, ctypes.c_float(1.0), None, None) == bd.BLSTM_EINVAL
    arr = (ctypes.c_void_p * 1)(None)
    assert L.replica_grad_reduce(ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p)), 17, 10,
                                 ctypes.c_float(1.0), ctypes.c_void_p(16), None) == bd.BLSTM_EUNSUPPORTED
    assert L.adpsgd_step(ctypes.c_void_p(16), ctypes.c_void_p(32), ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p)),
                         1, ctypes.c_float(1.0), 10, ctypes.c_float(0.1), 8, None, None) == bd.BLSTM_EINVAL
