"""C-ABI checks that need no GPU: the library loads, exports every declared
symbol, and rejects host-visible argument errors before touching a device."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2606_09312_amd as wm
from paper_2606_09312_amd import binding as B
from oracle import wm_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    with open(os.path.join(ROOT, "include", "wm.h")) as f:
        src = f.read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(wm_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    lib = wm.load_library()
    names = _declared()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(names) == sorted(wm.SYMBOLS)


def _seg(a):
    a = np.asarray(a, dtype=np.int32)
    return a, a.ctypes.data_as(ctypes.c_void_p)


@pytest.mark.parametrize("seg_off,S,B,k,want", [
    ([0, 8], 1, 8, 9, B.WM_ERR_INVALID_ARGUMENT),        # k > segment
    ([0, 8], 1, 8, 0, B.WM_ERR_INVALID_ARGUMENT),        # k < 1
    ([0, 7], 1, 8, 2, B.WM_ERR_INVALID_ARGUMENT),        # does not end at B
    ([1, 8], 1, 8, 2, B.WM_ERR_INVALID_ARGUMENT),        # does not start at 0
    ([0, 5, 3, 8], 3, 8, 1, B.WM_ERR_INVALID_ARGUMENT),  # not monotone
    ([0, 4, 8], 2, 8, 5, B.WM_ERR_INVALID_ARGUMENT),     # k > smallest segment
])
def test_topk_host_validation_matches_oracle(seg_off, S, B, k, want):
    lib = wm.load_library()
    arr, p = _seg(seg_off)
    fake = ctypes.c_void_p(256)   # never dereferenced: validation fails first
    st = lib.wm_topk(fake, 1, B, p, S, k, fake, None, None)
    assert st == want
    assert lib.wm_last_error().decode() != ""
    assert O.validate({"n_kinds": 1}, B=B, T_max=0, seg_off=seg_off, k=k) == want


def test_model_create_rejects_before_device_work():
    lib = wm.load_library()
    h = ctypes.c_void_p()
    assert lib.wm_model_create(None, None, ctypes.byref(h)) == B.WM_ERR_INVALID_ARGUMENT
    # unsupported latent width, bad transition form, hidden width
    w = {k: np.zeros(4, np.float32) for k in ("type_emb", "param_w", "param_b", "w1", "b1", "w2",
                                                 "b2", "wc1", "bc1", "wc2")}
    wts = B.Weights()
    keep = []
    for n in w:
        keep.append(w[n])
        setattr(wts, n, w[n].ctypes.data_as(B._FP))
    d = B.Dims(d=100, embed_dim=32, n_kinds=4, n_params=2, trans_hidden=64, cost_hidden=64,
               hw_dim=16, feat_dim=0, enc_hidden=0, precision=B.WM_FP32, norm=B.WM_NORM_NONE)
    assert lib.wm_model_create(ctypes.byref(d), ctypes.byref(wts), ctypes.byref(h)) == B.WM_ERR_UNSUPPORTED
    d.d = 64
    # the paper-form transition needs its hyperplane-normal map; unknown forms are rejected
    d.norm = B.WM_NORM_L2
    assert lib.wm_model_create(ctypes.byref(d), ctypes.byref(wts), ctypes.byref(h)) == B.WM_ERR_INVALID_ARGUMENT
    d.norm = 7
    assert lib.wm_model_create(ctypes.byref(d), ctypes.byref(wts), ctypes.byref(h)) == B.WM_ERR_INVALID_ARGUMENT
    d.norm = B.WM_NORM_NONE
    d.trans_hidden = 96   # not a multiple of 64
    assert lib.wm_model_create(ctypes.byref(d), ctypes.byref(wts), ctypes.byref(h)) == B.WM_ERR_UNSUPPORTED


def test_workspace_bytes_rejects_bad_arguments():
    lib = wm.load_library()
    assert lib.wm_workspace_bytes(None, 8, 4, 1, 1) == 0
    assert lib.wm_device_status(None, 0, None) == B.WM_ERR_INVALID_ARGUMENT
    assert lib.wm_timing_read(99, None, None) == B.WM_ERR_INVALID_ARGUMENT


def test_binding_raises_when_library_missing(tmp_path):
    saved = B._lib
    B._lib = None
    try:
        with pytest.raises(RuntimeError):
            B.load_library(str(tmp_path / "nope.so"))
    finally:
        B._lib = saved


def test_forest_create_validates_before_device_work():
    lib = wm.load_library()
    h = ctypes.c_void_p()
    feat = np.array([0, 1, 5], np.int32)
    thr = np.zeros(3, np.float32)
    leaf = np.zeros(4, np.float32)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    # feature index 5 >= n_features 5
    assert lib.wm_forest_create(1, 2, 5, p(feat), p(thr), p(leaf), 0.0, ctypes.byref(h)) == B.WM_ERR_INVALID_ARGUMENT
    assert "out of range" in lib.wm_last_error().decode()
    neg = np.array([0, -1, 2], np.int32)
    assert lib.wm_forest_create(1, 2, 6, p(neg), p(thr), p(leaf), 0.0, ctypes.byref(h)) == B.WM_ERR_INVALID_ARGUMENT
    for depth in (0, 13):
        assert lib.wm_forest_create(1, depth, 6, p(feat), p(thr), p(leaf), 0.0, ctypes.byref(h)) == B.WM_ERR_INVALID_ARGUMENT
    assert lib.wm_forest_create(1, 2, 6, None, p(thr), p(leaf), 0.0, ctypes.byref(h)) == B.WM_ERR_INVALID_ARGUMENT
    assert lib.wm_score_trees(None, None, 0, None, 0, 0, None, 1, 0, None, None) == B.WM_ERR_INVALID_ARGUMENT
    assert lib.wm_phi_struct(None, None, None, 4, 8, 33, 2, None, None) == B.WM_ERR_UNSUPPORTED
    assert lib.wm_phi_struct(None, None, None, -1, 8, 4, 2, None, None) == B.WM_ERR_INVALID_ARGUMENT


def test_rollout_loss_rejects_before_device_work():
    lib = wm.load_library()
    assert lib.wm_loss_workspace_bytes(None, 4, 4) == 0
    fake = ctypes.c_void_p(256)   # never dereferenced: validation fails first
    arr, p = _seg([0, 4])
    st = lib.wm_rollout_loss(None, fake, p, 1, fake, fake, fake, 4, 4, fake, fake, 2, 0.5, 0.3,
                             fake, None, None, fake, 1 << 20, None)
    assert st == B.WM_ERR_INVALID_ARGUMENT
    assert "model" in lib.wm_last_error().decode()


def test_noalloc_rejects_before_device_work():
    lib = wm.load_library()
    arr, p = _seg([0, 8])
    fake = ctypes.c_void_p(256)   # never dereferenced: validation fails first
    assert lib.wm_evaluate_noalloc(None, fake, 0, p, 1, fake, fake, fake, 8, 4, fake, 1, 2, fake,
                                   fake, fake, fake, None, fake, None) == B.WM_ERR_INVALID_ARGUMENT
    assert "model" in lib.wm_last_error().decode()
