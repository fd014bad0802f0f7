"""ctypes binding of libwm.so (the C ABI in include/wm.h).

Argument marshalling only: every step of the evaluator runs in the library's
HIP kernels.  Device buffers are torch CUDA (HIP) tensors; the stream is
torch's current stream unless one is given.  A missing library raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwm.so")

WM_OK, WM_ERR_INVALID_ARGUMENT, WM_ERR_UNSUPPORTED = 0, 1, 2
WM_ERR_OUT_OF_MEMORY, WM_ERR_DEVICE, WM_ERR_INPUT_RANGE = 3, 4, 5
WM_FP32, WM_BF16 = 0, 1
WM_NORM_NONE, WM_NORM_L2 = 0, 1
PRECISIONS = {"fp32": WM_FP32, "bf16": WM_BF16}
NORMS = {"none": WM_NORM_NONE, "l2": WM_NORM_L2}
KERNELS = {"rollout": 0, "score": 1, "topk": 2, "bucket": 3, "phi": 4, "encode": 5,
           "phi_struct": 6, "trees": 7, "loss_fwd": 8, "loss_steps": 9, "loss_bwd": 10,
           "loss_grads": 11, "text_gemm": 12, "text_attn": 13, "text_other": 14}

# Exported symbols (kept in step with include/wm.h).
SYMBOLS = (
    "wm_model_create", "wm_model_destroy", "wm_workspace_bytes", "wm_encode_init",
    "wm_rollout", "wm_score", "wm_topk", "wm_evaluate", "wm_device_status",
    "wm_last_error", "wm_timing_enable", "wm_timing_read", "wm_forest_create",
    "wm_forest_destroy", "wm_phi_struct", "wm_score_trees", "wm_evaluate_trees",
    "wm_loss_workspace_bytes", "wm_rollout_loss", "wm_text_model_create", "wm_text_model_destroy",
    "wm_text_chunks", "wm_text_workspace_bytes", "wm_encode_text", "wm_evaluate_noalloc",
)


class WMError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"wm status {status}: {msg}")
        self.status = status
        self.msg = msg


class Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "d", "embed_dim", "n_kinds", "n_params", "trans_hidden", "cost_hidden", "hw_dim",
        "feat_dim", "enc_hidden", "precision", "norm")]


_FP = ctypes.POINTER(ctypes.c_float)


class Weights(ctypes.Structure):
    _fields_ = [
        ("type_emb", _FP), ("param_w", _FP), ("param_b", _FP),
        ("w1", _FP), ("b1", _FP), ("w2", _FP), ("b2", _FP),
        ("wc1", _FP), ("bc1", _FP), ("wc2", _FP), ("bc2", ctypes.c_float),
        ("we1", _FP), ("be1", _FP), ("we2", _FP), ("be2", _FP),
        ("wh", _FP),
    ]


class Grads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "w1", "b1", "w2", "b2", "type_emb", "param_w", "param_b", "z0", "wh")]


GRAD_KEYS = ("w1", "b1", "w2", "b2", "type_emb", "param_w", "param_b")


class TextDims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "vocab", "hidden", "heads", "ffn", "layers", "window", "stride", "d", "precision")]


TEXT_WEIGHT_KEYS = ("tok_emb", "pos_emb", "ln0_g", "ln0_b", "wqkv", "bqkv", "wo", "bo", "ln1_g",
                    "ln1_b", "w1", "b1", "w2", "b2", "ln2_g", "ln2_b", "wp", "bp")


class TextWeights(ctypes.Structure):
    _fields_ = [(n, _FP) for n in TEXT_WEIGHT_KEYS]

_lib = None


def load_library(path: str = LIB_PATH):
    """Load libwm.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2606_09312_amd.build.build()")
    # Load torch first so the library binds to the HIP runtime torch uses
    # (one runtime per process; device buffers and streams come from torch).
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    lib.wm_model_create.argtypes = [ctypes.POINTER(Dims), ctypes.POINTER(Weights), ctypes.POINTER(vp)]
    lib.wm_model_create.restype = i32
    lib.wm_model_destroy.argtypes = [vp]
    lib.wm_model_destroy.restype = None
    lib.wm_workspace_bytes.argtypes = [vp, i32, i32, i32, i32]
    lib.wm_workspace_bytes.restype = sz
    lib.wm_encode_init.argtypes = [vp, vp, i32, vp, vp]
    lib.wm_encode_init.restype = i32
    lib.wm_rollout.argtypes = [vp, vp, vp, i32, vp, vp, vp, i32, i32, vp, vp, vp, sz, vp]
    lib.wm_rollout.restype = i32
    lib.wm_score.argtypes = [vp, vp, vp, i32, vp, i32, vp, vp]
    lib.wm_score.restype = i32
    lib.wm_topk.argtypes = [vp, i32, i32, vp, i32, i32, vp, vp, vp]
    lib.wm_topk.restype = i32
    lib.wm_evaluate.argtypes = [vp, vp, i32, vp, i32, vp, vp, vp, i32, i32, vp, i32, i32,
                                vp, vp, vp, vp, vp, sz, vp]
    lib.wm_evaluate.restype = i32
    lib.wm_evaluate_noalloc.argtypes = [vp, vp, i32, vp, i32, vp, vp, vp, i32, i32, vp, i32, i32,
                                        vp, vp, vp, vp, vp, vp, vp]
    lib.wm_evaluate_noalloc.restype = i32
    lib.wm_device_status.argtypes = [vp, sz, vp]
    lib.wm_device_status.restype = i32
    lib.wm_last_error.argtypes = []
    lib.wm_last_error.restype = ctypes.c_char_p
    lib.wm_timing_enable.argtypes = [i32]
    lib.wm_timing_enable.restype = i32
    lib.wm_timing_read.argtypes = [i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]
    lib.wm_timing_read.restype = i32
    lib.wm_forest_create.argtypes = [i32, i32, i32, vp, vp, vp, ctypes.c_float, ctypes.POINTER(vp)]
    lib.wm_forest_create.restype = i32
    lib.wm_forest_destroy.argtypes = [vp]
    lib.wm_forest_destroy.restype = None
    lib.wm_phi_struct.argtypes = [vp, vp, vp, i32, i32, i32, i32, vp, vp]
    lib.wm_phi_struct.restype = i32
    lib.wm_score_trees.argtypes = [vp, vp, i32, vp, i32, i32, vp, i32, i32, vp, vp]
    lib.wm_score_trees.restype = i32
    lib.wm_evaluate_trees.argtypes = [vp, vp, vp, i32, vp, i32, vp, vp, vp, i32, i32, vp, i32, i32,
                                      vp, vp, vp, vp, vp, sz, vp]
    lib.wm_evaluate_trees.restype = i32
    lib.wm_loss_workspace_bytes.argtypes = [vp, i32, i32]
    lib.wm_loss_workspace_bytes.restype = sz
    lib.wm_rollout_loss.argtypes = [vp, vp, vp, i32, vp, vp, vp, i32, i32, vp, vp, i32,
                                    ctypes.c_float, ctypes.c_float, vp, vp, ctypes.POINTER(Grads),
                                    vp, sz, vp]
    lib.wm_rollout_loss.restype = i32
    lib.wm_text_model_create.argtypes = [ctypes.POINTER(TextDims), ctypes.POINTER(TextWeights),
                                         ctypes.POINTER(vp)]
    lib.wm_text_model_create.restype = i32
    lib.wm_text_model_destroy.argtypes = [vp]
    lib.wm_text_model_destroy.restype = None
    lib.wm_text_chunks.argtypes = [vp, vp, i32]
    lib.wm_text_chunks.restype = i32
    lib.wm_text_workspace_bytes.argtypes = [vp, i32]
    lib.wm_text_workspace_bytes.restype = sz
    lib.wm_encode_text.argtypes = [vp, vp, vp, i32, vp, vp, sz, vp]
    lib.wm_encode_text.restype = i32
    _lib = lib
    return lib


def _check(status: int):
    if status != WM_OK:
        raise WMError(status, load_library().wm_last_error().decode())


def _ptr(t):
    """Device pointer of a torch tensor (or None)."""
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _host_i32(a):
    a = np.ascontiguousarray(np.asarray(a), dtype=np.int32)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


class Model:
    """Device copy of the evaluator's weights (wm_model_create)."""

    def __init__(self, dims: Dict[str, int], weights: Dict[str, np.ndarray], precision: str = "bf16",
                 norm: str = "none"):
        """norm="l2" selects the paper-form transition (hyperplane projection
        and unit length; needs weights["wh"])."""
        lib = load_library()
        self.dims = dict(dims)
        self.precision = precision
        self.norm = norm
        d = Dims(d=dims["d"], embed_dim=dims["e"], n_kinds=dims["n_kinds"],
                 n_params=dims["n_params"], trans_hidden=dims["H"], cost_hidden=dims["C"],
                 hw_dim=dims["hw_dim"], feat_dim=dims.get("feat_dim", 0),
                 enc_hidden=dims.get("enc_hidden", 0), precision=PRECISIONS[precision],
                 norm=NORMS[norm])
        self._keep = {k: np.ascontiguousarray(v, dtype=np.float32) for k, v in weights.items()}
        w = Weights()
        for name, _ in Weights._fields_:
            if name == "bc2":
                w.bc2 = float(np.asarray(self._keep["bc2"]).reshape(-1)[0])
            elif name in self._keep:
                setattr(w, name, self._keep[name].ctypes.data_as(_FP))
        h = ctypes.c_void_p()
        _check(lib.wm_model_create(ctypes.byref(d), ctypes.byref(w), ctypes.byref(h)))
        self.handle = h

    def close(self):
        if getattr(self, "handle", None):
            load_library().wm_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace_bytes(self, B: int, T_max: int, S: int, n_hw: int) -> int:
        return int(load_library().wm_workspace_bytes(self.handle, B, T_max, S, n_hw))

    def workspace(self, B: int, T_max: int, S: int, n_hw: int, device="cuda"):
        """Zero-filled workspace tensor (uint8) of the required size."""
        import torch
        return torch.zeros(self.workspace_bytes(B, T_max, S, n_hw), dtype=torch.uint8, device=device)


def encode_init(model: Model, feats, z0, stream=None):
    S = feats.shape[0]
    _check(load_library().wm_encode_init(model.handle, _ptr(feats), S, _ptr(z0), _stream(stream)))


def rollout(model: Model, z0, seg_off, types, params, lens, zT, phi, ws, stream=None):
    seg, segp = _host_i32(seg_off)
    B, T_max = types.shape[0], types.shape[1]
    _check(load_library().wm_rollout(
        model.handle, _ptr(z0), segp, len(seg) - 1, _ptr(types), _ptr(params), _ptr(lens),
        B, T_max, _ptr(zT), _ptr(phi), _ptr(ws), ws.numel(), _stream(stream)))


def score(model: Model, zT, phi, hw, scores, stream=None):
    _check(load_library().wm_score(model.handle, _ptr(zT), _ptr(phi), zT.shape[0], _ptr(hw),
                                   hw.shape[0], _ptr(scores), _stream(stream)))


def topk(scores, seg_off, k, idx, val=None, stream=None):
    seg, segp = _host_i32(seg_off)
    _check(load_library().wm_topk(_ptr(scores), scores.shape[0], scores.shape[1], segp,
                                  len(seg) - 1, k, _ptr(idx), _ptr(val), _stream(stream)))


class Forest:
    """Device copy of a tree-ensemble ranker (wm_forest_create)."""

    def __init__(self, feat, thr, leaf, base: float, n_features: int):
        lib = load_library()
        feat = np.ascontiguousarray(feat, dtype=np.int32)
        self._keep = (feat, np.ascontiguousarray(thr, dtype=np.float32),
                      np.ascontiguousarray(leaf, dtype=np.float32))
        n_trees, n_int = feat.shape
        depth = int(round(np.log2(n_int + 1)))
        self.n_trees, self.depth, self.n_features = n_trees, depth, n_features
        h = ctypes.c_void_p()
        _check(lib.wm_forest_create(n_trees, depth, n_features,
                                    *[a.ctypes.data_as(ctypes.c_void_p) for a in self._keep],
                                    float(base), ctypes.byref(h)))
        self.handle = h

    def close(self):
        if getattr(self, "handle", None):
            load_library().wm_forest_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def phi_struct(types, params, lens, n_kinds: int, phi_s, stream=None):
    B, T_max = types.shape[0], types.shape[1]
    _check(load_library().wm_phi_struct(_ptr(types), _ptr(params), _ptr(lens), B, T_max, n_kinds,
                                        params.shape[2], _ptr(phi_s), _stream(stream)))


def score_trees(forest: Forest, zT, phi_s, hw, scores, stream=None):
    _check(load_library().wm_score_trees(forest.handle, _ptr(zT), zT.shape[1], _ptr(phi_s),
                                         phi_s.shape[1], zT.shape[0], _ptr(hw), hw.shape[0],
                                         hw.shape[1], _ptr(scores), _stream(stream)))


def evaluate(model: Model, init, seg_off, types, params, lens, hw, k, *, init_is_feats=False,
             scores=None, zT=None, idx=None, val=None, ws=None, stream=None, forest=None):
    """Fused [encode,] rollout, score and top-k (wm_evaluate) on device tensors;
    with a Forest, the tree-ensemble ranker on structured action features
    (wm_evaluate_trees).

    Returns a dict with idx [n_hw][S][k], val, and scores / zT when given.
    """
    import torch
    seg, segp = _host_i32(seg_off)
    S = len(seg) - 1
    B, T_max = types.shape[0], types.shape[1]
    n_hw = hw.shape[0]
    dev = types.device
    if idx is None:
        idx = torch.empty((n_hw, S, k), dtype=torch.int32, device=dev)
    if val is None:
        val = torch.empty((n_hw, S, k), dtype=torch.float32, device=dev)
    if ws is None:
        ws = model.workspace(B, T_max, S, n_hw, device=dev)
    args = (_ptr(init), 1 if init_is_feats else 0, segp, S, _ptr(types), _ptr(params),
            _ptr(lens), B, T_max, _ptr(hw), n_hw, k, _ptr(scores), _ptr(zT), _ptr(idx), _ptr(val),
            _ptr(ws), ws.numel(), _stream(stream))
    if forest is None:
        _check(load_library().wm_evaluate(model.handle, *args))
    else:
        _check(load_library().wm_evaluate_trees(model.handle, forest.handle, *args))
    return {"idx": idx, "val": val, "scores": scores, "zT": zT, "ws": ws}


def evaluate_noalloc(model: Model, init, seg_off, types, params, lens, hw, k, *, scores, zT, phi,
                     idx, status, val=None, init_is_feats=False, stream=None):
    """wm_evaluate_noalloc: the fused path with every output supplied by the
    caller (scores [n_hw][B], zT [B][d], phi [B][e], idx [n_hw][S][k], val or
    None, status int32 [64]) and no workspace; nothing is allocated.  Check
    the device error word with device_status(status)."""
    seg, segp = _host_i32(seg_off)
    S = len(seg) - 1
    B, T_max = types.shape[0], types.shape[1]
    n_hw = hw.shape[0]
    _check(load_library().wm_evaluate_noalloc(
        model.handle, _ptr(init), 1 if init_is_feats else 0, segp, S, _ptr(types), _ptr(params),
        _ptr(lens), B, T_max, _ptr(hw), n_hw, k, _ptr(scores), _ptr(zT), _ptr(phi), _ptr(idx),
        _ptr(val), _ptr(status), _stream(stream)))
    return {"idx": idx, "val": val, "scores": scores, "zT": zT, "phi": phi, "status": status}


def grad_shapes(model: Model) -> Dict[str, tuple]:
    """Shapes of the weight gradients of a model (PyTorch Linear layout)."""
    d = model.dims
    shapes = {"w1": (d["H"], d["d"] + d["e"]), "b1": (d["H"],), "w2": (d["d"], d["H"]),
              "b2": (d["d"],), "type_emb": (d["n_kinds"], d["e"]),
              "param_w": (d["e"], d["n_params"]), "param_b": (d["e"],)}
    if model.norm == "l2":
        shapes["wh"] = (d["d"], d["e"])
    return shapes


def loss_workspace(model: Model, B: int, T_max: int, device="cuda"):
    """Zero-filled workspace tensor (uint8) for rollout_loss."""
    import torch
    n = int(load_library().wm_loss_workspace_bytes(model.handle, B, T_max))
    return torch.zeros(n, dtype=torch.uint8, device=device)


def rollout_loss(model: Model, z0, seg_off, types, params, lens, targets, negatives, lam: float,
                 gamma: float, *, grads=True, dz0=True, loss=None, total=None, out=None, ws=None,
                 stream=None):
    """Rollout loss and its gradients (wm_rollout_loss) on device tensors.

    targets [B][T_max][d], negatives [B][T_max][n_neg][d].  Returns a dict
    with loss [B], total [1] and, when grads is true, the weight gradients
    (keys of grad_shapes) and z0 [B][d] (when dz0 is true).  `out` may hold
    preallocated gradient tensors under the same keys.
    """
    import torch
    seg, segp = _host_i32(seg_off)
    S = len(seg) - 1
    B, T_max = types.shape[0], types.shape[1]
    dev = types.device
    if loss is None:
        loss = torch.empty(B, dtype=torch.float32, device=dev)
    if total is None:
        total = torch.empty(1, dtype=torch.float32, device=dev)
    if ws is None:
        ws = loss_workspace(model, B, T_max, device=dev)
    res = {"loss": loss, "total": total, "ws": ws}
    gp = None
    if grads:
        out = dict(out or {})
        for k, shp in grad_shapes(model).items():
            if k not in out:
                out[k] = torch.empty(shp, dtype=torch.float32, device=dev)
        if dz0 and "z0" not in out:
            out["z0"] = torch.empty((B, model.dims["d"]), dtype=torch.float32, device=dev)
        g = Grads(**{k: _ptr(v).value for k, v in out.items() if k in dict(Grads._fields_)})
        gp = ctypes.byref(g)
        res.update(out)
    _check(load_library().wm_rollout_loss(
        model.handle, _ptr(z0), segp, S, _ptr(types), _ptr(params), _ptr(lens), B, T_max,
        _ptr(targets), _ptr(negatives), negatives.shape[2] if negatives.dim() == 4 else 0,
        float(lam), float(gamma), _ptr(loss), _ptr(total), gp, _ptr(ws), ws.numel(),
        _stream(stream)))
    return res


class TextModel:
    """Device copy of the chunked transformer state encoder (wm_text_model_create)."""

    def __init__(self, w, weights: Dict[str, np.ndarray], precision: str = "bf16"):
        """w: object with vocab, hidden, heads, ffn, layers, window, stride, d."""
        lib = load_library()
        self.w = w
        self.precision = precision
        d = TextDims(vocab=w.vocab, hidden=w.hidden, heads=w.heads, ffn=w.ffn, layers=w.layers,
                     window=w.window, stride=w.stride, d=w.d, precision=PRECISIONS[precision])
        self._keep = {k: np.ascontiguousarray(weights[k], dtype=np.float32) for k in TEXT_WEIGHT_KEYS}
        tw = TextWeights(**{k: self._keep[k].ctypes.data_as(_FP) for k in TEXT_WEIGHT_KEYS})
        h = ctypes.c_void_p()
        _check(lib.wm_text_model_create(ctypes.byref(d), ctypes.byref(tw), ctypes.byref(h)))
        self.handle = h
        self._keep = None           # copied to the device

    def close(self):
        if getattr(self, "handle", None):
            load_library().wm_text_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def chunks(self, tok_off) -> int:
        off, offp = _host_i32(tok_off)
        n = int(load_library().wm_text_chunks(self.handle, offp, len(off) - 1))
        if n < 0:
            raise WMError(WM_ERR_INVALID_ARGUMENT, "bad tok_off")
        return n

    def workspace(self, tok_off, device="cuda"):
        import torch
        n = int(load_library().wm_text_workspace_bytes(self.handle, self.chunks(tok_off)))
        return torch.zeros(n, dtype=torch.uint8, device=device)


def encode_text(model: TextModel, tokens, tok_off, z0=None, ws=None, stream=None):
    """z0 [S][d] from concatenated token ids (device int32) and HOST tok_off [S+1]."""
    import torch
    off, offp = _host_i32(tok_off)
    S = len(off) - 1
    dev = tokens.device
    if z0 is None:
        z0 = torch.empty((S, model.w.d), dtype=torch.float32, device=dev)
    if ws is None:
        ws = model.workspace(off, device=dev)
    _check(load_library().wm_encode_text(model.handle, _ptr(tokens), offp, S, _ptr(z0), _ptr(ws),
                                         ws.numel(), _stream(stream)))
    return {"z0": z0, "ws": ws}


def device_status(ws, stream=None) -> int:
    """Synchronise and read/clear the workspace error word; raises on an error."""
    _check(load_library().wm_device_status(_ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))
    return WM_OK


def timing_enable(on: bool):
    _check(load_library().wm_timing_enable(1 if on else 0))


def timing_read(kernel: str):
    """(total milliseconds, launches) recorded for a kernel family since enabling."""
    ms, n = ctypes.c_double(), ctypes.c_int64()
    _check(load_library().wm_timing_read(KERNELS[kernel], ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value
