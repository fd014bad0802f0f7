"""Seeded synthetic workloads for the batched latent-rollout evaluator.

This module only draws random numbers: the five workload shapes, the
weights (N(0, 1/fan_in)) and the candidate batches (initial latents or
program-feature vectors, ragged action sequences, hardware vectors). It holds
none of the evaluator's arithmetic, so both the CPU oracle and the HIP path
can take their inputs from here without sharing any computation.

Workloads stand in for the paper's Ansor/TenSet candidate populations
(Sec. 4.1 and the online integration of Sec. 3.6): the tuning logs, models and
trained weights are not available, so shapes and distributions are synthetic.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass
from typing import Dict, Optional

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "workload", "make_weights", "make_inputs",
    "scaled", "WEIGHT_ORDER", "make_forest", "make_loss_targets", "TextWorkload",
    "TEXT_WORKLOADS", "TEXT_WEIGHT_ORDER", "make_text_weights", "make_programs",
]


@dataclass(frozen=True)
class Workload:
    """Shape and distribution of one synthetic candidate batch.

    d: latent width; e: action-embedding width; n_kinds/n_params: action
    types and integer parameters per step; H: transition hidden width;
    C: cost-model hidden width; hw_dim/n_hw: hardware vector width and count;
    S: subgraphs (contiguous candidate segments); feat_dim/enc_hidden: width
    of the program-feature vector and encoder hidden layer (0 = the initial
    latent is given directly); lengths: action-sequence length law.
    """
    name: str
    B: int
    d: int
    e: int
    n_kinds: int
    n_params: int
    H: int
    C: int
    hw_dim: int
    n_hw: int
    k: int
    S: int = 1
    feat_dim: int = 0
    enc_hidden: int = 0
    lengths: str = "uniform"       # "uniform" | "geometric"
    len_lo: int = 1
    len_hi: int = 8                # inclusive upper bound (uniform)
    geo_mean: float = 24.0         # geometric law on {1,2,...}
    T_max: int = 8                 # padded width of the action tensors
    precisions: tuple = ("fp32",)
    n_trees: int = 256             # tree-ensemble ranker: trees and depth
    tree_depth: int = 8

    @property
    def in_dim(self) -> int:
        """Width of the transition input [z; e]."""
        return self.d + self.e

    @property
    def cost_in(self) -> int:
        """Width of the cost-model input [z_T; phi; h]."""
        return self.d + self.e + self.hw_dim


WORKLOADS: Dict[str, Workload] = {
    # Tiny rollout, fp32.
    "tiny": Workload(
        name="tiny", B=256, d=64, e=32, n_kinds=12, n_params=4, H=128, C=128,
        hw_dim=16, n_hw=1, k=16, lengths="uniform", len_lo=1, len_hi=8,
        T_max=8, precisions=("fp32",)),
    # One Ansor search round: 2048 candidates, top-64 measured.
    "ansor_round": Workload(
        name="ansor_round", B=2048, d=256, e=64, n_kinds=16, n_params=6,
        H=512, C=512, hw_dim=32, n_hw=1, k=64, lengths="uniform", len_lo=1,
        len_hi=32, T_max=32, precisions=("fp32", "bf16")),
    # Long schedules with skewed (geometric, capped) lengths.
    "long_schedule": Workload(
        name="long_schedule", B=8192, d=256, e=64, n_kinds=16, n_params=6,
        H=1024, C=512, hw_dim=32, n_hw=1, k=64, lengths="geometric",
        geo_mean=24.0, T_max=64, precisions=("bf16",)),
    # Large-latent throughput: the dense-contraction-bound shape.
    "large_latent": Workload(
        name="large_latent", B=65536, d=512, e=128, n_kinds=16, n_params=6,
        H=2048, C=1024, hw_dim=32, n_hw=1, k=256, lengths="uniform",
        len_lo=8, len_hi=48, T_max=48, precisions=("bf16",)),
    # 32 subgraphs x 2048 candidates, encoder MLP for the initial states,
    # every candidate scored under two hardware vectors.
    "multi_subgraph": Workload(
        name="multi_subgraph", B=65536, S=32, d=256, e=64, n_kinds=16,
        n_params=6, H=512, C=512, hw_dim=32, n_hw=2, k=32, feat_dim=164,
        enc_hidden=512, lengths="uniform", len_lo=1, len_hi=48, T_max=48,
        precisions=("bf16",)),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def scaled(w: Workload, B: int, S: Optional[int] = None, **kw) -> Workload:
    """Same model shapes, smaller batch (and optionally fewer segments)."""
    S = w.S if S is None else S
    if B % S:
        raise ValueError("B must be a multiple of S")
    return dataclasses.replace(w, B=B, S=S, **kw)


# Fixed draw order of the weight tensors.  Each is N(0, 1/fan_in); a bias uses
# the standard deviation of its layer's weight.
WEIGHT_ORDER = (
    "type_emb", "param_w", "param_b", "w1", "b1", "w2", "b2",
    "wc1", "bc1", "wc2", "bc2", "we1", "be1", "we2", "be2", "wh",
)


def _weight_shapes(w: Workload):
    """(shape, fan_in) per weight, PyTorch Linear layout [out][in]."""
    s = {
        "type_emb": ((w.n_kinds, w.e), w.n_kinds),     # one-hot linear
        "param_w": ((w.e, w.n_params), w.n_params),
        "param_b": ((w.e,), w.n_params),
        "w1": ((w.H, w.in_dim), w.in_dim),
        "b1": ((w.H,), w.in_dim),
        "w2": ((w.d, w.H), w.H),
        "b2": ((w.d,), w.H),
        "wc1": ((w.C, w.cost_in), w.cost_in),
        "bc1": ((w.C,), w.cost_in),
        "wc2": ((w.C,), w.C),
        "bc2": ((), w.C),
        # hyperplane-normal map of the paper-form transition (drawn last, so
        # the tensors above do not depend on whether it is used)
        "wh": ((w.d, w.e), w.e),
    }
    if w.feat_dim:
        s.update({
            "we1": ((w.enc_hidden, w.feat_dim), w.feat_dim),
            "be1": ((w.enc_hidden,), w.feat_dim),
            "we2": ((w.d, w.enc_hidden), w.enc_hidden),
            "be2": ((w.d,), w.enc_hidden),
        })
    return s


def make_weights(w: Workload, seed: int) -> Dict[str, np.ndarray]:
    """All weights as float32 arrays, drawn in WEIGHT_ORDER from PCG64(seed)."""
    rng = np.random.default_rng(seed)
    shapes = _weight_shapes(w)
    out = {}
    for name in WEIGHT_ORDER:
        if name not in shapes:
            continue
        shape, fan_in = shapes[name]
        out[name] = (rng.standard_normal(shape) / np.sqrt(fan_in)).astype(np.float32)
    return out


def _lengths(w: Workload, rng: np.random.Generator) -> np.ndarray:
    if w.lengths == "uniform":
        L = rng.integers(w.len_lo, w.len_hi + 1, size=w.B)
    elif w.lengths == "geometric":
        L = np.minimum(rng.geometric(1.0 / w.geo_mean, size=w.B), w.T_max)
    else:
        raise ValueError(w.lengths)
    return L.astype(np.int32)


def make_inputs(w: Workload, seed: int, pad: str = "zero") -> Dict[str, np.ndarray]:
    """One candidate batch.

    Returns int32 `types [B][T_max]`, `params [B][T_max][P]`, `lens [B]`,
    `seg_off [S+1]`, float32 `hw [n_hw][hw_dim]`, and either `z0 [S][d]`
    (N(0,1)) or `feats [S][feat_dim]` (|N(0,1)|).  Parameters are
    floor(2**U[0,10)), i.e. log-uniform integers in [1, 1023].  Entries at
    t >= lens[i] are padding: zeros (pad="zero") or arbitrary, partly invalid
    integers (pad="garbage") that a correct evaluator never reads.
    """
    rng = np.random.default_rng(seed)
    lens = _lengths(w, rng)
    types = rng.integers(0, w.n_kinds, size=(w.B, w.T_max)).astype(np.int32)
    params = np.floor(2.0 ** rng.uniform(0.0, 10.0, size=(w.B, w.T_max, w.n_params))).astype(np.int32)
    if w.feat_dim:
        init = {"feats": np.abs(rng.standard_normal((w.S, w.feat_dim))).astype(np.float32)}
    else:
        init = {"z0": rng.standard_normal((w.S, w.d)).astype(np.float32)}
    hw = rng.standard_normal((w.n_hw, w.hw_dim)).astype(np.float32)
    t = np.arange(w.T_max)[None, :]
    pad_mask = t >= lens[:, None]
    if pad == "zero":
        types[pad_mask] = 0
        params[pad_mask] = 0
    elif pad == "garbage":
        g = np.random.default_rng(seed ^ 0x5EED)
        types[pad_mask] = g.integers(-1000, 1000, size=int(pad_mask.sum()))
        params[pad_mask] = g.integers(-(2 ** 31), 2 ** 31 - 1, size=(int(pad_mask.sum()), w.n_params))
    else:
        raise ValueError(pad)
    seg = w.B // w.S
    seg_off = (np.arange(w.S + 1) * seg).astype(np.int32)
    out = {"types": types, "params": params, "lens": lens, "hw": hw, "seg_off": seg_off}
    out.update(init)
    return out


def make_forest(w: Workload, seed: int, n_trees: Optional[int] = None, depth: Optional[int] = None,
                z_scale: float = 1.0) -> Dict[str, np.ndarray]:
    """A random tree ensemble over x = [z_T ; phi_s ; h] (a stand-in for a
    trained ranker).  Complete trees of the given depth, breadth-first:
    `feat` [NT][2^D - 1] int32 feature indices drawn uniformly, `thr`
    [NT][2^D - 1] float32 thresholds drawn from a range that suits the
    feature's block (z: N(0, z_scale); kind counts: U(0, 2 T_max / K);
    length: U(1, T_max); log2-parameter statistics: U(0, 10); hardware:
    N(0, 1)), `leaf` [NT][2^D] float32 ~ N(0, 0.1), `base` 0.5.
    """
    rng = np.random.default_rng(seed)
    NT = w.n_trees if n_trees is None else n_trees
    D = w.tree_depth if depth is None else depth
    K, P = w.n_kinds, w.n_params
    n_phi = K + 1 + 2 * P
    F = w.d + n_phi + w.hw_dim
    n_int = 2 ** D - 1
    feat = rng.integers(0, F, size=(NT, n_int)).astype(np.int32)
    r = rng.random((NT, n_int))
    g = rng.standard_normal((NT, n_int))
    thr = np.empty((NT, n_int))
    j = feat - w.d                                   # index within phi_s (when >= 0)
    is_z = feat < w.d
    is_cnt = (j >= 0) & (j < K)
    is_len = j == K
    is_par = (j > K) & (j < n_phi)
    is_hw = feat >= w.d + n_phi
    thr[is_z] = z_scale * g[is_z]
    thr[is_cnt] = r[is_cnt] * 2.0 * w.T_max / K
    thr[is_len] = 1.0 + r[is_len] * (w.T_max - 1)
    thr[is_par] = 10.0 * r[is_par]
    thr[is_hw] = g[is_hw]
    leaf = 0.1 * rng.standard_normal((NT, n_int + 1))
    return {"feat": feat, "thr": thr.astype(np.float32), "leaf": leaf.astype(np.float32),
            "base": np.float32(0.5)}


def make_loss_targets(w: Workload, seed: int, n_neg: int, lens=None):
    """Rollout-loss inputs of the batch's shape: targets [B][T_max][d] and
    negatives [B][T_max][n_neg][d], N(0,1) float32 (a stand-in for encoded
    observed next states and sampled negative states); entries at
    t >= lens[i] are NaN when lens is given (a correct loss never reads them).
    """
    rng = np.random.default_rng(seed)
    tgt = rng.standard_normal((w.B, w.T_max, w.d), dtype=np.float32)
    neg = rng.standard_normal((w.B, w.T_max, n_neg, w.d), dtype=np.float32)
    if lens is not None:
        pad = np.arange(w.T_max)[None, :] >= np.asarray(lens)[:, None]
        tgt[pad] = np.nan
        neg[pad] = np.nan
    return tgt, neg


# ---- chunked transformer state encoder (Sec. 3.3) -------------------------

@dataclass(frozen=True)
class TextWorkload:
    """Shape of the chunked transformer encoder and of a batch of programs.

    vocab/hidden/heads/ffn/layers: the backbone (the CodeBERT shape is
    RoBERTa-base); window/stride: the sliding-window chunks; d: the latent
    width of the projection head; S programs with token counts uniform in
    [len_lo, len_hi].
    """
    name: str
    S: int
    vocab: int
    hidden: int
    heads: int
    ffn: int
    layers: int
    window: int
    stride: int
    d: int
    len_lo: int
    len_hi: int


TEXT_WORKLOADS: Dict[str, TextWorkload] = {
    # small backbone for whole-batch parity checks
    "tiny_text": TextWorkload(name="tiny_text", S=6, vocab=1000, hidden=128, heads=4, ffn=256,
                              layers=2, window=64, stride=32, d=64, len_lo=0, len_hi=200),
    # CodeBERT (RoBERTa-base) backbone, 512-token windows with half overlap,
    # 32 programs of 256..2048 tokens, projected to the 256-d latent
    "codebert": TextWorkload(name="codebert", S=32, vocab=50265, hidden=768, heads=12, ffn=3072,
                             layers=12, window=512, stride=256, d=256, len_lo=256, len_hi=2048),
}

TEXT_WEIGHT_ORDER = ("tok_emb", "pos_emb", "ln0_g", "ln0_b", "wqkv", "bqkv", "wo", "bo", "ln1_g",
                     "ln1_b", "w1", "b1", "w2", "b2", "ln2_g", "ln2_b", "wp", "bp")


def make_text_weights(w: TextWorkload, seed: int) -> Dict[str, np.ndarray]:
    """Random encoder weights, float32: matrices, embeddings and biases
    N(0, 0.02^2) (the usual initialisation of this backbone family), LayerNorm
    gains 1 + N(0, 0.02^2) and shifts N(0, 0.02^2); the projection head
    N(0, 1/hidden).  Layers are stacked on a leading axis."""
    rng = np.random.default_rng(seed)
    H, F, L = w.hidden, w.ffn, w.layers
    shapes = {
        "tok_emb": (w.vocab, H), "pos_emb": (w.window, H), "ln0_g": (H,), "ln0_b": (H,),
        "wqkv": (L, 3 * H, H), "bqkv": (L, 3 * H), "wo": (L, H, H), "bo": (L, H),
        "ln1_g": (L, H), "ln1_b": (L, H), "w1": (L, F, H), "b1": (L, F), "w2": (L, H, F),
        "b2": (L, H), "ln2_g": (L, H), "ln2_b": (L, H), "wp": (w.d, H), "bp": (w.d,),
    }
    out = {}
    for k in TEXT_WEIGHT_ORDER:
        std = 1.0 / np.sqrt(H) if k in ("wp", "bp") else 0.02
        a = rng.standard_normal(shapes[k], dtype=np.float32) * np.float32(std)
        if k.endswith("_g"):
            a += np.float32(1.0)
        out[k] = a
    return out


def make_programs(w: TextWorkload, seed: int):
    """S programs of token ids (int32, uniform over the vocabulary) with
    lengths uniform in [len_lo, len_hi]; returns (tokens [N_total],
    tok_off [S+1])."""
    rng = np.random.default_rng(seed)
    lens = rng.integers(w.len_lo, w.len_hi + 1, size=w.S)
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    tokens = rng.integers(0, w.vocab, size=int(off[-1])).astype(np.int32)
    return tokens, off
