"""Reference oracle for the structured action features and the tree-ensemble
ranker (float64 features, float32 decisions; NumPy).

TEST INFRASTRUCTURE ONLY: the plain definition used to check the HIP path.
Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import it; the product path never calls it.

What is computed (paper, Sec. 3.5: the ranking model G is a gradient-boosted
tree ensemble over the predicted terminal state, a structured action-feature
vector and the hardware vector; the structured features are action counts,
the sequence length and action-specific numeric attributes):

  u_{t,p} = log2(params[t, p])
  phi_s   = [ n_0 .. n_{K-1},  T,  mean_t u_{t,0..P-1},  max_t u_{t,0..P-1} ]
            (n_k = number of steps of kind k; all zero when T = 0)
  x       = [ z_T ; phi_s ; h ]
  y       = base + sum over trees of the leaf reached by x

A tree of depth D is complete and stored breadth-first: internal node i
(0 <= i < 2^D - 1) holds a feature index f_i and a threshold c_i, and x goes
to child 2i+1 when x[f_i] < c_i, else to child 2i+2 (so a NaN feature goes
right); the leaf reached is node 2^D - 1 + l, with value leaf[l].  The
decisions compare float32 feature values with float32 thresholds, as the
GPU does (a comparison decides an integer path, so both sides take it in the
same precision); leaf values are summed in float64.

Pinned by tests/test_oracle_tree_pins.py (scikit-learn's decision-tree
inference, hand-built stumps, hand-computed feature vectors).
"""
from __future__ import annotations

import numpy as np


def phi_dim(n_kinds: int, n_params: int) -> int:
    """Width of the structured action-feature vector."""
    return n_kinds + 1 + 2 * n_params


def structured_phi(types, params, lens, n_kinds: int) -> np.ndarray:
    """phi_s for every candidate; entries at t >= lens[i] are never read.

    types [B][T_max] int, params [B][T_max][P] int (>= 1 at valid steps),
    lens [B]  ->  [B][K + 1 + 2P] float64.
    """
    types = np.asarray(types)
    params = np.asarray(params)
    lens = np.asarray(lens, dtype=np.int64)
    B = lens.shape[0]
    P = params.shape[2]
    out = np.zeros((B, phi_dim(n_kinds, P)))
    for i in range(B):
        L = int(lens[i])
        if L == 0:
            continue
        ty = types[i, :L]
        u = np.log2(params[i, :L, :].astype(np.float64))
        for k in range(n_kinds):
            out[i, k] = np.count_nonzero(ty == k)
        out[i, n_kinds] = L
        out[i, n_kinds + 1:n_kinds + 1 + P] = u.mean(axis=0)
        out[i, n_kinds + 1 + P:] = u.max(axis=0)
    return out


def tree_features(zT, phi_s, hw_row) -> np.ndarray:
    """x = [z_T ; phi_s ; h] for every candidate under one hardware vector."""
    zT = np.asarray(zT, dtype=np.float64)
    B = zT.shape[0]
    h = np.broadcast_to(np.asarray(hw_row, dtype=np.float64), (B, len(hw_row)))
    return np.concatenate([zT, np.asarray(phi_s, dtype=np.float64), h], axis=1)


def forest_predict(x, feat, thr, leaf, base: float) -> np.ndarray:
    """Sum of the leaves reached in every tree, plus base.

    x [B][F]; feat [NT][2^D - 1] int; thr [NT][2^D - 1]; leaf [NT][2^D].
    Decisions: float32(x[f]) < float32(c) goes left.
    """
    x32 = np.asarray(x, dtype=np.float64).astype(np.float32)
    feat = np.asarray(feat)
    thr32 = np.asarray(thr, dtype=np.float32)
    leaf = np.asarray(leaf, dtype=np.float64)
    NT, n_int = feat.shape
    depth = int(round(np.log2(n_int + 1)))
    B = x32.shape[0]
    rows = np.arange(B)
    y = np.full(B, float(base))
    for t in range(NT):
        node = np.zeros(B, dtype=np.int64)
        for _ in range(depth):
            f = feat[t, node]
            go_left = x32[rows, f] < thr32[t, node]
            node = 2 * node + np.where(go_left, 1, 2)
        y += leaf[t, node - n_int]
    return y


def score_trees(zT, phi_s, hw, feat, thr, leaf, base: float) -> np.ndarray:
    """Tree-ensemble score y [n_hw][B] (higher is better)."""
    hw = np.atleast_2d(np.asarray(hw, dtype=np.float64))
    return np.stack([forest_predict(tree_features(zT, phi_s, hw[j]), feat, thr, leaf, base)
                     for j in range(hw.shape[0])])


def decision_margin(x, feat, thr, n_check=None) -> np.ndarray:
    """Smallest |float32(x[f]) - float32(c)| over the nodes each row visits
    (only nodes testing a feature f < n_check when given): how far the row
    stays from flipping a decision."""
    x32 = np.asarray(x, dtype=np.float64).astype(np.float32)
    feat = np.asarray(feat)
    thr32 = np.asarray(thr, dtype=np.float32)
    NT, n_int = feat.shape
    depth = int(round(np.log2(n_int + 1)))
    B = x32.shape[0]
    rows = np.arange(B)
    m = np.full(B, np.inf)
    for t in range(NT):
        node = np.zeros(B, dtype=np.int64)
        for _ in range(depth):
            f = feat[t, node]
            c = thr32[t, node].astype(np.float64)
            v = x32[rows, f].astype(np.float64)
            gap = np.abs(v - c)
            if n_check is not None:
                gap = np.where(f < n_check, gap, np.inf)
            m = np.minimum(m, gap)
            node = 2 * node + np.where(v < c, 1, 2)
    return m
