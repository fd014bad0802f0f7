"""Pins for the oracle of the structured action features and the
tree-ensemble ranker (Sec. 3.5): scikit-learn's decision-tree inference,
hand-built stumps (ties, NaN), hand-computed feature vectors."""
import numpy as np
import pytest
from sklearn.tree import DecisionTreeRegressor

import synth
from oracle import trees as T


def _complete_from_sklearn(tree, depth):
    """Convert a fitted sklearn tree (x <= threshold goes left) to the
    complete breadth-first layout (float32 x < c goes left).  A leaf above the
    last level becomes a subtree whose nodes always go left and whose leaves
    all carry its value."""
    t = tree.tree_
    n_int = 2 ** depth - 1
    feat = np.zeros(n_int, np.int32)
    thr = np.full(n_int, np.inf, np.float32)
    leaf = np.zeros(n_int + 1, np.float32)

    def fill(sk, pos, level, const=None):
        if level == depth:
            leaf[pos - n_int] = const if const is not None else t.value[sk].ravel()[0]
            return
        if const is None and t.children_left[sk] == -1:
            const = t.value[sk].ravel()[0]
        if const is not None:
            feat[pos], thr[pos] = 0, np.inf
            fill(sk, 2 * pos + 1, level + 1, const)
            fill(sk, 2 * pos + 2, level + 1, const)
            return
        c = np.float32(t.threshold[sk])
        if float(c) <= t.threshold[sk]:            # smallest float32 above the threshold
            c = np.nextafter(c, np.float32(np.inf))
        feat[pos], thr[pos] = t.feature[sk], c
        fill(t.children_left[sk], 2 * pos + 1, level + 1)
        fill(t.children_right[sk], 2 * pos + 2, level + 1)

    fill(0, 0, 0)
    return feat, thr, leaf


@pytest.mark.parametrize("depth", [1, 3, 6])
def test_forest_matches_sklearn_tree_inference(depth):
    rng = np.random.default_rng(depth)
    X = rng.standard_normal((400, 7)).astype(np.float32)
    X[:, 3] = np.round(X[:, 3], 1)                 # repeated values: thresholds between ties
    models = []
    for k in range(4):
        y = np.sin(X[:, k]) + X[:, (k + 3) % 7] ** 2 + 0.1 * rng.standard_normal(len(X))
        models.append(DecisionTreeRegressor(max_depth=depth, random_state=k).fit(X, y))
    conv = [_complete_from_sklearn(m, depth) for m in models]
    feat, thr, leaf = (np.stack([c[i] for c in conv]) for i in range(3))
    Xt = rng.standard_normal((300, 7)).astype(np.float32)
    Xt[:50] = X[:50]                               # rows that sit on training values
    for data in (X, Xt):
        want = sum(m.predict(data) for m in models)
        got = T.forest_predict(data, feat, thr, leaf, 0.0)
        np.testing.assert_allclose(got, want, rtol=1e-6, atol=1e-6)


def test_stump_by_hand_ties_and_nan():
    feat = np.array([[2]], np.int32)
    thr = np.array([[0.5]], np.float32)
    leaf = np.array([[-1.0, 3.0]], np.float32)
    x = np.array([[9, 9, 0.25, 9], [9, 9, 0.5, 9], [9, 9, 0.75, 9], [9, 9, np.nan, 9]])
    got = T.forest_predict(x, feat, thr, leaf, 0.5)
    np.testing.assert_array_equal(got, [-0.5, 3.5, 3.5, 3.5])     # tie and NaN go right
    m = T.decision_margin(x, feat, thr)
    assert m[1] == 0.0 and m[0] == pytest.approx(0.25)
    assert np.all(T.decision_margin(x, feat, thr, n_check=2) == np.inf)   # feature 2 not checked


def test_depth_two_paths_by_hand():
    # node 0: x0 < 0 ; node 1 (left): x1 < 1 ; node 2 (right): x2 < -1
    feat = np.array([[0, 1, 2]], np.int32)
    thr = np.array([[0.0, 1.0, -1.0]], np.float32)
    leaf = np.array([[10.0, 20.0, 30.0, 40.0]], np.float32)
    x = np.array([[-1, 0, 0], [-1, 2, 0], [1, 0, -2], [1, 0, 0]], np.float64)
    np.testing.assert_array_equal(T.forest_predict(x, feat, thr, leaf, 0.0), [10, 20, 30, 40])


def test_float32_decisions():
    """A feature that differs from the threshold only below float32
    resolution compares equal in float32 and goes right."""
    feat = np.array([[0]], np.int32)
    thr = np.array([[1.0]], np.float32)
    leaf = np.array([[0.0, 1.0]], np.float32)
    x = np.array([[1.0 - 1e-12], [1.0 - 1e-6]])
    np.testing.assert_array_equal(T.forest_predict(x, feat, thr, leaf, 0.0), [1.0, 0.0])


def test_structured_phi_by_hand():
    types = np.array([[0, 2, 2, 1, 7, 7], [1, 1, -5, -5, -5, -5], [0, 0, 0, 0, 0, 0]])
    params = np.array([
        [[1, 8], [4, 2], [16, 2], [2, 1], [0, 0], [-3, 99]],
        [[1024, 1], [2, 512], [0, 0], [0, 0], [0, 0], [0, 0]],
        [[0, 0]] * 6,
    ])
    lens = np.array([4, 2, 0])
    phi = T.structured_phi(types, params, lens, n_kinds=3)
    # counts (3), length, mean log2 per slot, max log2 per slot
    np.testing.assert_array_equal(phi[0], [1, 1, 2, 4, (0 + 2 + 4 + 1) / 4, (3 + 1 + 1 + 0) / 4, 4, 3])
    np.testing.assert_array_equal(phi[1], [0, 2, 0, 2, (10 + 1) / 2, (0 + 9) / 2, 10, 9])
    np.testing.assert_array_equal(phi[2], 0.0)
    assert T.phi_dim(3, 2) == 8


def test_forest_generator_shapes_and_features():
    w = synth.workload("ansor_round")
    f = synth.make_forest(w, 3, n_trees=5, depth=4)
    assert f["feat"].shape == (5, 15) and f["leaf"].shape == (5, 16)
    assert f["feat"].min() >= 0 and f["feat"].max() < w.d + T.phi_dim(w.n_kinds, w.n_params) + w.hw_dim
