"""Pins for the oracle's paper-form transition (norm="l2": hyperplane
projection before the residual update, unit length after it; Sec. 3.4 with
the TransH construction of Wang et al., AAAI 2014).

Each test names what pins it: a library routine (an SVD null-space basis for
the hyperplane), an invariant (unit length, orthogonality, idempotence), a
special case that reduces to the separately pinned plain transition, a hand
computation on tabulated values of the normal CDF, or the independent scalar
transcription.
"""
import math

import numpy as np
import pytest
from scipy.linalg import null_space

import synth
from oracle import scalar as S
from oracle import wm_oracle as O

PHI1 = 0.8413447460685429          # Phi(1), standard normal table


def _tiny(d=4, e=3, H=5, C=4, hw=2, K=3, P=2, B=8, T=5, S_=1, feat=0, n_hw=1, seed=0,
          len_lo=0):
    w = synth.Workload(name="t", B=B, d=d, e=e, n_kinds=K, n_params=P, H=H, C=C,
                       hw_dim=hw, n_hw=n_hw, k=2, S=S_, feat_dim=feat,
                       enc_hidden=4 if feat else 0, lengths="uniform", len_lo=len_lo,
                       len_hi=T, T_max=T)
    return w, synth.make_weights(w, seed), synth.make_inputs(w, seed + 1, pad="garbage")


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_every_step_has_unit_length_and_empty_sequence_keeps_z0(prec):
    """Invariant: each transition output has Euclidean length 1; finished
    candidates stay frozen; an empty sequence returns z0 itself, unscaled."""
    w, Wt, I = _tiny(B=10, T=6)
    I["z0"] = I["z0"] * 3.0
    I["lens"][0] = 0
    W = O.prepare(Wt, prec)
    zT, phi, traj = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"],
                              prec, trajectory=True, norm="l2")
    for t in range(1, len(traj)):
        act = I["lens"] >= t
        np.testing.assert_allclose(np.linalg.norm(traj[t][act], axis=1), 1.0, rtol=0, atol=1e-14)
        np.testing.assert_array_equal(traj[t][~act], traj[t - 1][~act])
    np.testing.assert_array_equal(zT[0], I["z0"][0])
    # phi does not depend on the transition form
    _, phi_plain = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"], prec)
    np.testing.assert_array_equal(phi, phi_plain)


def test_projection_equals_null_space_projection():
    """W2 = 0, b2 = 0: one step is the unit vector of z0 projected onto the
    hyperplane orthogonal to Wh e (orthonormal hyperplane basis from an SVD,
    scipy.linalg.null_space), and the result is orthogonal to Wh e."""
    w, Wt, I = _tiny(B=6, T=1, len_lo=1)
    Wt = dict(Wt, w2=np.zeros_like(Wt["w2"]), b2=np.zeros_like(Wt["b2"]))
    W = O.prepare(Wt, "fp32")
    zT, _ = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"], "fp32",
                      norm="l2")
    z0 = I["z0"][0].astype(np.float64)
    for i in range(w.B):
        e = O.embed(W, I["types"][i:i + 1, 0], I["params"][i:i + 1, 0])[0]
        v = W["wh"] @ e
        N = null_space(v[None, :])              # d x (d-1), orthonormal columns
        p = N @ (N.T @ z0)
        np.testing.assert_allclose(zT[i], p / np.linalg.norm(p), rtol=0, atol=1e-13)
        assert abs(zT[i] @ v) <= 1e-13 * np.linalg.norm(v)


def test_same_action_twice_is_a_fixed_point():
    """W2 = 0, b2 = 0: projecting twice onto the same hyperplane changes
    nothing (a projection is idempotent), so the second step repeats the first."""
    w, Wt, I = _tiny(B=6, T=2, len_lo=2)
    Wt = dict(Wt, w2=np.zeros_like(Wt["w2"]), b2=np.zeros_like(Wt["b2"]))
    I["types"][:, 1] = I["types"][:, 0]
    I["params"][:, 1] = I["params"][:, 0]
    W = O.prepare(Wt, "fp32")
    _, _, traj = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"], "fp32",
                           trajectory=True, norm="l2")
    np.testing.assert_allclose(traj[2], traj[1], rtol=0, atol=1e-14)


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_zero_normal_map_reduces_to_normalised_plain_step(prec):
    """Wh = 0 (no hyperplane): the step is the plain residual step (pinned on
    its own) scaled to unit length with numpy's vector norm."""
    w, Wt, I = _tiny(B=7, T=1, len_lo=1)
    Wt = dict(Wt, wh=np.zeros_like(Wt["wh"]))
    W = O.prepare(Wt, prec)
    got, _ = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"], prec,
                       norm="l2")
    plain, _ = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"], prec)
    want = plain / np.linalg.norm(plain, axis=1, keepdims=True)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-15)


def _two_dim_weights():
    """d = 2, e = H = K = P = C = hw = 1.  The action embeds to e = 1 (type
    embedding 1, parameter 1 so log2 = 0), its hyperplane normal is Wh e =
    (2, 0), so z0 = (3, 4) projects to (0, 4); W1 [z'; e] = 0.25 * 4 = 1,
    where the normal table gives GELU(1) = Phi(1)."""
    return {
        "type_emb": np.array([[1.0]]), "param_w": np.array([[0.0]]), "param_b": np.array([0.0]),
        "wh": np.array([[2.0], [0.0]]),
        "w1": np.array([[0.0, 0.25, 0.0]]), "b1": np.array([0.0]),
        "w2": np.array([[1.0], [0.0]]), "b2": np.array([0.5, -2.0]),
        "wc1": np.array([[1.0, 0.0, 0.0, 0.0]]), "bc1": np.array([0.0]),
        "wc2": np.array([1.0]), "bc2": np.array(0.0),
    }


@pytest.mark.parametrize("prec,g", [
    ("fp32", PHI1),
    ("bf16", 215.0 / 256.0),     # Phi(1) = 0.84134... rounded to 8 significant bits
])
def test_two_dimensional_hand_computation(prec, g):
    """u = z' + W2 GELU(1) + b2 = (g + 0.5, 4 - 2); z1 = u / |u|."""
    W = O.prepare(_two_dim_weights(), prec)
    zT, phi = O.rollout(W, np.array([[3.0, 4.0]]), [0, 1], np.array([[0]]),
                        np.array([[[1]]]), np.array([1]), prec, norm="l2")
    u = np.array([g + 0.5, 2.0])
    want = u / math.sqrt(u[0] ** 2 + u[1] ** 2)
    np.testing.assert_allclose(zT[0], want, rtol=0, atol=1e-15)
    assert phi[0, 0] == 1.0


def test_degenerate_zero_state_and_zero_normal_stay_finite():
    """z0 along the normal with W2 = 0, b2 = 0 projects to 0 and stays 0 (no
    division by a zero length); an all-zero embedding gives a zero normal and
    no projection."""
    W = O.prepare(dict(_two_dim_weights(), w2=np.zeros((2, 1)), b2=np.zeros(2)), "fp32")
    zT, _ = O.rollout(W, np.array([[5.0, 0.0]]), [0, 1], np.array([[0]]), np.array([[[1]]]),
                      np.array([1]), "fp32", norm="l2")
    np.testing.assert_array_equal(zT, 0.0)
    W = O.prepare(dict(_two_dim_weights(), type_emb=np.array([[0.0]]), w2=np.zeros((2, 1)),
                       b2=np.zeros(2)), "fp32")
    zT, _ = O.rollout(W, np.array([[3.0, 4.0]]), [0, 1], np.array([[0]]), np.array([[[1]]]),
                      np.array([1]), "fp32", norm="l2")
    np.testing.assert_allclose(zT[0], [0.6, 0.8], rtol=0, atol=1e-15)


def test_l2_rollout_is_composition_of_steps():
    w, Wt, I = _tiny(B=9, T=5)
    for prec in ("fp32", "bf16"):
        W = O.prepare(Wt, prec)
        zT, _, traj = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"],
                                prec, trajectory=True, norm="l2")
        for i in range(w.B):
            z = I["z0"][0][None, :].astype(np.float64)
            for t in range(int(I["lens"][i])):
                e = O.embed(W, I["types"][i:i + 1, t], I["params"][i:i + 1, t])
                z = O.transition(W, z, e, prec, norm="l2")
                np.testing.assert_allclose(traj[t + 1][i], z[0], rtol=1e-13, atol=1e-13)
            np.testing.assert_allclose(zT[i], z[0], rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
@pytest.mark.parametrize("shape", [
    dict(d=2, e=1, H=1, C=1, hw=1, K=2, P=1, B=4, T=3),
    dict(d=4, e=3, H=5, C=4, hw=2, K=3, P=2, B=9, T=5),
    dict(d=8, e=8, H=8, C=8, hw=3, K=4, P=3, B=8, T=4, S_=2, feat=6, n_hw=2),
])
def test_l2_vectorised_equals_scalar(prec, shape):
    w, Wt, I = _tiny(**shape, seed=13)
    k = min(3, w.B // w.S)
    a = O.evaluate(Wt, I, k, prec, norm="l2")
    b = S.evaluate(Wt, I, k, prec, norm="l2")
    np.testing.assert_allclose(a["zT"], np.array(b["zT"]), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(a["scores"], np.array(b["scores"]), rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(a["idx"], np.array(b["idx"]))


def test_bf16_rounds_the_normal_map_operands():
    """bf16: the hyperplane normal is R(Wh) R(e) and the projected state is
    rounded as the operand z' of W1 (scalar rounding, SVD projection)."""
    w, Wt, I = _tiny(B=5, T=1, len_lo=1, seed=5)
    Wb = O.prepare(Wt, "bf16")
    Wf = O.prepare(Wt, "fp32")
    z = np.asarray(I["z0"][[0] * 5], dtype=np.float64) * 1.7
    e = O.embed(Wf, I["types"][:, 0] % w.n_kinds, np.abs(I["params"][:, 0]) + 1)
    got = O.transition(Wb, z, e, "bf16", norm="l2")
    r = np.vectorize(S.round_bf16)
    wh, w1, w2 = r(Wt["wh"].astype(np.float64)), r(Wt["w1"].astype(np.float64)), r(Wt["w2"].astype(np.float64))
    for i in range(5):
        N = null_space((wh @ r(e[i]))[None, :])
        zp = N @ (N.T @ z[i])
        x = r(np.concatenate([zp, e[i]]))
        g = r(np.array([S.gelu(float(v)) for v in w1 @ x + Wf["b1"]]))
        u = zp + w2 @ g + Wf["b2"]
        np.testing.assert_allclose(got[i], u / np.linalg.norm(u), rtol=0, atol=1e-13)


def test_unknown_norm_is_rejected():
    w, Wt, I = _tiny(B=2, T=1)
    W = O.prepare(Wt, "fp32")
    with pytest.raises(ValueError):
        O.transition(W, I["z0"][[0, 0]].astype(np.float64), np.zeros((2, w.e)), "fp32", norm="l1")
