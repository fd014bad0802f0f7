"""Pins for the CPU oracle: checks against facts fixed outside the oracle.

Each test states what pins it: a textbook value, a closed form, a library
routine, a brute-force search, or the independent scalar transcription.
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import scalar as S
from oracle import wm_oracle as O

GOLDEN = __file__.rsplit("/", 1)[0] + "/golden"


def _load_cdf():
    rows = []
    with open(GOLDEN + "/normal_cdf.txt") as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                x, p = line.split()
                rows.append((float(x), float(p)))
    return rows


# ----------------------------------------------------------------------------
# bfloat16 rounding R


def _torch_bf16(x32):
    """Library reference: PyTorch's float32 -> bfloat16 conversion (RNE)."""
    t = torch.from_numpy(np.ascontiguousarray(x32, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float64).numpy()


def test_bf16_round_matches_library_conversion():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
        rng.standard_normal(2000) * 1e-39,                 # subnormal range
    ]).astype(np.float32)
    # exact halfway cases: bf16 value + half a spacing, both parities
    base = rng.standard_normal(5000).astype(np.float32)
    bits = base.view(np.uint32) & np.uint32(0xFFFF0000)
    ties = (bits | np.uint32(0x8000)).view(np.float32)
    x = np.concatenate([x, ties, np.float32([0.0, -0.0, 1.0, -2.5])])
    ref = _torch_bf16(x)
    got = O.bf16_round(x.astype(np.float64))
    np.testing.assert_array_equal(got, ref)
    got2 = np.array([S.round_bf16(float(v)) for v in x[:3000]])
    np.testing.assert_array_equal(got2, ref[:3000])


@pytest.mark.parametrize("x,want", [
    (1.0 + 2.0 ** -8, 1.0),                  # tie -> even mantissa
    (1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -6),  # tie -> even mantissa (upwards)
    (math.pi, 3.140625),
    (0.1, 0.10009765625),
    (2.2826894921370859, 2.28125),
    (-1.0 - 2.0 ** -9, -1.0),
])
def test_bf16_round_hand_values(x, want):
    assert O.bf16_round(x) == want
    assert S.round_bf16(x) == want


# ----------------------------------------------------------------------------
# GELU


def test_gelu_textbook_normal_cdf():
    """GELU(x) = x * Phi(x); Phi from a printed standard normal table."""
    for x, p in _load_cdf():
        assert O.gelu(x) == pytest.approx(x * p, rel=1e-10, abs=1e-12)
        assert S.gelu(x) == pytest.approx(x * p, rel=1e-10, abs=1e-12)
        assert O.gelu(-x) == pytest.approx(-x * (1.0 - p), rel=1e-9, abs=1e-12)


def test_gelu_identities():
    x = np.linspace(-12, 12, 4001)
    g = O.gelu(x)
    # GELU(x) - GELU(-x) = x  (Phi(x) + Phi(-x) = 1)
    assert np.all(np.abs((g - O.gelu(-x)) - x) <= 4e-15 * np.maximum(1, np.abs(x)))
    assert O.gelu(0.0) == 0.0
    np.testing.assert_allclose(O.gelu(np.array([40.0, -40.0])), [40.0, 0.0], atol=1e-300)


# ----------------------------------------------------------------------------
# Embedding, transition, rollout


def _tiny(d=3, e=2, H=4, C=5, hw=2, K=3, P=2, B=6, T=4, S_=1, feat=0, n_hw=1, seed=0):
    w = synth.Workload(name="t", B=B, d=d, e=e, n_kinds=K, n_params=P, H=H, C=C,
                       hw_dim=hw, n_hw=n_hw, k=2, S=S_, feat_dim=feat,
                       enc_hidden=4 if feat else 0, lengths="uniform", len_lo=0,
                       len_hi=T, T_max=T)
    return w, synth.make_weights(w, seed), synth.make_inputs(w, seed + 1, pad="garbage")


def test_embed_closed_forms():
    w, Wt, _ = _tiny()
    W = O.prepare(Wt, "fp32")
    types = np.array([0, 1, 2])
    ones = np.ones((3, w.n_params), dtype=np.int32)
    np.testing.assert_array_equal(O.embed(W, types, ones), W["type_emb"][types] + W["param_b"])
    pw2 = np.array([[4, 1], [1, 1024], [8, 2]], dtype=np.int32)   # log2 -> integers
    u = np.array([[2, 0], [0, 10], [3, 1]], dtype=np.float64)
    want = W["type_emb"][types] + np.stack([W["param_w"] @ r for r in u]) + W["param_b"]
    np.testing.assert_allclose(O.embed(W, types, pw2), want, rtol=1e-15, atol=1e-15)


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_transition_identity_when_output_layer_zero(prec):
    w, Wt, I = _tiny(T=5)
    Wt = dict(Wt, w2=np.zeros_like(Wt["w2"]), b2=np.zeros_like(Wt["b2"]))
    W = O.prepare(Wt, prec)
    zT, _ = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"], prec)
    np.testing.assert_array_equal(zT, np.broadcast_to(I["z0"][0].astype(np.float64), zT.shape))


def test_transition_closed_form_when_input_layer_zero():
    """W1 = 0: every step adds the same vector W2 GELU(b1) + b2."""
    w, Wt, I = _tiny(T=6)
    Wt = dict(Wt, w1=np.zeros_like(Wt["w1"]))
    W = O.prepare(Wt, "fp32")
    zT, _ = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"], "fp32")
    step = W["w2"] @ np.array([S.gelu(float(v)) for v in W["b1"]]) + W["b2"]
    want = I["z0"][0][None, :] + I["lens"][:, None] * step[None, :]
    np.testing.assert_allclose(zT, want, rtol=1e-13, atol=1e-13)


def _one_dim_weights():
    """d = e = H = C = P = 1, two action kinds; chosen so GELU arguments are
    exactly 1 and 2 where the normal table gives Phi."""
    phi1 = 0.8413447460685429
    z1 = 0.5 + 2.0 * 1.0 * phi1 - 1.0
    return {
        "type_emb": np.array([[0.25], [0.5]]), "param_w": np.array([[0.125]]),
        "param_b": np.array([0.0]), "w1": np.array([[1.0, 1.0]]), "b1": np.array([0.0]),
        "w2": np.array([[2.0]]), "b2": np.array([-1.0]),
        "wc1": np.array([[1.0, 0.0, 0.0]]), "bc1": np.array([2.0 - z1]),
        "wc2": np.array([3.0]), "bc2": np.array(0.25),
    }, z1


def test_one_dimensional_hand_computation():
    """One step by hand: e = 0.25 + 0.125 log2(4) = 0.5; W1 [z; e] = 1;
    z1 = 0.5 + 2 Phi(1) - 1; score argument 2 so y = 3 * 2 Phi(2) + 0.25."""
    Wt, z1 = _one_dim_weights()
    phi2 = 0.9772498680518208
    W = O.prepare(Wt, "fp32")
    types = np.array([[0, 1]]); params = np.array([[[4], [1]]]); lens = np.array([1])
    zT, phi = O.rollout(W, np.array([[0.5]]), [0, 1], types, params, lens, "fp32")
    assert zT[0, 0] == pytest.approx(z1, rel=1e-14)
    assert phi[0, 0] == 0.5
    y = O.score(W, zT, phi, np.array([[7.0]]), "fp32")
    assert y[0, 0] == pytest.approx(3.0 * 2.0 * phi2 + 0.25, rel=1e-12)
    # second step: type 1, param 1 -> e = 0.5; argument z1 + 0.5
    zT2, phi2v = O.rollout(W, np.array([[0.5]]), [0, 1], types, params, np.array([2]), "fp32")
    a = z1 + 0.5
    want = z1 + 2.0 * a * 0.5 * (1 + math.erf(a / math.sqrt(2))) - 1.0
    assert zT2[0, 0] == pytest.approx(want, rel=1e-14)
    assert phi2v[0, 0] == 0.5


def test_rollout_is_composition_of_steps_and_prefix_consistent():
    w, Wt, I = _tiny(T=5, B=12)
    for prec in ("fp32", "bf16"):
        W = O.prepare(Wt, prec)
        zT, phi, traj = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"],
                                  I["lens"], prec, trajectory=True)
        for i in range(w.B):
            z = I["z0"][0][None, :].astype(np.float64)
            for t in range(int(I["lens"][i])):
                e = O.embed(W, I["types"][i:i + 1, t], I["params"][i:i + 1, t])
                z = O.transition(W, z, e, prec)
                # prefix state (BLAS may round a 1-row product differently: 1e-13)
                np.testing.assert_allclose(traj[t + 1][i], z[0], rtol=1e-13, atol=1e-13)
            np.testing.assert_allclose(zT[i], z[0], rtol=1e-13, atol=1e-13)


def test_zero_length_returns_initial_state_and_zero_phi():
    w, Wt, I = _tiny(T=4, B=8)
    I["lens"][:] = 0
    W = O.prepare(Wt, "bf16")
    zT, phi = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"], "bf16")
    np.testing.assert_array_equal(zT, np.broadcast_to(I["z0"][0], zT.shape))
    np.testing.assert_array_equal(phi, 0.0)


def test_padding_is_never_read():
    w, Wt, I = _tiny(T=6, B=10)
    W = O.prepare(Wt, "fp32")
    a = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"], "fp32")
    t2, p2 = I["types"].copy(), I["params"].copy()
    pad = np.arange(w.T_max)[None, :] >= I["lens"][:, None]
    t2[pad] = 12345
    p2[pad] = -7
    b = O.rollout(W, I["z0"], I["seg_off"], t2, p2, I["lens"], "fp32")
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    assert O.validate({"n_kinds": w.n_kinds}, B=w.B, T_max=w.T_max, seg_off=I["seg_off"],
                      types=t2, params=p2, lens=I["lens"]) == O.OK


# ----------------------------------------------------------------------------
# Score and ranking


def test_score_permutation_equivariant_and_batch_split():
    w, Wt, I = _tiny(B=16, T=5)
    for prec in ("fp32", "bf16"):
        W = O.prepare(Wt, prec)
        zT, phi = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"], prec)
        y = O.score(W, zT, phi, I["hw"], prec)
        p = np.random.default_rng(3).permutation(w.B)
        np.testing.assert_allclose(O.score(W, zT[p], phi[p], I["hw"], prec), y[:, p],
                                   rtol=1e-13, atol=1e-13)
        y_a = O.score(W, zT[:7], phi[:7], I["hw"], prec)
        np.testing.assert_allclose(y_a, y[:, :7], rtol=1e-13, atol=1e-13)


def test_score_constant_when_cost_input_layer_zero():
    w, Wt, I = _tiny(B=5)
    Wt = dict(Wt, wc1=np.zeros_like(Wt["wc1"]))
    W = O.prepare(Wt, "fp32")
    zT, phi = O.rollout(W, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"], "fp32")
    y = O.score(W, zT, phi, I["hw"], "fp32")
    want = sum(float(W["wc2"][r]) * S.gelu(float(W["bc1"][r])) for r in range(w.C)) + float(W["bc2"])
    np.testing.assert_allclose(y, want, rtol=1e-14)


def test_topk_matches_brute_force_sort():
    rng = np.random.default_rng(5)
    y = np.round(rng.standard_normal((2, 60)), 1)        # many exact ties
    seg_off = np.array([0, 13, 40, 60])
    idx, val = O.topk(y, seg_off, 13)
    for j in range(2):
        for s in range(3):
            lo, hi = seg_off[s], seg_off[s + 1]
            brute = sorted(range(lo, hi), key=lambda i: (-y[j, i], i))[:13]
            assert list(idx[j, s]) == brute
            np.testing.assert_array_equal(val[j, s], y[j, brute])


def test_topk_duplicates_nan_and_full_segment():
    y = np.array([[1.0, 3.0, 3.0, np.nan, -0.0, 0.0, 3.0, -np.inf, np.inf]])
    idx, val = O.topk(y, [0, 9], 9)
    # +inf first, ties to the lower index, -0 == +0, -inf before NaN (last)
    assert list(idx[0, 0]) == [8, 1, 2, 6, 0, 4, 5, 7, 3]


# ----------------------------------------------------------------------------
# Encoder


def test_encoder_closed_form_when_input_layer_zero():
    w, Wt, I = _tiny(feat=5, S_=2, B=4)
    Wt = dict(Wt, we1=np.zeros_like(Wt["we1"]))
    for prec in ("fp32", "bf16"):
        W = O.prepare(Wt, prec)
        z0 = O.encode(W, I["feats"], prec)
        hid = np.array([S.gelu(float(v)) for v in W["be1"]])
        if prec == "bf16":
            hid = np.array([S.round_bf16(v) for v in hid])
        want = W["we2"] @ hid + W["be2"]
        np.testing.assert_allclose(z0, np.stack([want, want]), rtol=1e-14)


# ----------------------------------------------------------------------------
# Vectorised oracle == independent scalar transcription


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
@pytest.mark.parametrize("shape", [
    dict(d=1, e=1, H=1, C=1, hw=1, K=2, P=1, B=4, T=3),
    dict(d=3, e=2, H=4, C=5, hw=2, K=3, P=2, B=9, T=5),
    dict(d=8, e=8, H=8, C=8, hw=3, K=4, P=3, B=8, T=4, S_=2, feat=6, n_hw=2),
])
def test_vectorised_equals_scalar(prec, shape):
    w, Wt, I = _tiny(**shape, seed=11)
    k = min(3, w.B // w.S)
    a = O.evaluate(Wt, I, k, prec)
    b = S.evaluate(Wt, I, k, prec)
    np.testing.assert_allclose(a["zT"], np.array(b["zT"]), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(a["phi"], np.array(b["phi"]), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(a["scores"], np.array(b["scores"]), rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(a["idx"], np.array(b["idx"]))


def test_bf16_mode_rounds_transition_operands():
    """In bf16 mode the step result equals the fp32-mode step on pre-rounded
    operands: R applied to W1, W2, [z; e] and GELU output (a planted missing
    rounding on any of them changes this)."""
    w, Wt, I = _tiny(B=6, T=1, seed=4)
    Wb = O.prepare(Wt, "bf16")
    Wf = O.prepare(Wt, "fp32")
    z = np.asarray(I["z0"][[0] * 6], dtype=np.float64) * 3.1
    e = O.embed(Wf, I["types"][:, 0] % w.n_kinds, np.abs(I["params"][:, 0]) + 1)
    got = O.transition(Wb, z, e, "bf16")
    x = np.array([[S.round_bf16(float(v)) for v in row] for row in np.concatenate([z, e], 1)])
    w1 = np.array([[S.round_bf16(float(v)) for v in r] for r in Wt["w1"]])
    w2 = np.array([[S.round_bf16(float(v)) for v in r] for r in Wt["w2"]])
    g = np.array([[S.round_bf16(S.gelu(float(v))) for v in row] for row in x @ w1.T + Wf["b1"]])
    want = z + (g @ w2.T + Wf["b2"])
    np.testing.assert_allclose(got, want, rtol=1e-14, atol=1e-14)


# ----------------------------------------------------------------------------
# Validation statuses


def test_validate_statuses():
    w, Wt, I = _tiny(B=8, T=4)
    dims = {"n_kinds": w.n_kinds}
    kw = dict(B=w.B, T_max=w.T_max, types=I["types"], params=I["params"])
    assert O.validate(dims, seg_off=[0, 8], lens=I["lens"], k=2, n_hw=1, **kw) == O.OK
    assert O.validate(dims, seg_off=[0, 7], lens=I["lens"], **kw) == O.ERR_INVALID_ARGUMENT
    assert O.validate(dims, seg_off=[0, 5, 3, 8], lens=I["lens"], **kw) == O.ERR_INVALID_ARGUMENT
    assert O.validate(dims, seg_off=[0, 8], k=9, lens=I["lens"], **kw) == O.ERR_INVALID_ARGUMENT
    assert O.validate(dims, seg_off=[0, 8], k=0, lens=I["lens"], **kw) == O.ERR_INVALID_ARGUMENT
    assert O.validate(dims, seg_off=[0, 8], n_hw=0, lens=I["lens"], **kw) == O.ERR_INVALID_ARGUMENT
    bad = I["lens"].copy(); bad[3] = w.T_max + 1
    assert O.validate(dims, seg_off=[0, 8], lens=bad, **kw) == O.ERR_INPUT_RANGE
    L = I["lens"].copy(); L[2] = 2
    t0 = I["types"].copy(); t0[2, :2] = 0
    p0 = I["params"].copy(); p0[2, :2] = 1
    assert O.validate(dims, seg_off=[0, 8], lens=L, B=8, T_max=4, types=t0, params=p0) == O.OK
    t = t0.copy(); t[2, 1] = w.n_kinds
    assert O.validate(dims, seg_off=[0, 8], lens=L, B=8, T_max=4, types=t, params=p0) == O.ERR_INPUT_RANGE
    t = t0.copy(); t[2, 1] = -1
    assert O.validate(dims, seg_off=[0, 8], lens=L, B=8, T_max=4, types=t, params=p0) == O.ERR_INPUT_RANGE
    p = p0.copy(); p[2, 1, 0] = 0
    assert O.validate(dims, seg_off=[0, 8], lens=L, B=8, T_max=4, types=t0, params=p) == O.ERR_INPUT_RANGE
    t = t0.copy(); t[2, 2] = 99     # step 2 is padding for candidate 2: not inspected
    assert O.validate(dims, seg_off=[0, 8], lens=L, B=8, T_max=4, types=t, params=p0) == O.OK
