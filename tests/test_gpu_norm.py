"""GPU parity of the paper-form transition (WM_NORM_L2: hyperplane
projection before and unit length after every step, Sec. 3.4) against the
CPU oracle, through the C ABI, in every kernel family that runs it: the
small-batch split kernel, the persistent kernel with 1, 2 and 4 wavefronts
per workgroup, the LDS- and L2-resident forms of the normal map."""
import numpy as np
import pytest

import synth
from oracle import wm_oracle as O

from parity_util import (TOL, check_topk_self_consistent, check_topk_vs_oracle, latent_rel,
                         run_evaluate, score_rel, sub_batch)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def wm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_09312_amd as wm
    wm.load_library()
    return wm


_models = {}


def model_for(wm, name, prec, W=None, tag=""):
    key = (name, prec, tag)
    if key not in _models:
        w = synth.workload(name)
        W = synth.make_weights(w, 1000) if W is None else W
        _models[key] = (wm.Model(wm.model_dims(w), W, precision=prec, norm="l2"), W)
    return _models[key]


def _check_unit(g, lens, z0_of):
    """Outputs of non-empty sequences have unit length; empty ones are z0."""
    n = np.linalg.norm(g["zT"], axis=1)
    pos = lens > 0
    assert np.abs(n[pos] - 1.0).max() <= 1e-5
    np.testing.assert_array_equal(g["zT"][~pos], z0_of[~pos])


# Scaled batches (two 16-candidate tiles per compute unit or fewer): narrow
# tiles at d = 256 and d = 64, the persistent kernel at d = 512
CASES = [
    ("tiny", "fp32", 300, 1),
    ("tiny", "bf16", 300, 1),
    ("ansor_round", "fp32", 300, 1),
    ("ansor_round", "bf16", 300, 1),
    ("ansor_round", "bf16", 5000, 1),
    ("ansor_round", "fp32", 5000, 1),
    ("long_schedule", "bf16", 270, 1),
    ("large_latent", "bf16", 150, 1),
    ("multi_subgraph", "bf16", 4 * 70, 4),
]


@pytest.mark.parametrize("name,prec,B,S", CASES)
def test_l2_parity_scaled(wm, name, prec, B, S):
    base = synth.workload(name)
    w = synth.scaled(base, B=B, S=S)
    k = min(base.k, B // S)
    print(f"[l2 parity] {name} {prec} B={B} S={S} k={k}", flush=True)
    model, W = model_for(wm, name, prec)
    I = synth.make_inputs(w, 3000 + B, pad="garbage")
    I["lens"][:3] = 0                              # empty sequences keep z0
    g = run_evaluate(model, w, I, k)
    assert g["status"] == 0
    ref = O.evaluate(W, I, k, prec, norm="l2")
    tol = TOL[prec]
    rel = latent_rel(g["zT"], ref["zT"])
    assert rel.max() <= tol, f"z_T rel err {rel.max():.3e}"
    srel = score_rel(g["scores"], ref["scores"], I["seg_off"])
    assert srel.max() <= tol, f"score rel err {srel.max():.3e}"
    check_topk_self_consistent(g["idx"], g["val"], g["scores"], I["seg_off"], k)
    check_topk_vs_oracle(g["idx"], ref["scores"], I["seg_off"], k, tol)
    seg_of = O.segment_of(I["seg_off"], w.B)
    if "feats" in I:        # z0 comes from the GPU encoder: compared above, within tolerance
        assert np.abs(np.linalg.norm(g["zT"][I["lens"] > 0], axis=1) - 1.0).max() <= 1e-5
    else:
        _check_unit(g, I["lens"], ref["z0"][seg_of].astype(np.float32).astype(np.float64))
    print(f"  z_T max rel {rel.max():.2e}, score max rel {srel.max():.2e}", flush=True)


# More than 256 tiles of the small model: the persistent kernel with 1 and 2
# wavefronts per workgroup (normal map in LDS), oracle on the whole batch.
@pytest.mark.parametrize("prec,B", [("fp32", 8224), ("bf16", 16448)])
def test_l2_parity_persistent_small_model(wm, prec, B):
    w = synth.scaled(synth.workload("tiny"), B=B)
    print(f"[l2 persistent] tiny {prec} B={B}", flush=True)
    model, W = model_for(wm, "tiny", prec)
    I = synth.make_inputs(w, 41, pad="garbage")
    g = run_evaluate(model, w, I, w.k)
    assert g["status"] == 0
    ref = O.evaluate(W, I, w.k, prec, norm="l2")
    rel = latent_rel(g["zT"], ref["zT"])
    assert rel.max() <= TOL[prec], f"z_T rel err {rel.max():.3e}"
    srel = score_rel(g["scores"], ref["scores"], I["seg_off"])
    assert srel.max() <= TOL[prec], f"score rel err {srel.max():.3e}"
    check_topk_vs_oracle(g["idx"], ref["scores"], I["seg_off"], w.k, TOL[prec])


# Full-size batches in the benchmark's launch configurations; the oracle
# recomputes a sample of candidates one by one.
FULL = [("ansor_round", "fp32"), ("ansor_round", "bf16"), ("long_schedule", "bf16"),
        ("large_latent", "bf16"), ("multi_subgraph", "bf16")]


@pytest.mark.parametrize("name,prec", FULL)
def test_l2_parity_full_size_sampled(wm, name, prec):
    w = synth.workload(name)
    print(f"[l2 full] {name} {prec} B={w.B}", flush=True)
    model, W = model_for(wm, name, prec)
    I = synth.make_inputs(w, 2000)
    g = run_evaluate(model, w, I, w.k)
    assert g["status"] == 0
    check_topk_self_consistent(g["idx"], g["val"], g["scores"], I["seg_off"], w.k)
    assert np.abs(np.linalg.norm(g["zT"], axis=1) - 1.0).max() <= 1e-5
    rng = np.random.default_rng(8)
    order = np.argsort(I["lens"], kind="stable")
    pick = np.unique(np.concatenate([order[:4], order[-4:], rng.choice(w.B, 16, replace=False)]))
    Wd = O.prepare(W, prec)
    z0 = O.encode(Wd, I["feats"], prec) if "feats" in I else I["z0"].astype(np.float64)
    seg_of = O.segment_of(I["seg_off"], w.B)
    sb = sub_batch(I, pick, seg_of, z0)
    zT, phi = O.rollout(Wd, sb["z0"], sb["seg_off"], sb["types"], sb["params"], sb["lens"], prec,
                        norm="l2")
    y = O.score(Wd, zT, phi, I["hw"], prec)
    tol = TOL[prec]
    rel = latent_rel(g["zT"][pick], zT)
    assert rel.max() <= tol, f"z_T rel err {rel.max():.3e}"
    seg_rms = np.array([[np.sqrt(np.mean(g["scores"][j, I["seg_off"][s]:I["seg_off"][s + 1]] ** 2))
                         for s in seg_of[pick]] for j in range(w.n_hw)])
    srel = np.abs(g["scores"][:, pick] - y) / np.maximum(np.abs(y), seg_rms)
    assert srel.max() <= tol, f"score rel err {srel.max():.3e}"
    print(f"  sampled {len(pick)}: z_T max rel {rel.max():.2e}, score max rel {srel.max():.2e}",
          flush=True)


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_l2_zero_normal_map_skips_projection(wm, prec):
    """Wh = 0: every hyperplane normal is zero, the step is the plain residual
    step scaled to unit length (the kernels' zero-normal branch)."""
    base = synth.workload("ansor_round")
    W = dict(synth.make_weights(base, 1000))
    W["wh"] = np.zeros_like(W["wh"])
    model, W = model_for(wm, "ansor_round", prec, W=W, tag="wh0")
    w = synth.scaled(base, B=100)
    I = synth.make_inputs(w, 43)
    g = run_evaluate(model, w, I, 8)
    ref = O.evaluate(W, I, 8, prec, norm="l2")
    assert latent_rel(g["zT"], ref["zT"]).max() <= TOL[prec]


def test_l2_deterministic_and_permutation_invariant(wm):
    w = synth.scaled(synth.workload("ansor_round"), B=500)
    model, W = model_for(wm, "ansor_round", "bf16")
    I = synth.make_inputs(w, 47, pad="garbage")
    a = run_evaluate(model, w, I, 16)
    b = run_evaluate(model, w, I, 16)
    for key in ("zT", "scores", "idx", "val"):
        np.testing.assert_array_equal(a[key], b[key])
    p = np.random.default_rng(2).permutation(w.B)
    Ip = dict(I, types=I["types"][p], params=I["params"][p], lens=I["lens"][p])
    c = run_evaluate(model, w, Ip, 16)
    np.testing.assert_array_equal(c["zT"], a["zT"][p])
