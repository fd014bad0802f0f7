"""GPU parity of the structured action features and the tree-ensemble ranker
(the paper's G, Sec. 3.5) against the CPU oracle, through the C ABI: the
feature kernel, the tree kernel on identical float32 features (decisions
must agree exactly), and the fused rollout + features + trees + top-k path
(decisions near a threshold may flip with the rollout's rounding; those
candidates are identified from the oracle's decision margin)."""
import numpy as np
import pytest

import synth
from oracle import trees as TR
from oracle import wm_oracle as O

from parity_util import TOL, check_topk_self_consistent, latent_rel, sub_batch, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def wm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_09312_amd as wm
    wm.load_library()
    return wm


def _forest(wm, w, seed, **kw):
    f = synth.make_forest(w, seed, **kw)
    n_feat = w.d + TR.phi_dim(w.n_kinds, w.n_params) + w.hw_dim
    return wm.Forest(f["feat"], f["thr"], f["leaf"], float(f["base"]), n_feat), f


@pytest.mark.parametrize("T_max,len_lo", [(32, 0), (100, 60)])
def test_phi_struct_matches_oracle(wm, T_max, len_lo):
    w = synth.scaled(synth.workload("ansor_round"), B=333, len_lo=len_lo, len_hi=T_max, T_max=T_max)
    I = synth.make_inputs(w, 61, pad="garbage")
    I["lens"][:4] = 0
    t = to_dev(I, "cuda")
    out = torch.empty((w.B, TR.phi_dim(w.n_kinds, w.n_params)), device="cuda")
    wm.phi_struct(t["types"], t["params"], t["lens"], w.n_kinds, out)
    got = out.cpu().numpy().astype(np.float64)
    want = TR.structured_phi(I["types"], I["params"], I["lens"], w.n_kinds)
    K = w.n_kinds
    np.testing.assert_array_equal(got[:, :K + 1], want[:, :K + 1])      # counts and length exact
    np.testing.assert_allclose(got[:, K + 1:], want[:, K + 1:], rtol=2e-6, atol=2e-6)


@pytest.mark.parametrize("n_trees,depth", [(256, 8), (300, 6), (5, 1), (64, 12)])
def test_score_trees_exact_decisions(wm, n_trees, depth):
    """Identical float32 features on both sides: every decision agrees, so
    the scores differ only by the order of the float32 leaf sum."""
    w = synth.workload("ansor_round")
    forest, f = _forest(wm, w, 5 + depth, n_trees=n_trees, depth=depth)
    rng = np.random.default_rng(depth)
    B = 257
    zT = rng.standard_normal((B, w.d)).astype(np.float32)
    I = synth.make_inputs(synth.scaled(w, B=B), 63)
    phi = TR.structured_phi(I["types"], I["params"], I["lens"], w.n_kinds).astype(np.float32)
    zT[0, :] = f["thr"][0, 0]                      # features sitting exactly on thresholds
    hw = rng.standard_normal((2, w.hw_dim)).astype(np.float32)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    sc = torch.empty((2, B), device="cuda")
    wm.score_trees(forest, d(zT), d(phi), d(hw), sc)
    got = sc.cpu().numpy().astype(np.float64)
    want = TR.score_trees(zT, phi, hw, f["feat"], f["thr"], f["leaf"], float(f["base"]))
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-6 * n_trees)


def _check_fused(wm, name, prec, B, S, seed, norm="none"):
    """The fused path equals the composition of its parts, each checked on
    its own: z_T against the oracle within the latent tolerance, phi_s
    against the oracle, the tree kernel exactly (see above).  Trees are
    discontinuous, so a latent rounding difference can move a candidate to
    another leaf; in fp32 that must stay rare."""
    base = synth.workload(name)
    w = synth.scaled(base, B=B, S=S)
    k = min(base.k, B // S)
    W = synth.make_weights(base, 1000)
    model = wm.Model(wm.model_dims(base), W, precision=prec, norm=norm)
    forest, f = _forest(wm, base, 77, z_scale=0.05 if norm == "l2" else 1.0)
    I = synth.make_inputs(w, seed, pad="garbage")
    t = to_dev(I, "cuda")
    init = t["feats"] if "feats" in t else t["z0"]
    sc = torch.empty((w.n_hw, B), device="cuda")
    zT = torch.empty((B, w.d), device="cuda")
    out = wm.evaluate(model, init, I["seg_off"], t["types"], t["params"], t["lens"], t["hw"], k,
                      init_is_feats="feats" in t, scores=sc, zT=zT, forest=forest)
    wm.device_status(out["ws"])
    g_sc = sc.cpu().numpy().astype(np.float64)
    ref = O.evaluate(W, I, k, prec, norm=norm)
    # parts: latent and structured features against the oracle
    assert latent_rel(zT.cpu().numpy().astype(np.float64), ref["zT"]).max() <= TOL[prec]
    phi_g = torch.empty((B, TR.phi_dim(w.n_kinds, w.n_params)), device="cuda")
    wm.phi_struct(t["types"], t["params"], t["lens"], w.n_kinds, phi_g)
    phi = TR.structured_phi(I["types"], I["params"], I["lens"], w.n_kinds)
    np.testing.assert_allclose(phi_g.cpu().numpy(), phi, rtol=2e-6, atol=2e-6)
    # composition: the fused scores are the tree kernel's on the fused path's own inputs
    sc2 = torch.empty_like(sc)
    wm.score_trees(forest, zT, phi_g, t["hw"], sc2)
    np.testing.assert_array_equal(sc2.cpu().numpy(), sc.cpu().numpy())
    check_topk_self_consistent(out["idx"].cpu().numpy(), out["val"].cpu().numpy(), g_sc,
                               I["seg_off"], k)
    # against the oracle end to end
    want = TR.score_trees(ref["zT"], phi, I["hw"], f["feat"], f["thr"], f["leaf"], float(f["base"]))
    same = np.abs(g_sc - want) <= 1e-6 * f["feat"].shape[0]
    if prec == "fp32":
        assert same.mean() >= 0.95, f"only {same.mean():.3f} of scores agree with the oracle"
    print(f"[trees fused] {name} {prec} {norm}: {same.mean():.3f} of scores equal to the oracle's",
          flush=True)


@pytest.mark.parametrize("name,prec,B,S,norm", [
    ("tiny", "fp32", 300, 1, "none"),
    ("ansor_round", "fp32", 300, 1, "none"),
    ("ansor_round", "bf16", 300, 1, "none"),
    ("ansor_round", "fp32", 300, 1, "l2"),
    ("multi_subgraph", "bf16", 4 * 70, 4, "none"),
    ("large_latent", "bf16", 150, 1, "none"),
])
def test_evaluate_trees_matches_oracle(wm, name, prec, B, S, norm):
    _check_fused(wm, name, prec, B, S, 3100 + B, norm)


def test_evaluate_trees_full_size_sampled(wm):
    """The benchmark configuration: all candidates ranked on the GPU; the
    fused scores equal the tree kernel's on the fused path's own latents, and
    a sample of latents is recomputed by the oracle."""
    w = synth.workload("ansor_round")
    W = synth.make_weights(w, 1000)
    model = wm.Model(wm.model_dims(w), W, precision="bf16")
    forest, f = _forest(wm, w, 77)
    I = synth.make_inputs(w, 2000)
    t = to_dev(I, "cuda")
    sc = torch.empty((1, w.B), device="cuda")
    zT = torch.empty((w.B, w.d), device="cuda")
    out = wm.evaluate(model, t["z0"], I["seg_off"], t["types"], t["params"], t["lens"], t["hw"],
                      w.k, scores=sc, zT=zT, forest=forest)
    wm.device_status(out["ws"])
    g_sc = sc.cpu().numpy().astype(np.float64)
    check_topk_self_consistent(out["idx"].cpu().numpy(), out["val"].cpu().numpy(), g_sc,
                               I["seg_off"], w.k)
    phi_g = torch.empty((w.B, TR.phi_dim(w.n_kinds, w.n_params)), device="cuda")
    wm.phi_struct(t["types"], t["params"], t["lens"], w.n_kinds, phi_g)
    sc2 = torch.empty_like(sc)
    wm.score_trees(forest, zT, phi_g, t["hw"], sc2)
    np.testing.assert_array_equal(sc2.cpu().numpy(), sc.cpu().numpy())
    pick = np.random.default_rng(9).choice(w.B, 24, replace=False)
    Wd = O.prepare(W, "bf16")
    sb = sub_batch(I, pick, O.segment_of(I["seg_off"], w.B), I["z0"].astype(np.float64))
    zr, _ = O.rollout(Wd, sb["z0"], sb["seg_off"], sb["types"], sb["params"], sb["lens"], "bf16")
    assert latent_rel(zT.cpu().numpy()[pick].astype(np.float64), zr).max() <= TOL["bf16"]
    phi = TR.structured_phi(I["types"], I["params"], I["lens"], w.n_kinds)
    np.testing.assert_allclose(phi_g.cpu().numpy(), phi, rtol=2e-6, atol=2e-6)
