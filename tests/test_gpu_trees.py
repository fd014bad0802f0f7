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

from parity_util import TOL, check_topk_self_consistent, latent_rel, to_dev

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


def _certain(ref_zT, g_zT, phi, hw_j, f, d):
    """Candidates whose path through every tree cannot differ between the
    oracle's latents and the GPU's: on the oracle's path each latent
    decision's margin |x_f - c| exceeds the candidate's largest latent
    deviation (the structured features and hardware vectors are exact)."""
    x = np.concatenate([ref_zT, phi, np.broadcast_to(hw_j, (ref_zT.shape[0], hw_j.shape[0]))], axis=1)
    margin = TR.decision_margin(x, f["feat"], f["thr"], n_check=d)
    dev = np.abs(g_zT.astype(np.float32).astype(np.float64) - ref_zT.astype(np.float32)).max(axis=1)
    return margin > dev


def _check_fused(wm, name, prec, B, S, seed, norm="none"):
    """The fused path against the oracle end to end.  z_T within the latent
    tolerance and phi_s against the oracle; the tree kernel exactly on its
    own inputs (above); the fused scores equal to the oracle's exactly for
    every candidate whose tree decisions are beyond its latent deviation
    (trees are discontinuous, so a candidate with a threshold inside that
    deviation may take another leaf), and the top-k equal to the ranking of
    those oracle scores, the other candidates entering with the GPU's
    scores."""
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
    g_z = zT.cpu().numpy().astype(np.float64)
    g_idx = out["idx"].cpu().numpy()
    ref = O.evaluate(W, I, k, prec, norm=norm)
    # parts: latent and structured features against the oracle
    assert latent_rel(g_z, ref["zT"]).max() <= TOL[prec]
    phi_g = torch.empty((B, TR.phi_dim(w.n_kinds, w.n_params)), device="cuda")
    wm.phi_struct(t["types"], t["params"], t["lens"], w.n_kinds, phi_g)
    phi = TR.structured_phi(I["types"], I["params"], I["lens"], w.n_kinds)
    np.testing.assert_allclose(phi_g.cpu().numpy(), phi, rtol=2e-6, atol=2e-6)
    check_topk_self_consistent(g_idx, out["val"].cpu().numpy(), g_sc, I["seg_off"], k)
    # composition: the fused scores are the tree kernel's on the fused path's own inputs
    sc2 = torch.empty_like(sc)
    wm.score_trees(forest, zT, phi_g, t["hw"], sc2)
    np.testing.assert_array_equal(sc2.cpu().numpy(), sc.cpu().numpy())
    # against the oracle end to end
    want = TR.score_trees(ref["zT"], phi, I["hw"], f["feat"], f["thr"], f["leaf"], float(f["base"]))
    atol = 1e-6 * f["feat"].shape[0]               # leaf sums in float32, fixed order
    checked = []
    for j in range(w.n_hw):
        cert = _certain(ref["zT"], g_z, phi, I["hw"][j], f, w.d)
        checked.append(cert.mean())
        np.testing.assert_allclose(g_sc[j, cert], want[j, cert], rtol=0, atol=atol)
        # ranking: oracle scores where the paths are certain, the GPU's elsewhere
        y = np.where(cert, want[j], g_sc[j])
        for s in range(len(I["seg_off"]) - 1):
            lo, hi = I["seg_off"][s], I["seg_off"][s + 1]
            order = lo + np.lexsort((np.arange(hi - lo), -y[lo:hi]))[:k]
            kth = y[order[-1]]
            # the same set up to near-ties (leaf-sum rounding) at the boundary
            diff = set(order.tolist()) ^ set(g_idx[j, s].tolist())
            assert all(abs(y[i] - kth) <= atol for i in diff), f"top-k differs (hw {j}, seg {s})"
    if prec == "fp32":
        assert min(checked) >= 0.5, f"only {min(checked):.3f} of candidates have certain tree paths"
    print(f"[trees fused] {name} {prec} {norm}: scores of {np.mean(checked):.3f} of the candidates "
          f"(those with certain tree paths) equal to the oracle's", flush=True)


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


def test_evaluate_trees_full_size(wm):
    """The benchmark configuration (ansor_round, 2048 candidates, bf16, the
    benchmark's inputs): every candidate against the oracle as above."""
    w = synth.workload("ansor_round")
    _check_fused(wm, "ansor_round", "bf16", w.B, 1, 2000)
