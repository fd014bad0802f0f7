"""The allocation-free entry point (wm_evaluate_noalloc) against wm_evaluate
on the same inputs: two calls in a row on one GPU, the second with a smaller
batch (the scratch keeps the first call's contents), with and without the
initial-latent encoder.  Both run the same kernels in the same order, so the
outputs are compared bit for bit."""
import numpy as np
import pytest

import synth

from parity_util import to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def wm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_09312_amd as wm
    wm.load_library()
    return wm


@pytest.mark.parametrize("name,prec,sizes", [
    ("ansor_round", "bf16", [(12000, 1), (3000, 1)]),      # persistent kernel, then narrow tiles
    ("multi_subgraph", "bf16", [(32 * 200, 32), (8 * 100, 8)]),   # encoder into the scratch
])
def test_noalloc_matches_evaluate(wm, name, prec, sizes):
    base = synth.workload(name)
    W = synth.make_weights(base, 1000)
    model = wm.Model(wm.model_dims(base), W, precision=prec)
    dev = torch.device("cuda")
    for call, (B, S) in enumerate(sizes):
        w = synth.scaled(base, B=B, S=S)
        k = min(base.k, B // S)
        print(f"[noalloc] {name} {prec} call {call}: B={B} S={S}", flush=True)
        I = synth.make_inputs(w, 4100 + call)
        t = to_dev(I, dev)
        feats = "feats" in t
        init = t["feats"] if feats else t["z0"]
        n_hw = w.n_hw
        ref_sc = torch.empty((n_hw, B), device=dev)
        ref_z = torch.empty((B, w.d), device=dev)
        ref = wm.evaluate(model, init, I["seg_off"], t["types"], t["params"], t["lens"], t["hw"], k,
                          init_is_feats=feats, scores=ref_sc, zT=ref_z)
        wm.device_status(ref["ws"])
        sc = torch.full((n_hw, B), float("nan"), device=dev)
        z = torch.full((B, w.d), float("nan"), device=dev)
        phi = torch.empty((B, w.e), device=dev)
        idx = torch.empty((n_hw, S, k), dtype=torch.int32, device=dev)
        val = torch.empty((n_hw, S, k), device=dev)
        status = torch.full((64,), -1, dtype=torch.int32, device=dev)   # cleared by the call
        wm.evaluate_noalloc(model, init, I["seg_off"], t["types"], t["params"], t["lens"], t["hw"], k,
                            scores=sc, zT=z, phi=phi, idx=idx, val=val, status=status,
                            init_is_feats=feats)
        wm.device_status(status)
        torch.cuda.synchronize()
        assert torch.equal(z, ref_z), "z_T differs"
        assert torch.equal(sc, ref_sc), "scores differ"
        assert torch.equal(idx, ref["idx"]), "top-k indices differ"
        assert torch.equal(val, ref["val"]), "top-k values differ"
        # phi: the mean step embedding (finite, zero for empty sequences)
        assert torch.isfinite(phi).all()


def test_noalloc_rejects_oversized_batches(wm):
    base = synth.workload("ansor_round")
    W = synth.make_weights(base, 1000)
    model = wm.Model(wm.model_dims(base), W, precision="bf16")
    B = (4 << 20) // 8 + 1           # the permutation alone exceeds the scratch
    dev = torch.device("cuda")
    types = torch.zeros((B, 1), dtype=torch.int32, device=dev)
    with pytest.raises(wm.WMError) as e:
        wm.evaluate_noalloc(model, torch.zeros((1, base.d), device=dev), np.array([0, B], np.int32),
                            types, torch.ones((B, 1, base.n_params), dtype=torch.int32, device=dev),
                            torch.zeros(B, dtype=torch.int32, device=dev),
                            torch.zeros((1, base.hw_dim), device=dev), 4,
                            scores=torch.empty((1, B), device=dev), zT=torch.empty((B, base.d), device=dev),
                            phi=torch.empty((B, base.e), device=dev),
                            idx=torch.empty((1, 1, 4), dtype=torch.int32, device=dev),
                            status=torch.zeros(64, dtype=torch.int32, device=dev))
    assert e.value.status == 1 and "scratch" in str(e.value)
