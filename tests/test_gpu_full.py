"""GPU parity over whole benchmark batches.

Every candidate's terminal latent and every score are compared with the
float64 oracle on the benchmark's own seeded inputs and in the launch
configuration the benchmark times, and the whole top-k is checked against
the oracle's ranking (Sec. 3.5 ranking within a workload; Eq. 1 / Eq. 8 for
the rollout, Eq. 3 for the score).  The oracle runs on sub-batches in worker
processes (candidates are independent).  Also the batch sizes that select
the persistent kernels with two and four wavefronts per workgroup.
"""
import numpy as np
import pytest

import synth

from parity_util import (bounds, check_topk_self_consistent, check_topk_vs_oracle, latent_rel,
                         oracle_full, oracle_sensitivity, run_evaluate, score_rel)

# Tolerances: 1e-4 relative in fp32 and 2e-2 in bf16 (latents norm-wise per
# candidate, scores against max(|o|, rms of the segment's oracle scores)).
# For bf16, each bound is widened to twice the oracle's own change under a
# seeded 1e-6 relative perturbation of its inputs when that is larger: with
# rounding to bf16 at every step's operands, 48-step rollouts of the
# large-latent model move by up to 1.5e-2 (scores) under such a perturbation,
# so no implementation that sums in a different order can promise 2e-2 on
# every one of 65536 candidates.

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def wm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_09312_amd as wm
    wm.load_library()
    return wm


def compare(wm, w, prec, norm, seed, k):
    W = synth.make_weights(w, 1000)
    model = wm.Model(wm.model_dims(w), W, precision=prec, norm=norm)
    I = synth.make_inputs(w, seed)
    g = run_evaluate(model, w, I, k)
    assert g["status"] == 0
    ref = oracle_full(W, I, prec, k, norm=norm)
    # the bound: the stated tolerance, widened to twice the oracle's own
    # sensitivity where that is larger (bf16 long rollouts only)
    sz, ss = oracle_sensitivity(W, I, prec, k, norm, ref, full=True) if prec == "bf16" else (0.0, 0.0)
    tol_z, tol_s = bounds(prec, (sz, ss))
    rel = latent_rel(g["zT"], ref["zT"])
    srel = score_rel(g["scores"], ref["scores"], I["seg_off"])
    print(f"  z_T max rel {rel.max():.2e} (mean {rel.mean():.1e}, bound {tol_z:.2e}; oracle sensitivity "
          f"{sz:.2e}), score max rel {srel.max():.2e} (bound {tol_s:.2e}; oracle sensitivity {ss:.2e})",
          flush=True)
    assert rel.max() <= tol_z, f"z_T rel err {rel.max():.3e}"
    assert srel.max() <= tol_s, f"score rel err {srel.max():.3e}"
    check_topk_self_consistent(g["idx"], g["val"], g["scores"], I["seg_off"], k)
    check_topk_vs_oracle(g["idx"], ref["scores"], I["seg_off"], k, tol_s)
    agree = np.mean([len(set(g["idx"][j, s]) & set(ref["idx"][j, s])) / k
                     for j in range(g["idx"].shape[0]) for s in range(g["idx"].shape[1])])
    print(f"  top-k sets agree with the oracle's on {agree:.4f} of the entries", flush=True)


# (workload, precision, transition form): the benchmark workloads at full size
FULL = [
    ("tiny", "fp32", "none"),
    ("ansor_round", "fp32", "none"),
    ("ansor_round", "bf16", "none"),
    ("long_schedule", "bf16", "none"),
    ("large_latent", "bf16", "none"),
    ("multi_subgraph", "bf16", "none"),
    ("ansor_round", "bf16", "l2"),
    ("large_latent", "bf16", "l2"),
]


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("name,prec,norm", FULL)
def test_full_batch(wm, name, prec, norm):
    w = synth.workload(name)
    print(f"[full batch] {name} {prec} {norm} B={w.B}", flush=True)
    compare(wm, w, prec, norm, 2000, w.k)


# Batches of 16384 <= B < 32768 candidates run the persistent kernels with
# two wavefronts per workgroup, 32768 and more with four.
WAVES = [
    ("ansor_round", "bf16", 20000),
    ("ansor_round", "fp32", 20000),
    ("large_latent", "bf16", 20000),
    ("ansor_round", "bf16", 32768),
    ("large_latent", "bf16", 32768 + 17),
]


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("name,prec,B", WAVES)
def test_persistent_waves(wm, name, prec, B):
    base = synth.workload(name)
    w = synth.scaled(base, B=B, S=1)
    print(f"[waves] {name} {prec} B={B}", flush=True)
    compare(wm, w, prec, "none", 2300 + B, base.k)
