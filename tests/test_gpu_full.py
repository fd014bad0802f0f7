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


# One- and two-step sequences through the persistent kernels at every
# wavefront count and through the narrow-tile kernels, with a bound on the
# batch mean of the per-candidate errors.
# Within one or two steps the operands the kernel and the oracle round to
# bf16 differ only where a different fp32 accumulation order (about 1e-6
# relative) moves a value across a rounding boundary: a rare, independent
# event that changes one operand by one bf16 step (2^-8 relative).  One such
# operand among the H GELU outputs moves z by about 2^-8 / sqrt(H), i.e.
# 1e-4 to 2e-4 relative for H = 2048 to 512, and most candidates see none,
# so the batch mean stays below that (the largest single differences, a few
# 1e-3, stay under the standard tolerance checked as well).  A matrix product whose result is
# read before it completes, or a contraction step left out, shifts every
# candidate by about a whole term (1e-2 and more) and fails the mean bound
# even where long rollouts hide it inside their per-candidate bound.
SHORT_MEAN = 5e-4
SHORT = [
    ("large_latent", "none", 300),           # one wavefront per workgroup
    ("large_latent", "none", 20000),         # two
    ("large_latent", "none", 20000 + 13),    # two, ragged last tile
    ("large_latent", "none", 32768 + 17),    # four, ragged last tile
    ("ansor_round", "none", 20000 + 13),     # d = 256 persistent, two, ragged
    ("large_latent", "l2", 20000),
    ("multi_subgraph", "none", 20000),
    ("multi_subgraph", "none", 32768),
    ("ansor_round", "none", 2048),           # narrow tiles (H = 512)
    ("ansor_round", "l2", 2048),
    ("long_schedule", "none", 8192),         # narrow tiles, two per compute unit (H = 1024)
]


@pytest.mark.parametrize("name,norm,B", SHORT)
@pytest.mark.timeout(600)
def test_short_sequences_tight(wm, name, norm, B):
    """Persistent (and, for the smaller batches, narrow-tile) kernels on one-
    and two-step sequences in bf16: batch-mean errors against the oracle."""
    base = synth.workload(name)
    w = synth.scaled(base, B=B, S=base.S if B % base.S == 0 else 1, len_lo=1, len_hi=2, T_max=2)
    print(f"[short] {name} {norm} B={B} S={w.S}", flush=True)
    W = synth.make_weights(w, 1000)
    model = wm.Model(wm.model_dims(w), W, precision="bf16", norm=norm)
    I = synth.make_inputs(w, 4100 + B)
    k = base.k
    g = run_evaluate(model, w, I, k)
    assert g["status"] == 0
    ref = oracle_full(W, I, "bf16", k, norm=norm)
    tol_z, tol_s = bounds("bf16", (0.0, 0.0))
    rel = latent_rel(g["zT"], ref["zT"])
    srel = score_rel(g["scores"], ref["scores"], I["seg_off"])
    print(f"  z_T mean rel {rel.mean():.1e} (bound {SHORT_MEAN:.0e}), max {rel.max():.2e}; score mean "
          f"rel {srel.mean():.1e} (bound {SHORT_MEAN:.0e}), max {srel.max():.2e}", flush=True)
    assert rel.mean() <= SHORT_MEAN, f"z_T mean rel err {rel.mean():.3e}"
    assert srel.mean() <= SHORT_MEAN, f"score mean rel err {srel.mean():.3e}"
    assert rel.max() <= tol_z, f"z_T rel err {rel.max():.3e}"
    assert srel.max() <= tol_s, f"score rel err {srel.max():.3e}"
    check_topk_self_consistent(g["idx"], g["val"], g["scores"], I["seg_off"], k)
    check_topk_vs_oracle(g["idx"], ref["scores"], I["seg_off"], k, tol_s)
