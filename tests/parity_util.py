"""Helpers shared by the GPU parity tests: running the HIP path through the
C ABI on seeded inputs and comparing with the oracle.

Comparison rules (tolerances from the evaluator's accuracy target: 1e-4
relative in fp32, 2e-2 relative in bf16):
  * terminal latents: per candidate ||g - o||_2 / ||o||_2 <= tol;
  * scores: |g - o| / max(|o|, rms of the segment's oracle scores) <= tol;
  * top-k: with delta = tol * max(|s_k|, rms), the selected set must equal
    the oracle's whenever the oracle gap s_k - s_{k+1} exceeds delta, rank r
    must match wherever both neighbouring gaps exceed delta, and any index
    outside the oracle set must score within delta of s_k.  Independently, the
    returned order must be exactly the order of the GPU's own scores by
    (-score, index).
"""
from __future__ import annotations

import numpy as np

TOL = {"fp32": 1e-4, "bf16": 2e-2}


def to_dev(I, dev):
    import torch
    return {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for k, v in I.items() if k != "seg_off"}


def run_evaluate(model, w, I, k, dev="cuda", scores=True, zT=True):
    """wm_evaluate on the inputs; returns numpy outputs and the device status."""
    import torch
    import paper_2606_09312_amd as wm
    t = to_dev(I, dev)
    init = t["feats"] if "feats" in t else t["z0"]
    B = I["lens"].shape[0]
    n_hw = I["hw"].shape[0]
    sc = torch.empty((n_hw, B), dtype=torch.float32, device=dev) if scores else None
    z = torch.empty((B, w.d), dtype=torch.float32, device=dev) if zT else None
    out = wm.evaluate(model, init, I["seg_off"], t["types"], t["params"], t["lens"], t["hw"], k,
                      init_is_feats="feats" in t, scores=sc, zT=z)
    status = 0
    try:
        wm.device_status(out["ws"])
    except wm.WMError as e:
        status = e.status
    res = {"idx": out["idx"].cpu().numpy(), "val": out["val"].cpu().numpy(), "status": status}
    if scores:
        res["scores"] = sc.cpu().numpy().astype(np.float64)
    if zT:
        res["zT"] = z.cpu().numpy().astype(np.float64)
    return res


def latent_rel(g, o):
    num = np.linalg.norm(g - o, axis=1)
    den = np.maximum(np.linalg.norm(o, axis=1), 1e-30)
    return num / den


def score_rel(g, o, seg_off):
    g = np.atleast_2d(g)
    o = np.atleast_2d(o)
    out = np.zeros_like(o)
    for s in range(len(seg_off) - 1):
        lo, hi = seg_off[s], seg_off[s + 1]
        if hi == lo:
            continue
        rms = np.sqrt(np.mean(o[:, lo:hi] ** 2, axis=1, keepdims=True))
        out[:, lo:hi] = np.abs(g[:, lo:hi] - o[:, lo:hi]) / np.maximum(np.abs(o[:, lo:hi]), np.maximum(rms, 1e-30))
    return out


def check_topk_self_consistent(idx, val, scores, seg_off, k):
    """Returned order == exact (-score, index) order of the GPU's own scores."""
    scores = np.atleast_2d(scores)
    for j in range(idx.shape[0]):
        for s in range(len(seg_off) - 1):
            lo, hi = seg_off[s], seg_off[s + 1]
            y = scores[j, lo:hi].astype(np.float32).astype(np.float64)
            nan = np.isnan(y)
            want = lo + np.lexsort((np.arange(hi - lo), np.where(nan, 0.0, -y), nan))[:k]
            np.testing.assert_array_equal(idx[j, s], want)
            np.testing.assert_array_equal(val[j, s], scores[j, idx[j, s]].astype(np.float32))


def check_topk_vs_oracle(idx, oracle_scores, seg_off, k, tol):
    o = np.atleast_2d(oracle_scores)
    for j in range(idx.shape[0]):
        for s in range(len(seg_off) - 1):
            lo, hi = seg_off[s], seg_off[s + 1]
            y = o[j, lo:hi]
            order = np.lexsort((np.arange(hi - lo), -y))
            rms = np.sqrt(np.mean(y ** 2))
            sk = y[order[k - 1]]
            delta = tol * max(abs(sk), rms)
            gpu = np.asarray(idx[j, s]) - lo
            ref_set = set(order[:k].tolist())
            if k < hi - lo and sk - y[order[k]] > delta:
                assert set(gpu.tolist()) == ref_set, f"top-k set differs (hw {j}, seg {s})"
            for i in gpu.tolist():
                if i not in ref_set:
                    assert abs(y[i] - sk) <= delta, f"index {i} outside the oracle top-k"
            ys = y[order]
            for r in range(k):
                left = ys[r - 1] - ys[r] if r > 0 else np.inf
                right = ys[r] - ys[r + 1] if r + 1 < hi - lo else np.inf
                if left > delta and right > delta:
                    assert gpu[r] == order[r], f"rank {r} differs (hw {j}, seg {s})"


def sub_batch(I, pick, seg_of, z0_full):
    """Candidates `pick` as a batch of their own, one subgraph each."""
    n = len(pick)
    return {
        "types": I["types"][pick], "params": I["params"][pick], "lens": I["lens"][pick],
        "hw": I["hw"], "z0": z0_full[seg_of[pick]], "seg_off": np.arange(n + 1, dtype=np.int32),
    }


# --------------------------------------------------------------------------
# Whole-batch oracle: the candidates are independent (the oracle's
# batch-splitting pin), so the float64 oracle runs on sub-batches in worker
# processes with one BLAS thread each and the results are put back in order.

_W = {}


def _worker_init(W, prec, norm):
    from threadpoolctl import threadpool_limits
    from oracle import wm_oracle as O
    _W["Wd"] = O.prepare(W, prec)
    _W["prec"], _W["norm"] = prec, norm
    _W["limit"] = threadpool_limits(limits=1, user_api="blas")


def _oracle_part(z0s, types, params, lens, hw):
    from oracle import wm_oracle as O
    n = lens.shape[0]
    zT, phi = O.rollout(_W["Wd"], z0s, np.arange(n + 1), types, params, lens, _W["prec"],
                        norm=_W["norm"])
    return zT, O.score(_W["Wd"], zT, phi, hw, _W["prec"])


def oracle_full(W, I, prec, k, norm="none", workers=None, parts_per_worker=4):
    """O.evaluate over the whole batch, computed in parallel sub-batches:
    returns z_T [B][d], scores [n_hw][B], idx and val of the top-k."""
    import multiprocessing as mp
    import os
    import time
    from concurrent.futures import ProcessPoolExecutor
    from oracle import wm_oracle as O
    B = I["lens"].shape[0]
    Wd = O.prepare(W, prec)
    z0 = O.encode(Wd, I["feats"], prec) if "feats" in I else I["z0"].astype(np.float64)
    seg_of = O.segment_of(I["seg_off"], B)
    workers = workers or min(16, len(os.sched_getaffinity(0)))
    n_parts = max(1, min(B, workers * parts_per_worker))
    # balance by total steps: deal the candidates out in length order
    order = np.argsort(-I["lens"].astype(np.int64), kind="stable")
    parts = [np.sort(order[p::n_parts]) for p in range(n_parts)]
    zT = np.empty((B, W["w2"].shape[0]))
    y = np.empty((I["hw"].shape[0], B))
    ctx = mp.get_context("spawn")
    with ProcessPoolExecutor(max_workers=workers, mp_context=ctx, initializer=_worker_init,
                             initargs=(W, prec, norm)) as ex:
        futs = [ex.submit(_oracle_part, z0[seg_of[p]], I["types"][p], I["params"][p], I["lens"][p],
                          I["hw"]) for p in parts]
        t0 = last = time.time()
        for n, (p, f) in enumerate(zip(parts, futs)):
            zp, yp = f.result()
            zT[p] = zp
            y[:, p] = yp
            if time.time() - last > 20:      # a long oracle run reports progress
                last = time.time()
                print(f"    oracle: {n + 1}/{len(parts)} parts, {last - t0:.0f} s", flush=True)
    idx, val = O.topk(y, I["seg_off"], k)
    return {"zT": zT, "scores": y, "idx": idx, "val": val}


def oracle_sensitivity(W, I, prec, k, norm, ref, seeds=(77,), full=False):
    """How far the oracle's own z_T and scores move when its inputs move by a
    seeded 1e-6 relative perturbation (initial latents, or program features
    when the initial latents are encoded), maximised over `seeds`.  With
    rounding to bf16 at every step's operands, rollouts are sensitive at this
    level, and an implementation that accumulates in another order sees
    perturbations at least this large.  Computed from the oracle alone.
    Returns (latent, score) in the comparison norms of latent_rel and
    score_rel."""
    from oracle import wm_oracle as O
    key = "feats" if "feats" in I else "z0"
    sz = ss = 0.0
    for seed in seeds:
        rng = np.random.default_rng(seed)
        J = dict(I)
        J[key] = (I[key].astype(np.float64) * (1 + 1e-6 * rng.standard_normal(I[key].shape))).astype(np.float32)
        pert = oracle_full(W, J, prec, k, norm=norm) if full else O.evaluate(W, J, k, prec, norm=norm)
        sz = max(sz, float(latent_rel(pert["zT"], ref["zT"]).max()))
        ss = max(ss, float(score_rel(pert["scores"], ref["scores"], I["seg_off"]).max()))
    return sz, ss


def bounds(prec, sens):
    """The stated tolerance (1e-4 fp32, 2e-2 bf16), widened in bf16 to twice
    the oracle's own sensitivity where that is larger."""
    tol = TOL[prec]
    if prec != "bf16":
        return tol, tol
    return max(tol, 2 * sens[0]), max(tol, 2 * sens[1])
