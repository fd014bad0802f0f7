"""Reference oracle for the batched rollout loss and its gradients (float64).

TEST INFRASTRUCTURE ONLY: the plain definition used to check the HIP path.
Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import it; the product path never calls it.

Loss (paper, Sec. 3.4, the transition's training objective): starting from
z0 the transition is applied recurrently over the action sequence; at every
valid step t the predicted state p_t = z_{t+1} is compared with its target
z*_t and with a set of negative states, and

  match_t = |p_t - z*_t|^2
  rank_t  = max(0, d(p_t, z*_t) - min_n d(p_t, z-_{t,n}) + gamma)
  L       = sum_i sum_{t < len_i} ( lam * match_t + (1 - lam) * rank_t )

with d the Euclidean distance and the hardest negative the nearest one
(lowest index on ties).  The gradients are those of L with respect to the
transition weights (W1, b1, W2, b2, and Wh for the paper form), the action
embedding (type_emb, param_w, param_b) and every candidate's initial state,
obtained by the chain rule backwards through the steps (subgradient 0 at the
hinge, at a zero distance and at a zero hyperplane normal).  Both transition
forms: the residual MLP (norm="none") and the paper's form (norm="l2":
z' = z - (w . z) w with w = Wh e / |Wh e|, u = z' + MLP([z'; e]),
z_next = u / |u|), where the predictions compared with the targets are unit
vectors.

bf16 mode: every matrix product of the forward and of the backward takes
bfloat16-rounded operands (R) with float64 (here) / float32 (GPU)
accumulation, as in the evaluator: forward x = R([z; e]), g = R(GELU(a));
backward dg = R(W2)^T R(du), dx = R(W1)^T R(da) (du the gradient reaching
the un-normalised update u; du = delta in the residual form); weight
gradients dW2 = sum R(du) g^T, dW1 = sum R(da) x^T; in the paper form also
v = R(Wh) R(e), de += R(Wh)^T R(dv), dWh = sum R(dv) R(e)^T; the rounding
itself is passed through unchanged (its derivative is taken as one).

Pinned by tests/test_oracle_loss_pins.py (central finite differences in
float64, torch.autograd on an independent float64 forward, closed forms,
and the bf16 rounding points).
"""
from __future__ import annotations

from typing import Dict

import numpy as np
from scipy.special import erf as _erf

from . import wm_oracle as O


def _R(x, precision):
    return O.bf16_round(x) if precision == "bf16" else np.asarray(x, dtype=np.float64)


def gelu_grad(a) -> np.ndarray:
    """d/da of a*Phi(a) = Phi(a) + a*phi(a)."""
    a = np.asarray(a, dtype=np.float64)
    return 0.5 * (1.0 + _erf(a / np.sqrt(2.0))) + a * np.exp(-0.5 * a * a) / np.sqrt(2.0 * np.pi)


def _unit(v):
    n = np.sqrt(np.sum(v * v, axis=-1, keepdims=True))
    return np.divide(v, n, out=np.zeros_like(v), where=n > 0), n[..., 0]


def step_losses(p, target, negatives, lam: float, gamma: float):
    """Per-step loss and its gradient with respect to the prediction p.

    p, target [n][d]; negatives [n][NN][d].  Returns (loss [n], dL/dp [n][d],
    index of the hardest negative [n]).
    """
    diff = p - target
    match = np.sum(diff * diff, axis=1)
    upos, dpos = _unit(diff)
    dn = np.sqrt(np.sum((p[:, None, :] - negatives) ** 2, axis=2))      # [n][NN]
    hard = np.argmin(dn, axis=1)                                         # first minimum
    rows = np.arange(p.shape[0])
    dneg = dn[rows, hard]
    uneg, _ = _unit(p - negatives[rows, hard])
    hinge = dpos - dneg + gamma
    active = hinge > 0
    loss = lam * match + (1.0 - lam) * np.where(active, hinge, 0.0)
    grad = lam * 2.0 * diff + (1.0 - lam) * active[:, None] * (upos - uneg)
    return loss, grad, hard


def loss_and_grad(weights: Dict[str, np.ndarray], inputs: Dict[str, np.ndarray], targets,
                  negatives, lam: float, gamma: float, precision: str, norm: str = "none"):
    """Rollout loss L and its gradients.

    inputs: z0 [S][d], seg_off, types [B][T_max], params [B][T_max][P],
    lens [B]; targets [B][T_max][d] (target of the state after step t);
    negatives [B][T_max][NN][d].  Entries at t >= lens[i] are never read.
    norm: the transition form, "none" (residual MLP) or "l2" (the paper's
    form: hyperplane projection before, unit length after every step; the
    loss then compares unit-length predictions, as the paper computes both
    terms in the normalised state space).
    Returns (L, per-candidate losses [B], grads) with grads keys w1, b1, w2,
    b2, type_emb, param_w, param_b (the weight shapes), wh (norm "l2") and
    z0 [B][d] (the gradient with respect to each candidate's initial state).
    """
    if norm not in O.NORMS:
        raise ValueError(norm)
    l2 = norm == "l2"
    W = O.prepare(weights, precision)
    lens = np.asarray(inputs["lens"], dtype=np.int64)
    B = lens.shape[0]
    seg = O.segment_of(np.asarray(inputs["seg_off"]), B)
    z = np.asarray(inputs["z0"], dtype=np.float64)[seg].copy()
    types, params = inputs["types"], inputs["params"]
    targets = np.asarray(targets, dtype=np.float64)
    negatives = np.asarray(negatives, dtype=np.float64)
    d = z.shape[1]
    T = int(lens.max()) if B else 0

    # ---- forward: keep what the backward needs
    keep = []
    cand_loss = np.zeros(B)
    for t in range(T):
        act = np.nonzero(lens > t)[0]
        u = np.log2(np.asarray(params[act, t, :], dtype=np.float64))
        e = O.embed(W, types[act, t], params[act, t, :])
        zin = z[act]
        st = {"act": act, "u": u, "ty": types[act, t], "zin": zin}
        if l2:
            er = _R(e, precision)
            v = er @ W["wh"].T
            w, nv = _unit(v)
            wz = np.sum(w * zin, axis=1)
            zp = zin - wz[:, None] * w
            st.update(er=er, w=w, nv=nv, wz=wz)
        else:
            zp = zin
        x = _R(np.concatenate([zp, e], axis=1), precision)
        a = x @ W["w1"].T + W["b1"]
        g = _R(O.gelu(a), precision)
        un = zp + (g @ W["w2"].T + W["b2"])
        if l2:
            zn, nu = _unit(un)
            zn = np.where(nu[:, None] > 0, zn, un)
            st.update(zn=zn, nu=nu)
        else:
            zn = un
        z[act] = zn
        loss, grad, _ = step_losses(zn, targets[act, t], negatives[act, t], lam, gamma)
        cand_loss[act] += loss
        st.update(x=x, a=a, g=g, seed=grad)
        keep.append(st)

    # ---- backward through the steps
    keys = ("w1", "b1", "w2", "b2", "type_emb", "param_w", "param_b") + (("wh",) if l2 else ())
    grads = {k: np.zeros_like(W[k]) for k in keys}
    delta = np.zeros((B, d))
    for t in range(T - 1, -1, -1):
        st = keep[t]
        act = st["act"]
        delta[act] += st["seed"]                  # gradient reaching the state after step t
        dz_new = delta[act]
        if l2:                                    # through z = u / |u|
            zh, nu = st["zn"], st["nu"]
            du = np.where(nu[:, None] > 0,
                          (dz_new - np.sum(dz_new * zh, axis=1, keepdims=True) * zh)
                          / np.where(nu > 0, nu, 1.0)[:, None],
                          dz_new)
        else:
            du = dz_new
        dl = _R(du, precision)
        grads["w2"] += dl.T @ st["g"]
        grads["b2"] += du.sum(axis=0)
        dg = dl @ W["w2"]                          # = R(W2)^T R(du), per row
        da = dg * gelu_grad(st["a"])
        dar = _R(da, precision)
        grads["w1"] += dar.T @ st["x"]
        grads["b1"] += da.sum(axis=0)
        dx = dar @ W["w1"]                         # = R(W1)^T R(da), per row
        dzp = du + dx[:, :d]                       # residual path plus the z' part of x
        de = dx[:, d:]
        if l2:                                     # through z' = z - (w . z) w, w = v / |v|
            w, nv, wz, zin = st["w"], st["nv"], st["wz"], st["zin"]
            wdz = np.sum(w * dzp, axis=1)
            dz = dzp - wdz[:, None] * w
            dw = -(wz[:, None] * dzp + wdz[:, None] * zin)
            dv = (dw - np.sum(dw * w, axis=1, keepdims=True) * w) / np.where(nv > 0, nv, 1.0)[:, None]
            dv[nv == 0] = 0.0                      # no hyperplane: the subgradient 0
            dvr = _R(dv, precision)
            grads["wh"] += dvr.T @ st["er"]
            de = de + dvr @ W["wh"]                # = R(Wh)^T R(dv), per row
        else:
            dz = dzp
        delta[act] = dz
        np.add.at(grads["type_emb"], st["ty"], de)
        grads["param_w"] += de.T @ st["u"]
        grads["param_b"] += de.sum(axis=0)
    grads["z0"] = delta
    return float(cand_loss.sum()), cand_loss, grads
