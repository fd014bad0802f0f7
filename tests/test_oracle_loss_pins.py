"""Pins for the oracle of the rollout loss and its gradients (Sec. 3.4):
central finite differences of the loss, torch.autograd on an independent
float64 forward, closed forms, the hardest-negative rule, and the bf16
rounding points of the backward products."""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import loss as LO
from oracle import scalar as S
from oracle import wm_oracle as O

KEYS = ("w1", "b1", "w2", "b2", "type_emb", "param_w", "param_b")


def _case(B=5, T=4, NN=3, d=3, e=2, H=4, K=3, P=2, seed=0, S_=1):
    w = synth.Workload(name="t", B=B, d=d, e=e, n_kinds=K, n_params=P, H=H, C=4, hw_dim=2,
                       n_hw=1, k=1, S=S_, lengths="uniform", len_lo=1, len_hi=T, T_max=T)
    W = synth.make_weights(w, seed)
    I = synth.make_inputs(w, seed + 1, pad="garbage")
    rng = np.random.default_rng(seed + 2)
    tgt = rng.standard_normal((B, T, d))
    neg = rng.standard_normal((B, T, NN, d))
    return w, W, I, tgt, neg


def _loss(W, I, tgt, neg, lam, gamma, prec="fp32"):
    return LO.loss_and_grad(W, I, tgt, neg, lam, gamma, prec)[0]


@pytest.mark.parametrize("lam,gamma", [(0.5, 0.3), (1.0, 0.0), (0.2, 5.0)])
def test_gradients_match_central_differences(lam, gamma):
    w, W, I, tgt, neg = _case(seed=3)
    W = {k: v.astype(np.float64) for k, v in W.items()}
    L, _, G = LO.loss_and_grad(W, I, tgt, neg, lam, gamma, "fp32")
    h = 1e-6
    for k in KEYS:
        flat = W[k].reshape(-1)
        for q in range(flat.size):
            Wp = {kk: vv.copy() for kk, vv in W.items()}
            Wm = {kk: vv.copy() for kk, vv in W.items()}
            Wp[k].reshape(-1)[q] += h
            Wm[k].reshape(-1)[q] -= h
            fd = (_loss(Wp, I, tgt, neg, lam, gamma) - _loss(Wm, I, tgt, neg, lam, gamma)) / (2 * h)
            assert fd == pytest.approx(G[k].reshape(-1)[q], rel=1e-5, abs=1e-7), (k, q)
    # the initial state: every candidate of the (single) segment shares z0
    for c in range(w.d):
        Ip, Im = dict(I), dict(I)
        Ip["z0"] = I["z0"].astype(np.float64).copy(); Ip["z0"][0, c] += h
        Im["z0"] = I["z0"].astype(np.float64).copy(); Im["z0"][0, c] -= h
        fd = (_loss(W, Ip, tgt, neg, lam, gamma) - _loss(W, Im, tgt, neg, lam, gamma)) / (2 * h)
        assert fd == pytest.approx(G["z0"][:, c].sum(), rel=1e-5, abs=1e-7)


def _torch_forward(W, I, tgt, neg, lam, gamma):
    """Independent float64 forward in torch (autograd takes the derivative)."""
    Wt = {k: torch.tensor(np.asarray(v, dtype=np.float64), requires_grad=True) for k, v in W.items()}
    seg_off = list(I["seg_off"])
    L = torch.zeros((), dtype=torch.float64)
    for i in range(len(I["lens"])):
        s = max(j for j in range(len(seg_off) - 1) if seg_off[j] <= i)
        z = torch.tensor(np.asarray(I["z0"][s], dtype=np.float64))
        for t in range(int(I["lens"][i])):
            u = torch.tensor(np.log2(np.asarray(I["params"][i, t], dtype=np.float64)))
            e = Wt["type_emb"][int(I["types"][i, t])] + Wt["param_w"] @ u + Wt["param_b"]
            a = Wt["w1"] @ torch.cat([z, e]) + Wt["b1"]
            g = a * 0.5 * (1 + torch.erf(a / math.sqrt(2)))
            z = z + Wt["w2"] @ g + Wt["b2"]
            y = torch.tensor(tgt[i, t])
            dpos = torch.linalg.vector_norm(z - y)
            dneg = torch.stack([torch.linalg.vector_norm(z - torch.tensor(n)) for n in neg[i, t]]).min()
            L = L + lam * torch.sum((z - y) ** 2) + (1 - lam) * torch.clamp(dpos - dneg + gamma, min=0)
    L.backward()
    return float(L.detach()), {k: Wt[k].grad.numpy() for k in KEYS}


def test_gradients_match_torch_autograd():
    w, W, I, tgt, neg = _case(B=7, T=5, NN=4, d=4, e=3, H=6, K=3, P=2, seed=8, S_=1)
    L, _, G = LO.loss_and_grad(W, I, tgt, neg, 0.4, 0.5, "fp32")
    Lt, Gt = _torch_forward(W, I, tgt, neg, 0.4, 0.5)
    assert L == pytest.approx(Lt, rel=1e-12)
    for k in KEYS:
        np.testing.assert_allclose(G[k], Gt[k], rtol=1e-10, atol=1e-12, err_msg=k)


def test_closed_form_without_output_layer():
    """W2 = 0, b2 = 0, one step, lam = 1: L = |z0 - z*|^2, dL/dz0 = 2(z0 - z*),
    dW2 = 2 (z0 - z*) g^T, and nothing reaches W1 or the embedding."""
    w, W, I, tgt, neg = _case(B=4, T=1, seed=5)
    W = dict(W, w2=np.zeros_like(W["w2"]), b2=np.zeros_like(W["b2"]))
    I["lens"][:] = 1
    L, per, G = LO.loss_and_grad(W, I, tgt, neg, 1.0, 0.0, "fp32")
    z0 = I["z0"][0].astype(np.float64)
    r = z0[None, :] - tgt[:, 0]
    np.testing.assert_allclose(per, np.sum(r * r, axis=1), rtol=1e-14)
    np.testing.assert_allclose(G["z0"], 2 * r, rtol=1e-14)
    np.testing.assert_allclose(G["b2"], 2 * r.sum(axis=0), rtol=1e-13)
    for k in ("w1", "b1", "type_emb", "param_w", "param_b"):
        np.testing.assert_array_equal(G[k], 0.0)


def test_inactive_hinge_and_zero_weight_give_zero_gradient():
    w, W, I, tgt, neg = _case(seed=6)
    L, per, G = LO.loss_and_grad(W, I, tgt, neg, 0.0, -1e6, "fp32")
    assert L == 0.0
    for k in KEYS + ("z0",):
        np.testing.assert_array_equal(G[k], 0.0)


def test_hardest_negative_is_nearest_lowest_index_on_ties():
    p = np.array([[0.0, 0.0], [0.0, 0.0]])
    tgt = np.array([[3.0, 4.0], [3.0, 4.0]])                  # distance 5
    neg = np.array([[[10.0, 0.0], [0.0, 2.0], [0.0, 1.0]],    # nearest: index 2 (distance 1)
                    [[0.0, 2.0], [2.0, 0.0], [0.0, 7.0]]])    # tie at 2: index 0
    loss, grad, hard = LO.step_losses(p, tgt, neg, 0.0, 0.5)
    np.testing.assert_array_equal(hard, [2, 0])
    np.testing.assert_allclose(loss, [5.0 - 1.0 + 0.5, 5.0 - 2.0 + 0.5])
    # d/dp (|p - t| - |p - n|) at p = 0: -t/|t| + n/|n|
    np.testing.assert_allclose(grad[0], [-0.6, -0.8 + 1.0])
    np.testing.assert_allclose(grad[1], [-0.6, -0.8 + 1.0])


def test_bf16_backward_rounds_product_operands():
    """One step in bf16: the gradients equal the float64 chain rule with R
    (the scalar oracle's rounding) applied to every product operand."""
    w, W, I, tgt, neg = _case(B=3, T=1, d=3, e=2, H=4, seed=9)
    I["lens"][:] = 1
    _, _, G = LO.loss_and_grad(W, I, tgt, neg, 0.7, 0.2, "bf16")
    r = np.vectorize(S.round_bf16)
    Wf = O.prepare(W, "fp32")
    w1, w2 = r(W["w1"].astype(np.float64)), r(W["w2"].astype(np.float64))
    gw2 = np.zeros_like(w2)
    gw1 = np.zeros_like(w1)
    for i in range(3):
        z0 = I["z0"][0].astype(np.float64)
        e = O.embed(Wf, I["types"][i:i + 1, 0], I["params"][i:i + 1, 0])[0]
        x = r(np.concatenate([z0, e]))
        a = w1 @ x + Wf["b1"]
        g = r(a * 0.5 * (1 + np.vectorize(math.erf)(a / math.sqrt(2))))
        p = z0 + w2 @ g + Wf["b2"]
        _, gp, _ = LO.step_losses(p[None], tgt[i:i + 1, 0], neg[i:i + 1, 0], 0.7, 0.2)
        dl = r(gp[0])
        gw2 += np.outer(dl, g)
        da = (dl @ w2) * LO.gelu_grad(a)
        gw1 += np.outer(r(da), x)
    np.testing.assert_allclose(G["w2"], gw2, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(G["w1"], gw1, rtol=1e-12, atol=1e-14)


def test_gelu_grad_matches_central_differences():
    a = np.linspace(-6, 6, 97)
    h = 1e-6
    fd = (O.gelu(a + h) - O.gelu(a - h)) / (2 * h)
    np.testing.assert_allclose(LO.gelu_grad(a), fd, rtol=1e-7, atol=1e-9)


# ---- the paper form (hyperplane projection, unit length; Sec. 3.4) ----------

KEYS_L2 = KEYS + ("wh",)


def _unit_targets(tgt, neg):
    """Targets and negatives on the unit sphere, where the predictions live."""
    return (tgt / np.linalg.norm(tgt, axis=-1, keepdims=True),
            neg / np.linalg.norm(neg, axis=-1, keepdims=True))


@pytest.mark.parametrize("lam,gamma", [(0.5, 0.3), (1.0, 0.0), (0.2, 5.0)])
def test_l2_gradients_match_central_differences(lam, gamma):
    w, W, I, tgt, neg = _case(seed=13)
    tgt, neg = _unit_targets(tgt, neg)
    W = {k: v.astype(np.float64) for k, v in W.items()}
    L, _, G = LO.loss_and_grad(W, I, tgt, neg, lam, gamma, "fp32", norm="l2")
    h = 1e-6
    for k in KEYS_L2:
        flat = W[k].reshape(-1)
        for q in range(flat.size):
            Wp = {kk: vv.copy() for kk, vv in W.items()}
            Wm = {kk: vv.copy() for kk, vv in W.items()}
            Wp[k].reshape(-1)[q] += h
            Wm[k].reshape(-1)[q] -= h
            fd = (LO.loss_and_grad(Wp, I, tgt, neg, lam, gamma, "fp32", norm="l2")[0]
                  - LO.loss_and_grad(Wm, I, tgt, neg, lam, gamma, "fp32", norm="l2")[0]) / (2 * h)
            assert fd == pytest.approx(G[k].reshape(-1)[q], rel=1e-5, abs=1e-7), (k, q)
    for c in range(w.d):
        Ip, Im = dict(I), dict(I)
        Ip["z0"] = I["z0"].astype(np.float64).copy(); Ip["z0"][0, c] += h
        Im["z0"] = I["z0"].astype(np.float64).copy(); Im["z0"][0, c] -= h
        fd = (LO.loss_and_grad(W, Ip, tgt, neg, lam, gamma, "fp32", norm="l2")[0]
              - LO.loss_and_grad(W, Im, tgt, neg, lam, gamma, "fp32", norm="l2")[0]) / (2 * h)
        assert fd == pytest.approx(G["z0"][:, c].sum(), rel=1e-5, abs=1e-7)


def _torch_forward_l2(W, I, tgt, neg, lam, gamma, project=True):
    """Independent float64 forward of the paper form in torch: TransH
    projection with the unit normal of Wh e, residual MLP, unit length."""
    Wt = {k: torch.tensor(np.asarray(v, dtype=np.float64), requires_grad=True) for k, v in W.items()}
    seg_off = list(I["seg_off"])
    L = torch.zeros((), dtype=torch.float64)
    for i in range(len(I["lens"])):
        s = max(j for j in range(len(seg_off) - 1) if seg_off[j] <= i)
        z = torch.tensor(np.asarray(I["z0"][s], dtype=np.float64))
        for t in range(int(I["lens"][i])):
            u = torch.tensor(np.log2(np.asarray(I["params"][i, t], dtype=np.float64)))
            e = Wt["type_emb"][int(I["types"][i, t])] + Wt["param_w"] @ u + Wt["param_b"]
            if project:
                v = Wt["wh"] @ e
                wn = v / torch.linalg.vector_norm(v)
                z = z - torch.dot(wn, z) * wn
            a = Wt["w1"] @ torch.cat([z, e]) + Wt["b1"]
            g = a * 0.5 * (1 + torch.erf(a / math.sqrt(2)))
            un = z + Wt["w2"] @ g + Wt["b2"]
            z = un / torch.linalg.vector_norm(un)
            y = torch.tensor(tgt[i, t])
            dpos = torch.linalg.vector_norm(z - y)
            dneg = torch.stack([torch.linalg.vector_norm(z - torch.tensor(n)) for n in neg[i, t]]).min()
            L = L + lam * torch.sum((z - y) ** 2) + (1 - lam) * torch.clamp(dpos - dneg + gamma, min=0)
    L.backward()
    return float(L.detach()), {k: (Wt[k].grad.numpy() if Wt[k].grad is not None else np.zeros_like(W[k]))
                               for k in KEYS_L2}


def test_l2_gradients_match_torch_autograd():
    w, W, I, tgt, neg = _case(B=7, T=5, NN=4, d=4, e=3, H=6, K=3, P=2, seed=18, S_=1)
    tgt, neg = _unit_targets(tgt, neg)
    L, _, G = LO.loss_and_grad(W, I, tgt, neg, 0.4, 0.5, "fp32", norm="l2")
    Lt, Gt = _torch_forward_l2(W, I, tgt, neg, 0.4, 0.5)
    assert L == pytest.approx(Lt, rel=1e-12)
    for k in KEYS_L2:
        np.testing.assert_allclose(G[k], Gt[k], rtol=1e-10, atol=1e-12, err_msg=k)


def test_l2_zero_normal_map_has_no_projection():
    """Wh = 0: no hyperplane (the zero normal skips the projection); the
    gradients equal autograd's for the plain step followed by unit length,
    and the gradient taken for Wh is the subgradient 0."""
    w, W, I, tgt, neg = _case(B=6, T=4, NN=3, d=4, e=3, H=5, seed=21)
    tgt, neg = _unit_targets(tgt, neg)
    W = dict(W, wh=np.zeros_like(W["wh"]))
    L, _, G = LO.loss_and_grad(W, I, tgt, neg, 0.5, 0.3, "fp32", norm="l2")
    Lt, Gt = _torch_forward_l2(W, I, tgt, neg, 0.5, 0.3, project=False)
    assert L == pytest.approx(Lt, rel=1e-12)
    for k in KEYS:
        np.testing.assert_allclose(G[k], Gt[k], rtol=1e-10, atol=1e-12, err_msg=k)
    np.testing.assert_array_equal(G["wh"], 0.0)


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_l2_loss_uses_the_rollout_oracles_predictions(prec):
    """The per-candidate losses equal the step losses of the (separately
    pinned) paper-form rollout trajectory."""
    w, W, I, tgt, neg = _case(B=6, T=5, seed=23)
    tgt, neg = _unit_targets(tgt, neg)
    _, per, _ = LO.loss_and_grad(W, I, tgt, neg, 0.6, 0.4, prec, norm="l2")
    Wd = O.prepare(W, prec)
    _, _, traj = O.rollout(Wd, I["z0"], I["seg_off"], I["types"], I["params"], I["lens"], prec,
                           trajectory=True, norm="l2")
    want = np.zeros(w.B)
    for t in range(w.T_max):
        act = np.nonzero(I["lens"] > t)[0]
        if act.size:
            want[act] += LO.step_losses(traj[t + 1][act], tgt[act, t], neg[act, t], 0.6, 0.4)[0]
    np.testing.assert_allclose(per, want, rtol=1e-12, atol=1e-12)


def test_l2_bf16_backward_rounds_the_normal_map_operands():
    """One step in bf16: dWh = R(dv) R(e)^T and the embedding receives
    R(Wh)^T R(dv), with dv from the float64 chain rule on the rounded
    forward (scalar oracle's rounding)."""
    w, W, I, tgt, neg = _case(B=3, T=1, d=3, e=2, H=4, seed=29)
    tgt, neg = _unit_targets(tgt, neg)
    I["lens"][:] = 1
    _, _, G = LO.loss_and_grad(W, I, tgt, neg, 0.7, 0.2, "bf16", norm="l2")
    r = np.vectorize(S.round_bf16)
    Wf = O.prepare(W, "fp32")
    wh, w1, w2 = (r(W[k].astype(np.float64)) for k in ("wh", "w1", "w2"))
    gwh = np.zeros_like(wh)
    gte = np.zeros_like(Wf["type_emb"])
    for i in range(3):
        z0 = I["z0"][0].astype(np.float64)
        e = O.embed(Wf, I["types"][i:i + 1, 0], I["params"][i:i + 1, 0])[0]
        v = wh @ r(e)
        wn = v / np.linalg.norm(v)
        zp = z0 - (wn @ z0) * wn
        x = r(np.concatenate([zp, e]))
        a = w1 @ x + Wf["b1"]
        g = r(a * 0.5 * (1 + np.vectorize(math.erf)(a / math.sqrt(2))))
        un = zp + w2 @ g + Wf["b2"]
        zh = un / np.linalg.norm(un)
        _, gp, _ = LO.step_losses(zh[None], tgt[i:i + 1, 0], neg[i:i + 1, 0], 0.7, 0.2)
        du = (gp[0] - (gp[0] @ zh) * zh) / np.linalg.norm(un)
        da = (r(du) @ w2) * LO.gelu_grad(a)
        dx = r(da) @ w1
        dzp = du + dx[:3]
        dw = -((wn @ z0) * dzp + (wn @ dzp) * z0)
        dv = (dw - (dw @ wn) * wn) / np.linalg.norm(v)
        gwh += np.outer(r(dv), r(e))
        gte[I["types"][i, 0]] += dx[3:] + r(dv) @ wh
    np.testing.assert_allclose(G["wh"], gwh, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(G["type_emb"], gte, rtol=1e-12, atol=1e-14)
