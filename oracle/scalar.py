"""Scalar brute-force oracle: one candidate at a time, plain Python loops.

TEST INFRASTRUCTURE ONLY (see oracle/wm_oracle.py).  This is a second,
independent transcription of the same definitions, written with Python floats
(IEEE binary64), math.erf and math.log2 and explicit loops, sharing no code
with the vectorised oracle.  It is only fast enough for tiny shapes and exists
so the two can be checked against each other.

Definitions: transition z <- z + W2 GELU(W1 [z; e] + b1) + b2 (Eq. 1, Eq. 8,
Sec. 3.4), recurrent rollout over the action sequence (Sec. 3.4, Sec. 3.6),
action features phi = mean of the step embeddings, score
y = wc2 GELU(Wc1 [z_T; phi; h] + bc1) + bc2 (Eq. 3, Eq. 12), within-workload
ranking by descending score with the lower index first on ties (Sec. 3.5).
The paper-form transition (norm="l2", Sec. 3.4 with TransH hyperplanes)
removes from z its component along the unit vector of Wh e before the
update and rescales the updated state to unit length.
"""
from __future__ import annotations

import math


def round_bf16(v: float) -> float:
    """Nearest bfloat16 to v, ties to even (8 significant bits)."""
    if v == 0.0 or math.isnan(v) or math.isinf(v):
        return v
    m, ex = math.frexp(v)            # v = m * 2**ex, 0.5 <= |m| < 1
    if ex < -125:
        ex = -125                    # subnormal bfloat16 spacing 2**-133
    scaled = math.ldexp(v, 8 - ex)   # exact
    r = round(scaled)                # Python rounds half to even
    out = math.ldexp(float(r), ex - 8)
    if abs(out) >= 2.0 ** 128:
        return math.copysign(math.inf, out)
    return out


def gelu(v: float) -> float:
    return v * 0.5 * (1.0 + math.erf(v / math.sqrt(2.0)))


def _rnd(v, bf16):
    return round_bf16(v) if bf16 else v


def _mat(W, name, bf16):
    """Weight matrix as nested lists, rounded in bf16 mode."""
    A = W[name]
    rows = []
    for r in range(len(A)):
        rows.append([_rnd(float(A[r][c]), bf16) for c in range(len(A[r]))])
    return rows


def _vec(W, name):
    return [float(x) for x in W[name]]


def _scale_to_unit(vec):
    """vec / |vec| (Euclidean); a zero vector is returned unchanged."""
    n = math.sqrt(math.fsum(x * x for x in vec))
    return [x / n for x in vec] if n > 0 else list(vec)


def candidate(W, z0_row, types_row, params_rows, length, hw_rows, bf16, norm="none"):
    """Roll out and score one candidate.  Returns (zT, phi, [y_j for each hw])."""
    W1, W2, Wc1 = _mat(W, "w1", bf16), _mat(W, "w2", bf16), _mat(W, "wc1", bf16)
    Wh = _mat(W, "wh", bf16) if norm == "l2" else None
    b1, b2, bc1, wc2 = _vec(W, "b1"), _vec(W, "b2"), _vec(W, "bc1"), _vec(W, "wc2")
    bc2 = float(W["bc2"])
    temb = [[float(x) for x in row] for row in W["type_emb"]]
    pw = [[float(x) for x in row] for row in W["param_w"]]
    pb = _vec(W, "param_b")
    d, E = len(z0_row), len(pb)
    z = [float(x) for x in z0_row]
    acc = [0.0] * E
    for t in range(length):
        ty = int(types_row[t])
        u = [math.log2(float(p)) for p in params_rows[t]]
        e = []
        for f in range(E):
            s = temb[ty][f]
            for p in range(len(u)):
                s += pw[f][p] * u[p]
            e.append(s + pb[f])
        if norm == "l2":
            # unit normal of the action's hyperplane, then drop z's part along it
            er = [_rnd(v, bf16) for v in e]
            nrm = _scale_to_unit([sum(Wh[r][c] * er[c] for c in range(E)) for r in range(d)])
            along = sum(nrm[r] * z[r] for r in range(d))
            z = [z[r] - along * nrm[r] for r in range(d)]
        x = [_rnd(v, bf16) for v in z + e]
        g = []
        for r in range(len(W1)):
            s = b1[r]
            for c in range(len(x)):
                s += W1[r][c] * x[c]
            g.append(_rnd(gelu(s), bf16))
        znew = []
        for r in range(d):
            s = 0.0
            for c in range(len(g)):
                s += W2[r][c] * g[c]
            znew.append(z[r] + (s + b2[r]))
        z = _scale_to_unit(znew) if norm == "l2" else znew
        for f in range(E):
            acc[f] += e[f]
    phi = [a / length for a in acc] if length > 0 else [0.0] * E
    ys = []
    for h in hw_rows:
        c_in = [_rnd(v, bf16) for v in z + phi + [float(x) for x in h]]
        y = bc2
        for r in range(len(Wc1)):
            s = bc1[r]
            for c in range(len(c_in)):
                s += Wc1[r][c] * c_in[c]
            y += wc2[r] * gelu(s)
        ys.append(y)
    return z, phi, ys


def encode_row(W, feat_row, bf16):
    We1, We2 = _mat(W, "we1", bf16), _mat(W, "we2", bf16)
    be1, be2 = _vec(W, "be1"), _vec(W, "be2")
    x = [_rnd(float(v), bf16) for v in feat_row]
    hid = []
    for r in range(len(We1)):
        s = be1[r]
        for c in range(len(x)):
            s += We1[r][c] * x[c]
        hid.append(_rnd(gelu(s), bf16))
    out = []
    for r in range(len(We2)):
        s = be2[r]
        for c in range(len(hid)):
            s += We2[r][c] * hid[c]
        out.append(s)
    return out


def evaluate(W, inputs, k, precision, norm="none"):
    """Whole path, candidate by candidate; top-k by a full Python sort."""
    bf16 = precision == "bf16"
    seg_off = [int(v) for v in inputs["seg_off"]]
    S = len(seg_off) - 1
    if "feats" in inputs:
        z0 = [encode_row(W, inputs["feats"][s], bf16) for s in range(S)]
    else:
        z0 = [[float(v) for v in inputs["z0"][s]] for s in range(S)]
    B = len(inputs["lens"])
    zT, phi, ys = [], [], []
    for s in range(S):
        for i in range(seg_off[s], seg_off[s + 1]):
            L = int(inputs["lens"][i])
            zi, pi, yi = candidate(W, z0[s], inputs["types"][i], inputs["params"][i], L,
                                   inputs["hw"], bf16, norm)
            zT.append(zi)
            phi.append(pi)
            ys.append(yi)
    n_hw = len(inputs["hw"])
    scores = [[ys[i][j] for i in range(B)] for j in range(n_hw)]
    idx, val = [], []
    for j in range(n_hw):
        idx_j, val_j = [], []
        for s in range(S):
            cand = list(range(seg_off[s], seg_off[s + 1]))
            cand.sort(key=lambda i: (-scores[j][i], i))
            idx_j.append(cand[:k])
            val_j.append([scores[j][i] for i in cand[:k]])
        idx.append(idx_j)
        val.append(val_j)
    return {"z0": z0, "zT": zT, "phi": phi, "scores": scores, "idx": idx, "val": val}
