"""Reference oracle for the batched latent-rollout evaluator (float64, NumPy).

TEST INFRASTRUCTURE ONLY.  This module is the plain, slow definition of what
the evaluator computes, used to check the HIP path.  Only the tests, the
smoke check and the benchmark's CPU-baseline leg may import it; the product
path never calls it.

What is computed (paper, Sec. 3.2 "Problem Formulation", Eq. 2-3; Sec. 2.1.2,
Eq. 1; Sec. 3.4 Eq. 8; Sec. 3.5 Eq. 12; Sec. 3.6):

  z_0     = E(s_0)                                   (given, or an encoder MLP)
  z_t     = F(z_{t-1}, a_t),  t = 1..T_i             (applied recurrently)
  phi_i   = mean_t embed(a_t)                        (action features)
  y_{j,i} = G(z_T, phi_i, h_j)                       (score, higher = better)
  top-k of y within each (hardware vector, subgraph) ordered by (-y, index)

with the instantiation used throughout (residual-MLP transition, MLP cost
model, type-embedding plus linear(log2 params) action embedding):

  e_t  = type_emb[type_t] + param_w . log2(params_t) + param_b
  z_t  = z_{t-1} + W2 . GELU(W1 . [z_{t-1}; e_t] + b1) + b2
  y    = wc2 . GELU(Wc1 . [z_T; phi; h] + bc1) + bc2
  GELU(x) = x * (1 + erf(x / sqrt 2)) / 2

Paper-form transition (norm="l2"; Sec. 3.4: the state is first moved into
an action-conditioned hyperplane in the manner of TransH [Wang et al., AAAI
2014], then updated by the residual network, then normalised; the losses
of Sec. 3.4 live in that normalised space):

  v    = Wh . e_t                  normal of the action's hyperplane
  z'   = z - (w . z) w,  w = v / ||v||_2   (z' = z when v = 0)
  u    = z' + W2 . GELU(W1 . [z'; e_t] + b1) + b2
  z_t  = u / ||u||_2                       (z_t = u when u = 0)

z_0 itself is used as given (only transition outputs are normalised), and
an empty sequence still returns z_0.

bf16 mode rounds, to the nearest bfloat16 with ties to even (function R),
exactly the matrix-product operands: the matrices W1, W2, Wc1, We1, We2 (and
Wh) once, and the vectors [z; e] (z' in the paper form), e as the operand of
Wh, GELU(.) of the transition, [z_T; phi; h], the encoder
input and the encoder hidden layer.  Everything else (biases, the embedding,
the residual sum, phi, the cost hidden layer and the final wc2 dot) stays
unrounded.  The oracle evaluates all of this in float64.

Pinned by tests/test_oracle_pins.py (closed forms, textbook values of the
normal CDF, library bf16 conversion, brute-force sorting, and agreement with
the independent scalar implementation in oracle/scalar.py).
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np
from scipy.special import erf as _erf

# Status codes (same meaning as the C-ABI's).
OK = 0
ERR_INVALID_ARGUMENT = 1
ERR_UNSUPPORTED = 2
ERR_INPUT_RANGE = 5

MATRICES = ("w1", "w2", "wc1", "we1", "we2", "wh")
NORMS = ("none", "l2")


def bf16_round(x) -> np.ndarray:
    """R(x): nearest bfloat16 value of x (round half to even), in float64.

    bfloat16 keeps 8 significant bits and the float32 exponent range, so with
    x = m * 2**ex (0.5 <= |m| < 1) the spacing near x is 2**(ex - 8); below the
    smallest normal 2**-126 the spacing stays 2**-133.  Scaling by powers of
    two is exact, and rint rounds half to even.
    """
    x = np.asarray(x, dtype=np.float64)
    _, ex = np.frexp(x)
    ex = np.maximum(ex, -125)
    q = np.ldexp(np.rint(np.ldexp(x, 8 - ex)), ex - 8)
    big = np.abs(q) >= 2.0 ** 128
    if np.any(big):
        q = np.where(big, np.copysign(np.inf, q), q)
    return q


def gelu(x) -> np.ndarray:
    """GELU with the exact Gaussian CDF: x * Phi(x) = x (1 + erf(x/sqrt2)) / 2."""
    x = np.asarray(x, dtype=np.float64)
    return 0.5 * x * (1.0 + _erf(x / np.sqrt(2.0)))


def prepare(weights: Dict[str, np.ndarray], precision: str) -> Dict[str, np.ndarray]:
    """float64 copies of the weights; in bf16 mode the matrices are rounded."""
    W = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}
    if precision == "bf16":
        for k in MATRICES:
            if k in W:
                W[k] = bf16_round(W[k])
    elif precision != "fp32":
        raise ValueError(precision)
    return W


def _R(x, precision):
    return bf16_round(x) if precision == "bf16" else x


def embed(W, types_t: np.ndarray, params_t: np.ndarray) -> np.ndarray:
    """Dense action embedding e_t for a batch of steps.

    types_t [n] int, params_t [n][P] int (>= 1)  ->  [n][e].
    """
    u = np.log2(np.asarray(params_t, dtype=np.float64))
    return W["type_emb"][types_t] + u @ W["param_w"].T + W["param_b"]


def _unit_rows(v: np.ndarray) -> np.ndarray:
    """Each row divided by its Euclidean norm; all-zero rows stay zero."""
    n = np.sqrt(np.sum(v * v, axis=1, keepdims=True))
    return np.divide(v, n, out=np.zeros_like(v), where=n > 0)


def hyperplane_project(W, z: np.ndarray, e: np.ndarray, precision: str) -> np.ndarray:
    """z - (w . z) w with w the unit normal Wh . e of the action (Sec. 3.4, TransH)."""
    w = _unit_rows(_R(e, precision) @ W["wh"].T)
    return z - np.sum(w * z, axis=1, keepdims=True) * w


def transition(W, z: np.ndarray, e: np.ndarray, precision: str, norm: str = "none") -> np.ndarray:
    """One application of F (Eq. 1 / Eq. 8): residual two-layer MLP on [z; e].

    norm="l2" is the paper's form (Sec. 3.4): project z onto the action's
    hyperplane first, and normalise the result to unit length.
    """
    if norm not in NORMS:
        raise ValueError(norm)
    if norm == "l2":
        z = hyperplane_project(W, z, e, precision)
    x = _R(np.concatenate([z, e], axis=1), precision)
    g = _R(gelu(x @ W["w1"].T + W["b1"]), precision)
    u = z + (g @ W["w2"].T + W["b2"])
    return _unit_rows(u) if norm == "l2" else u


def encode(W, feats: np.ndarray, precision: str) -> np.ndarray:
    """Initial latents z0 = We2 . GELU(We1 . x + be1) + be2, one per subgraph."""
    x = _R(np.asarray(feats, dtype=np.float64), precision)
    hid = _R(gelu(x @ W["we1"].T + W["be1"]), precision)
    return hid @ W["we2"].T + W["be2"]


def segment_of(seg_off: np.ndarray, B: int) -> np.ndarray:
    """Subgraph index of every candidate (segments are contiguous ranges)."""
    seg = np.zeros(B, dtype=np.int64)
    for s in range(len(seg_off) - 1):
        seg[seg_off[s]:seg_off[s + 1]] = s
    return seg


def rollout(W, z0: np.ndarray, seg_off, types, params, lens, precision: str,
            trajectory: bool = False, norm: str = "none"):
    """Multi-step latent rollout over ragged action sequences (Sec. 3.4, 3.6).

    Each candidate i starts from z0 of its subgraph and applies F once per
    action t < lens[i]; entries at t >= lens[i] are never read.  Returns
    (z_T [B][d], phi [B][e]) and, with trajectory=True, the list of states
    after every step (rows frozen once a candidate's sequence has ended).
    """
    lens = np.asarray(lens, dtype=np.int64)
    B = lens.shape[0]
    seg = segment_of(np.asarray(seg_off), B)
    z = np.asarray(z0, dtype=np.float64)[seg].copy()
    acc = np.zeros((B, W["param_b"].shape[0]))
    traj = [z.copy()]
    T = int(lens.max()) if B else 0
    for t in range(T):
        act = np.nonzero(lens > t)[0]
        e = embed(W, types[act, t], params[act, t, :])
        z[act] = transition(W, z[act], e, precision, norm)
        acc[act] += e
        if trajectory:
            traj.append(z.copy())
    phi = np.zeros_like(acc)
    pos = lens > 0
    phi[pos] = acc[pos] / lens[pos, None]
    return (z, phi, traj) if trajectory else (z, phi)


def score(W, zT: np.ndarray, phi: np.ndarray, hw: np.ndarray, precision: str) -> np.ndarray:
    """Cost model G (Eq. 3 / Eq. 12) for every candidate under every hw vector.

    Returns y [n_hw][B]; higher is better.
    """
    B = zT.shape[0]
    hw_dim = W["wc1"].shape[1] - zT.shape[1] - phi.shape[1]
    hw = np.asarray(hw, dtype=np.float64).reshape(-1, hw_dim)
    out = np.empty((hw.shape[0], B))
    for j in range(hw.shape[0]):
        c = np.concatenate([zT, phi, np.broadcast_to(hw[j], (B, hw.shape[1]))], axis=1)
        c = _R(c, precision)
        u = gelu(c @ W["wc1"].T + W["bc1"])
        out[j] = u @ W["wc2"] + W["bc2"]
    return out


def topk(scores: np.ndarray, seg_off, k: int):
    """k best candidates per (hw vector, segment), ordered by (-y, index).

    Ties in y go to the lower candidate index; NaN sorts last.  Indices are
    global candidate indices.  Returns idx [n_hw][S][k] int32 and the
    matching scores val [n_hw][S][k].
    """
    scores = np.atleast_2d(np.asarray(scores, dtype=np.float64))
    seg_off = np.asarray(seg_off)
    S = len(seg_off) - 1
    idx = np.empty((scores.shape[0], S, k), dtype=np.int32)
    val = np.empty((scores.shape[0], S, k))
    for j in range(scores.shape[0]):
        for s in range(S):
            lo, hi = int(seg_off[s]), int(seg_off[s + 1])
            y = scores[j, lo:hi]
            nan = np.isnan(y)
            # primary: NaN last; then descending score; then ascending index
            order = np.lexsort((np.arange(hi - lo), np.where(nan, 0.0, -y), nan))[:k]
            idx[j, s] = lo + order
            val[j, s] = y[order]
    return idx, val


def validate(dims: Dict[str, int], *, B, T_max, seg_off, k=None, n_hw=None,
             types=None, params=None, lens=None, max_k: int = 1024,
             max_segments: int = 512) -> int:
    """Argument and input checks, with the same statuses as the C-ABI.

    Shape/argument problems give ERR_INVALID_ARGUMENT; out-of-range data at a
    valid step (length outside [0, T_max], type outside [0, n_kinds),
    parameter < 1) gives ERR_INPUT_RANGE.  Padding is never inspected.
    """
    if B < 0 or T_max < 0:
        return ERR_INVALID_ARGUMENT
    seg_off = np.asarray(seg_off)
    S = len(seg_off) - 1
    if S < 1 or S > max_segments or seg_off[0] != 0 or seg_off[-1] != B:
        return ERR_INVALID_ARGUMENT
    if np.any(np.diff(seg_off) < 0):
        return ERR_INVALID_ARGUMENT
    if n_hw is not None and n_hw < 1:
        return ERR_INVALID_ARGUMENT
    if k is not None and (k < 1 or k > max_k or k > int(np.diff(seg_off).min())):
        return ERR_INVALID_ARGUMENT
    if lens is None:
        return OK
    lens = np.asarray(lens, dtype=np.int64)
    if np.any((lens < 0) | (lens > T_max)):
        return ERR_INPUT_RANGE
    valid = np.arange(T_max)[None, :] < lens[:, None]
    ty = np.asarray(types)[valid]
    if np.any((ty < 0) | (ty >= dims["n_kinds"])):
        return ERR_INPUT_RANGE
    pa = np.asarray(params)[valid]
    if np.any(pa < 1):
        return ERR_INPUT_RANGE
    return OK


def evaluate(weights: Dict[str, np.ndarray], inputs: Dict[str, np.ndarray], k: int,
             precision: str, dims: Optional[Dict[str, int]] = None,
             norm: str = "none") -> Dict[str, np.ndarray]:
    """The whole hot path: [encode], rollout, score, top-k (Eq. 2-3, Sec. 3.6)."""
    W = prepare(weights, precision)
    if "feats" in inputs:
        z0 = encode(W, inputs["feats"], precision)
    else:
        z0 = np.asarray(inputs["z0"], dtype=np.float64)
    zT, phi = rollout(W, z0, inputs["seg_off"], inputs["types"], inputs["params"],
                      inputs["lens"], precision, norm=norm)
    y = score(W, zT, phi, inputs["hw"], precision)
    idx, val = topk(y, inputs["seg_off"], k)
    return {"z0": z0, "zT": zT, "phi": phi, "scores": y, "idx": idx, "val": val}
