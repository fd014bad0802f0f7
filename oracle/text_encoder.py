"""Reference oracle for the chunked transformer state encoder (float64, NumPy).

TEST INFRASTRUCTURE ONLY: the plain definition used to check the HIP path.
Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import it; the product path never calls it.

What is computed (paper, Sec. 3.3: the state encoder E is a CodeBERT-based
model adapted to long TensorIR inputs; the token sequence is split into
overlapping chunks by a sliding window, every chunk is encoded on its own by
the backbone, masked mean pooling gives one vector per chunk, the chunk
vectors are aggregated into one program vector, and a projection head gives
z(s) = E(s) in R^d):

  chunks    window Wn, stride Sd: chunk c holds tokens [c Sd, min(c Sd + Wn, N)),
            n_chunks = 1 + max(0, ceil((N - Wn) / Sd))
  backbone  post-LayerNorm transformer encoder of the CodeBERT (RoBERTa) shape,
            on each chunk separately (position p = index within the chunk):
              h = LN(tok_emb[id] + pos_emb[p])
              per layer:  [q k v] = h Wqkv^T + bqkv
                          per head: o = softmax(q k^T / sqrt(dh)) v
                          h = LN(h + o Wo^T + bo)
                          h = LN(h + GELU(h W1^T + b1) W2^T + b2)
            LN(x) = (x - mean) / sqrt(var + 1e-5) * gamma + beta (biased var)
  pooling   chunk vector = mean of h over the chunk's tokens
  program   v = mean of its chunk vectors;  z = Wp v + bp

bf16 mode rounds, to the nearest bfloat16 (function R of wm_oracle), exactly
the matrix-product operands: the weight matrices Wqkv, Wo, W1, W2, Wp once,
and the activations entering each product: h before Wqkv and before W1, q
and k for q k^T, the probabilities and v for P v, the attention output
before Wo, the GELU output before W2, and the program vector before Wp.
Embeddings, biases, LayerNorm, softmax, residual sums and pooling stay
unrounded.

Pinned by tests/test_oracle_encoder_pins.py (torch.nn.TransformerEncoderLayer
on copied weights, torch's own bfloat16 conversion at the rounding points,
hand-computed chunk boundaries, and a closed form for pooling, aggregation
and projection).
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np

from .wm_oracle import bf16_round, gelu

LN_EPS = 1e-5
MATRICES = ("wqkv", "wo", "w1", "w2", "wp")


def _R(x, precision):
    return bf16_round(x) if precision == "bf16" else np.asarray(x, dtype=np.float64)


def prepare(weights: Dict[str, np.ndarray], precision: str) -> Dict[str, np.ndarray]:
    """float64 copies; in bf16 mode the weight matrices are rounded once."""
    W = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}
    if precision == "bf16":
        for k in MATRICES:
            W[k] = bf16_round(W[k])
    elif precision != "fp32":
        raise ValueError(precision)
    return W


def chunk_bounds(n_tokens: int, window: int, stride: int) -> List[tuple]:
    """[start, end) of every chunk of an n-token sequence (one chunk, possibly
    empty, when n <= window)."""
    n_chunks = 1 + max(0, -(-(n_tokens - window) // stride))
    return [(c * stride, min(c * stride + window, n_tokens)) for c in range(n_chunks)]


def layer_norm(x, gamma, beta):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + LN_EPS) * gamma + beta


def softmax_rows(s):
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


def encoder_layer(W, l: int, h, heads: int, precision: str):
    """One post-LN layer on the n x Hd states of one chunk."""
    n, Hd = h.shape
    dh = Hd // heads
    qkv = _R(h, precision) @ W["wqkv"][l].T + W["bqkv"][l]
    q, k, v = qkv[:, :Hd], qkv[:, Hd:2 * Hd], qkv[:, 2 * Hd:]
    o = np.empty((n, Hd))
    for a in range(heads):
        sl = slice(a * dh, (a + 1) * dh)
        s = (_R(q[:, sl], precision) @ _R(k[:, sl], precision).T) / np.sqrt(dh)
        p = softmax_rows(s)
        o[:, sl] = _R(p, precision) @ _R(v[:, sl], precision)
    h = layer_norm(h + _R(o, precision) @ W["wo"][l].T + W["bo"][l], W["ln1_g"][l], W["ln1_b"][l])
    f = gelu(_R(h, precision) @ W["w1"][l].T + W["b1"][l])
    h = layer_norm(h + _R(f, precision) @ W["w2"][l].T + W["b2"][l], W["ln2_g"][l], W["ln2_b"][l])
    return h


def encode_chunk(W, ids: np.ndarray, heads: int, precision: str):
    """Backbone output [n][Hd] of one chunk of token ids."""
    n = len(ids)
    h = layer_norm(W["tok_emb"][ids] + W["pos_emb"][:n], W["ln0_g"], W["ln0_b"])
    for l in range(W["wqkv"].shape[0]):
        h = encoder_layer(W, l, h, heads, precision)
    return h


def encode_program(W, ids: np.ndarray, window: int, stride: int, heads: int, precision: str):
    """z(s) of one program (token ids), W prepared."""
    ids = np.asarray(ids, dtype=np.int64)
    vecs = []
    for a, b in chunk_bounds(len(ids), window, stride):
        if b > a:
            vecs.append(encode_chunk(W, ids[a:b], heads, precision).mean(axis=0))
    v = np.mean(vecs, axis=0) if vecs else np.zeros(W["wp"].shape[1])
    return _R(v, precision) @ W["wp"].T + W["bp"]


def encode(weights, programs: Sequence[np.ndarray], window: int, stride: int, heads: int,
           precision: str) -> np.ndarray:
    """z [S][d] for a list of programs (token-id arrays; an empty program
    maps to the projection bias)."""
    W = prepare(weights, precision)
    return np.stack([encode_program(W, p, window, stride, heads, precision) for p in programs])
