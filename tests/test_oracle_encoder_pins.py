"""Pins for the oracle of the chunked transformer state encoder (Sec. 3.3):
torch.nn.TransformerEncoderLayer on copied weights (an independent library
implementation of the post-LayerNorm layer), torch's own bfloat16
conversion at the rounding points, hand-computed chunk boundaries, and a
closed form for the embedding normalisation, pooling over overlapping
chunks, aggregation and projection."""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import text_encoder as TE


def _tiny(seed=0, **kw):
    w = synth.TextWorkload(name="t", S=3, vocab=50, hidden=32, heads=4, ffn=48, layers=2,
                           window=8, stride=4, d=6, len_lo=0, len_hi=20)
    for k, v in kw.items():
        w = type(w)(**{**w.__dict__, k: v})
    return w, synth.make_text_weights(w, seed)


def _torch_layer(W, l, hidden, heads, ffn):
    layer = torch.nn.TransformerEncoderLayer(d_model=hidden, nhead=heads, dim_feedforward=ffn,
                                             dropout=0.0, activation="gelu", layer_norm_eps=1e-5,
                                             batch_first=True, norm_first=False, dtype=torch.float64)
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))
    with torch.no_grad():
        layer.self_attn.in_proj_weight.copy_(t(W["wqkv"][l]))
        layer.self_attn.in_proj_bias.copy_(t(W["bqkv"][l]))
        layer.self_attn.out_proj.weight.copy_(t(W["wo"][l]))
        layer.self_attn.out_proj.bias.copy_(t(W["bo"][l]))
        layer.linear1.weight.copy_(t(W["w1"][l]))
        layer.linear1.bias.copy_(t(W["b1"][l]))
        layer.linear2.weight.copy_(t(W["w2"][l]))
        layer.linear2.bias.copy_(t(W["b2"][l]))
        layer.norm1.weight.copy_(t(W["ln1_g"][l]))
        layer.norm1.bias.copy_(t(W["ln1_b"][l]))
        layer.norm2.weight.copy_(t(W["ln2_g"][l]))
        layer.norm2.bias.copy_(t(W["ln2_b"][l]))
    layer.train()          # dropout 0: the plain (non-fused) computation
    return layer


@pytest.mark.parametrize("n", [1, 5, 8])
def test_layer_matches_torch_transformer_layer(n):
    w, Wt = _tiny(seed=3)
    W = TE.prepare(Wt, "fp32")
    h = np.random.default_rng(n).standard_normal((n, w.hidden))
    for l in range(w.layers):
        got = TE.encoder_layer(W, l, h, w.heads, "fp32")
        ref = _torch_layer(Wt, l, w.hidden, w.heads, w.ffn)(torch.tensor(h)[None])[0].detach().numpy()
        np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-12)


def test_chunk_bounds_by_hand():
    assert TE.chunk_bounds(0, 4, 2) == [(0, 0)]
    assert TE.chunk_bounds(4, 4, 2) == [(0, 4)]
    assert TE.chunk_bounds(5, 4, 2) == [(0, 4), (2, 5)]
    assert TE.chunk_bounds(10, 4, 3) == [(0, 4), (3, 7), (6, 10)]
    assert TE.chunk_bounds(11, 4, 3) == [(0, 4), (3, 7), (6, 10), (9, 11)]


def test_pooling_aggregation_projection_closed_form():
    """Zero layer matrices and biases, unit LayerNorm gains, zero shifts and
    embeddings whose rows are +-1 patterns (mean 0, variance 1): every
    LayerNorm only rescales, h = f x with f from the scalar recurrence
    f <- f / sqrt(f^2 + eps) (2 L + 1 times from f = 1), so z = Wp (f * mean
    over chunks of the mean over each chunk's tokens of x) + bp."""
    w, Wt = _tiny(seed=5)
    rng = np.random.default_rng(0)
    signs = np.ones((w.vocab, w.hidden))
    for r in range(w.vocab):
        signs[r, rng.permutation(w.hidden)[: w.hidden // 2]] = -1.0
    Wt = dict(Wt, tok_emb=signs, pos_emb=np.zeros_like(Wt["pos_emb"]))
    for k in ("wqkv", "bqkv", "wo", "bo", "w1", "b1", "w2", "b2", "ln0_b", "ln1_b", "ln2_b"):
        Wt[k] = np.zeros_like(Wt[k])
    for k in ("ln0_g", "ln1_g", "ln2_g"):
        Wt[k] = np.ones_like(Wt[k])
    f = 1.0
    for _ in range(2 * w.layers + 1):
        f = f / math.sqrt(f * f + TE.LN_EPS)
    ids = rng.integers(0, w.vocab, size=13)            # chunks [0,8) [4,12) [8,13)
    chunk_means = [signs[ids[a:b]].mean(axis=0) for a, b in [(0, 8), (4, 12), (8, 13)]]
    want = Wt["wp"].astype(np.float64) @ (f * np.mean(chunk_means, axis=0)) + Wt["bp"]
    got = TE.encode(Wt, [ids], w.window, w.stride, w.heads, "fp32")[0]
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-14)
    # an empty program maps to the projection bias
    np.testing.assert_array_equal(TE.encode(Wt, [ids[:0]], w.window, w.stride, w.heads, "fp32")[0],
                                  Wt["bp"].astype(np.float64))


def test_bf16_layer_rounds_the_product_operands():
    """bf16 layer == torch float64 layer arithmetic with torch's bfloat16
    conversion applied at exactly the listed operands."""
    w, Wt = _tiny(seed=7)
    W = TE.prepare(Wt, "bf16")
    h = np.random.default_rng(2).standard_normal((7, w.hidden))
    R = lambda a: a.to(torch.bfloat16).to(torch.float64)
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))
    H, nh = w.hidden, w.heads
    dh = H // nh
    for l in range(w.layers):
        x = t(h)
        qkv = R(x) @ R(t(Wt["wqkv"][l])).T + t(Wt["bqkv"][l])
        q, k, v = qkv[:, :H], qkv[:, H:2 * H], qkv[:, 2 * H:]
        o = torch.empty_like(q)
        for a in range(nh):
            sl = slice(a * dh, (a + 1) * dh)
            p = torch.softmax((R(q[:, sl]) @ R(k[:, sl]).T) / math.sqrt(dh), dim=-1)
            o[:, sl] = R(p) @ R(v[:, sl])
        y = torch.nn.functional.layer_norm(x + R(o) @ R(t(Wt["wo"][l])).T + t(Wt["bo"][l]), (H,),
                                           t(Wt["ln1_g"][l]), t(Wt["ln1_b"][l]), eps=1e-5)
        g = torch.nn.functional.gelu(R(y) @ R(t(Wt["w1"][l])).T + t(Wt["b1"][l]))
        ref = torch.nn.functional.layer_norm(y + R(g) @ R(t(Wt["w2"][l])).T + t(Wt["b2"][l]), (H,),
                                             t(Wt["ln2_g"][l]), t(Wt["ln2_b"][l]), eps=1e-5)
        got = TE.encoder_layer(W, l, h, nh, "bf16")
        np.testing.assert_allclose(got, ref.numpy(), rtol=1e-12, atol=1e-12)


def test_encode_uses_each_chunk_and_the_mean():
    """A program shorter than the window is one chunk; the program vector
    of a two-chunk program is the mean of the two chunk encodings."""
    w, Wt = _tiny(seed=9)
    W = TE.prepare(Wt, "fp32")
    ids = np.random.default_rng(4).integers(0, w.vocab, size=10)     # chunks [0,8) [4,10)
    c0 = TE.encode_chunk(W, ids[0:8], w.heads, "fp32").mean(axis=0)
    c1 = TE.encode_chunk(W, ids[4:10], w.heads, "fp32").mean(axis=0)
    want = W["wp"] @ ((c0 + c1) / 2) + W["bp"]
    np.testing.assert_allclose(TE.encode(Wt, [ids], w.window, w.stride, w.heads, "fp32")[0], want,
                               rtol=1e-13, atol=1e-14)
