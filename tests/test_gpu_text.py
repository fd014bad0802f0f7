"""GPU parity of the chunked transformer state encoder (Sec. 3.3) against the
CPU oracle, through the C ABI: the small backbone on whole batches (empty,
one-chunk and many-chunk programs, a ragged last chunk), the CodeBERT-shaped
backbone on a batch whose programs cover one and several 512-token windows,
token-id validation, determinism, and the encoder feeding the evaluator.

Comparison: per program ||g - o||_2 / ||o||_2 (the latent rule), 1e-4 in
fp32 and 2e-2 in bf16."""
import numpy as np
import pytest

import synth
from oracle import text_encoder as TE
from oracle import wm_oracle as O

from parity_util import TOL, latent_rel

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def wm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_09312_amd as wm
    wm.load_library()
    return wm


_models = {}


def model_for(wm, name, prec):
    key = (name, prec)
    if key not in _models:
        w = synth.TEXT_WORKLOADS[name]
        W = synth.make_text_weights(w, 500)
        _models[key] = (wm.TextModel(w, W, precision=prec), W, w)
    return _models[key]


def run(wm, model, tokens, off):
    t = torch.from_numpy(np.ascontiguousarray(tokens, dtype=np.int32)).cuda()
    out = wm.encode_text(model, t, off)
    wm.device_status(out["ws"])
    return out["z0"].cpu().numpy().astype(np.float64)


def programs_of(tokens, off):
    return [tokens[off[s]:off[s + 1]] for s in range(len(off) - 1)]


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_small_backbone_whole_batch(wm, prec):
    model, W, w = model_for(wm, "tiny_text", prec)
    tokens, off = synth.make_programs(w, 11)
    # an empty program, one shorter than the window, one exactly a window
    lens = np.diff(off)
    lens[0], lens[1], lens[2] = 0, 17, w.window
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    tokens = np.random.default_rng(3).integers(0, w.vocab, size=int(off[-1])).astype(np.int32)
    print(f"[text] tiny_text {prec} lens={list(lens)} chunks={model.chunks(off)}", flush=True)
    g = run(wm, model, tokens, off)
    ref = TE.encode(W, programs_of(tokens, off), w.window, w.stride, w.heads, prec)
    rel = latent_rel(g, ref)
    assert rel.max() <= TOL[prec], f"z0 rel err {rel.max():.3e}"
    np.testing.assert_allclose(g[0], W["bp"], rtol=0, atol=0)      # empty program: the bias
    print(f"  max rel {rel.max():.2e}", flush=True)


def test_codebert_backbone(wm):
    """CodeBERT shape (12 layers, 768 wide, 12 heads, 512-token windows with
    stride 256): programs of 1, 300, 512, 700 and 1100 tokens (1, 1, 1, 2, 4
    chunks)."""
    model, W, w = model_for(wm, "codebert", "bf16")
    lens = np.array([1, 300, 512, 700, 1100])
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    tokens = np.random.default_rng(5).integers(0, w.vocab, size=int(off[-1])).astype(np.int32)
    print(f"[text] codebert bf16 chunks={model.chunks(off)}", flush=True)
    g = run(wm, model, tokens, off)
    ref = TE.encode(W, programs_of(tokens, off), w.window, w.stride, w.heads, "bf16")
    rel = latent_rel(g, ref)
    assert rel.max() <= TOL["bf16"], f"z0 rel err {rel.max():.3e}"
    print(f"  max rel {rel.max():.2e}", flush=True)


def test_token_out_of_range_is_reported(wm):
    model, W, w = model_for(wm, "tiny_text", "fp32")
    off = np.array([0, 5], dtype=np.int32)
    tokens = np.array([1, 2, w.vocab, 3, 4], dtype=np.int32)
    t = torch.from_numpy(tokens).cuda()
    out = wm.encode_text(model, t, off)
    with pytest.raises(wm.WMError) as e:
        wm.device_status(out["ws"])
    assert e.value.status == 5
    wm.device_status(out["ws"])          # cleared


def test_deterministic_and_independent_of_batch(wm):
    """Repeated calls give identical bits; a program's latent does not depend
    on the other programs of the batch."""
    model, W, w = model_for(wm, "tiny_text", "bf16")
    tokens, off = synth.make_programs(w, 19)
    a = run(wm, model, tokens, off)
    b = run(wm, model, tokens, off)
    np.testing.assert_array_equal(a, b)
    s = 3
    one = run(wm, model, tokens[off[s]:off[s + 1]], np.array([0, off[s + 1] - off[s]], dtype=np.int32))
    np.testing.assert_array_equal(one[0], a[s])


def test_encoder_feeds_the_evaluator(wm):
    """The encoded programs are the initial latents of a rollout batch: the
    evaluator run on the GPU latents matches the oracle run on the oracle's
    encodings (bf16 end to end, within the latent tolerance)."""
    model, Wt, wt = model_for(wm, "tiny_text", "bf16")
    tokens, off = synth.make_programs(wt, 23)
    z0 = run(wm, model, tokens, off)
    z0_ref = TE.encode(Wt, programs_of(tokens, off), wt.window, wt.stride, wt.heads, "bf16")
    base = synth.workload("tiny")
    w = synth.scaled(base, B=wt.S * 40, S=wt.S)
    W = synth.make_weights(w, 1000)
    ev = wm.Model(wm.model_dims(w), W, precision="bf16")
    I = synth.make_inputs(w, 29)
    I["z0"] = z0.astype(np.float32)
    from parity_util import run_evaluate
    g = run_evaluate(ev, w, I, 4)
    Iref = dict(I, z0=z0_ref)
    ref = O.evaluate(W, Iref, 4, "bf16")
    assert latent_rel(g["zT"], ref["zT"]).max() <= TOL["bf16"]
