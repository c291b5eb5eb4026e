"""Pins of the oracle's model assembly against an independent float64
reference written from the paper (``fake_quant_ref``).

The oracle folds the file's scales into per-channel constants (requant
multipliers, c_qk = s_q s_k / sqrt(d_head), c_pv = s_v / s_ctx, c_emb =
s_E sqrt(d), c_out = s_fin s_E) and wires LayerNorm, gamma and the scales
between layers.  Here every stage of an encoder layer, of the cross keys and
values, of teacher-forced decoder steps and of the logits is recomputed in
float64 from the stage's *oracle inputs* with the unfolded scales, and the
oracle's output must agree:

* int8 codes: equal, except +-1 where the float64 value lies within
  TOL_CODE * max(1, |v|) of a rounding boundary (x.5) -- the fp32 evaluation
  may land on either side there; such cases must stay rare;
* fp32 residual stream: within 1e-5 relative (plus a tiny absolute floor);
* logits: within 1e-5 relative.

A wrong constant (sqrt(d) for sqrt(d_head), swapped key/value scales, a
missing sqrt(d) on the embedding, the wrong input scale of W2 or of the cross
keys/values, gamma on the wrong branch, LayerNorm in the wrong place) moves
whole tensors by far more than these bounds.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from synth import generate as G

from .conftest import model_blob
from .fake_quant_ref import FakeQuantModel

TOL_CODE = 4e-5
MAX_BOUNDARY_FRAC = 2e-3

SMALL_PRE = G.ModelConfig("small-preln", 64, 4, 128, 2, 2, 500, ln_post=0, seed=77, random_gamma=True)
SMALL_POST = G.ModelConfig("small-postln", 64, 2, 128, 2, 2, 300, ln_post=1, seed=78, random_gamma=True,
                           weight_std=0.1)
VARIED = G.ModelConfig("varied-256", 256, 4, 1024, 2, 2, 32000, ln_post=0, seed=1102, random_gamma=True,
                       weight_std=0.2)
SMALL_W4 = dataclasses.replace(SMALL_PRE, name="small-preln-w4", w_bits=4, seed=80)
SHARED = G.ModelConfig("shared-preln", 64, 4, 128, 4, 3, 500, ln_post=0, seed=82, random_gamma=True,
                       weight_std=0.1, share_every=1)
FACTOR = G.ModelConfig("factorized-256", 256, 4, 512, 2, 2, 2000, ln_post=0, seed=83, random_gamma=True,
                       weight_std=0.2, emb_dim=128)
FACTOR_POST = G.ModelConfig("factorized-post", 128, 2, 256, 2, 1, 700, ln_post=1, seed=84, weight_std=0.1,
                            emb_dim=64)

MODELS = {
    "tiny": lambda: model_blob("TINY"),
    "small_pre_gamma": lambda: G.build_model(SMALL_PRE),
    "small_post_gamma": lambda: G.build_model(SMALL_POST),
    "small_pre_w4": lambda: G.build_model(SMALL_W4),
    "varied_256": lambda: G.build_model(VARIED),
    "shared_layers": lambda: G.build_model(SHARED),
    "factorized_embedding": lambda: G.build_model(FACTOR),
    "factorized_post_ln": lambda: G.build_model(FACTOR_POST),
    "mobile": lambda: model_blob("MOBILE"),
}


class Stats:
    def __init__(self):
        self.codes = 0
        self.boundary = 0


def check_codes(got, val, what, st: Stats):
    got = np.asarray(got).astype(np.int64)
    val = np.asarray(val, np.float64)
    assert got.shape == val.shape, what
    ref = np.clip(np.rint(val), -127, 127)
    diff = got - ref
    dist = np.abs(np.abs(val - np.floor(val)) - 0.5)  # distance to the nearest x.5
    near = (dist <= TOL_CODE * np.maximum(1.0, np.abs(val))) & (np.abs(val) < 127.5)
    bad = (diff != 0) & ~((np.abs(diff) == 1) & near)
    assert not bad.any(), (f"{what}: {int(bad.sum())} codes differ, e.g. oracle {got[bad][:5]} vs float64 "
                           f"{val[bad][:5]}")
    st.codes += got.size
    st.boundary += int((diff != 0).sum())


def check_f32(got, ref, what, rtol=1e-5):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    atol = 1e-7 * max(1.0, float(np.abs(ref).max()))
    err = np.abs(got - ref)
    ok = err <= rtol * np.abs(ref) + atol
    assert ok.all(), f"{what}: max rel err {float((err / (np.abs(ref) + atol)).max()):.3g}"


def encoder_stages(ref: FakeQuantModel, om, src, st: Stats):
    S = len(src)
    tr = om.encode_trace(src)
    d, F = ref.d, ref.F
    check_f32(tr["x"][0], ref.embed(src, np.arange(S)), "embedding + positions", rtol=1e-6)
    for l in range(ref.n_enc):
        p, u = ref.layer("enc", l), 2 * l
        x = tr["x"][u].astype(np.float64)
        a_val, qkv_val, ctx_val, x_next = ref.self_attention_sublayer(
            p, x, tr["a"][u], tr["pj"][u][:, : 3 * d], tr["ctx"][u], lambda i: np.arange(S))
        check_codes(tr["a"][u], a_val, f"{p} self-attention input", st)
        check_codes(tr["pj"][u][:, : 3 * d], qkv_val, f"{p} Q|K|V", st)
        check_codes(tr["ctx"][u], ctx_val, f"{p} attention context", st)
        check_f32(tr["x"][u + 1], x_next, f"{p} residual after self-attention")
        x = tr["x"][u + 1].astype(np.float64)
        a_val, h_val, x_next = ref.ffn_sublayer(p, x, tr["a"][u + 1], tr["pj"][u + 1][:, :F])
        check_codes(tr["a"][u + 1], a_val, f"{p} FFN input", st)
        check_codes(tr["pj"][u + 1][:, :F], h_val, f"{p} FFN hidden (ReLU)", st)
        check_f32(tr["x"][u + 2], x_next, f"{p} residual after FFN")
    check_codes(tr["enc"], ref.encoder_output(tr["x"][2 * ref.n_enc]), "encoder output", st)
    return tr["enc"]


def decoder_stages(ref: FakeQuantModel, om, src, tokens, st: Stats):
    d, F = ref.d, ref.F
    n = len(tokens)
    enc = om.encode(src[None, :], np.array([len(src)], np.int32))[0]
    kv = [om.cross_kv(enc[None], np.array([len(src)], np.int32), l)[0] for l in range(ref.n_dec)]
    for l in range(ref.n_dec):
        check_codes(kv[l], ref.cross_kv(enc, l), f"dec.{l} cross keys|values", st)
    tr = om.decoder_trace(src, tokens)
    inp = np.concatenate([[ref.hdr.bos_id], tokens[:-1]])
    check_f32(tr["x"][0], ref.embed(inp, np.arange(n)), "decoder embedding + positions", rtol=1e-6)
    for l in range(ref.n_dec):
        p, u = ref.layer("dec", l), 3 * l
        x = tr["x"][u].astype(np.float64)
        a_val, qkv_val, ctx_val, x_next = ref.self_attention_sublayer(
            p, x, tr["a"][u], tr["pj"][u][:, : 3 * d], tr["ctx"][u], lambda i: np.arange(i + 1))
        check_codes(tr["a"][u], a_val, f"{p} self-attention input", st)
        check_codes(tr["pj"][u][:, : 3 * d], qkv_val, f"{p} Q|K|V", st)
        check_codes(tr["ctx"][u], ctx_val, f"{p} causal self-attention context", st)
        check_f32(tr["x"][u + 1], x_next, f"{p} residual after self-attention")
        x = tr["x"][u + 1].astype(np.float64)
        a_val, q_val, ctx_val, x_next = ref.cross_attention_sublayer(
            p, x, tr["a"][u + 1], tr["pj"][u + 1][:, :d], tr["ctx"][u + 1], kv[l][: len(src)])
        check_codes(tr["a"][u + 1], a_val, f"{p} cross-attention input", st)
        check_codes(tr["pj"][u + 1][:, :d], q_val, f"{p} cross Q", st)
        check_codes(tr["ctx"][u + 1], ctx_val, f"{p} cross-attention context", st)
        check_f32(tr["x"][u + 2], x_next, f"{p} residual after cross-attention")
        x = tr["x"][u + 2].astype(np.float64)
        a_val, h_val, x_next = ref.ffn_sublayer(p, x, tr["a"][u + 2], tr["pj"][u + 2][:, :F])
        check_codes(tr["a"][u + 2], a_val, f"{p} FFN input", st)
        check_codes(tr["pj"][u + 2][:, :F], h_val, f"{p} FFN hidden (ReLU)", st)
        check_f32(tr["x"][u + 3], x_next, f"{p} residual after FFN")
    check_codes(tr["fin"], ref.final_input(tr["x"][3 * ref.n_dec]), "output projection input", st)
    if ref.factorized:
        check_codes(tr["fin_u"], ref.proj_back(tr["fin"]), "factorized embedding: final rows projected back", st)
    check_f32(tr["z"], ref.logits(tr["fin"], tr["fin_u"]), "logits (tied embedding, no bias)")
    return tr


@pytest.mark.parametrize("name", list(MODELS))
def test_assembly_matches_float64_reference(name):
    blob = MODELS[name]()
    om, ref = oracle.Model(blob), FakeQuantModel(blob)
    rng = np.random.default_rng(7)
    S = 30 if ref.d >= 256 else 11
    n = 4 if name == "mobile" else 7
    src = rng.integers(4, ref.V, S).astype(np.int32)
    toks = rng.integers(4, ref.V, n).astype(np.int32)
    st = Stats()
    encoder_stages(ref, om, src, st)
    decoder_stages(ref, om, src, toks, st)
    assert st.codes > 5000
    assert st.boundary <= MAX_BOUNDARY_FRAC * st.codes, f"{st.boundary} boundary cases of {st.codes}"


@pytest.mark.parametrize("name", ["small_pre_gamma", "varied_256"])
def test_assembly_check_rejects_other_readings(name):
    """The checks above tell the readings apart: recomputing a self-attention
    context with 1/sqrt(d) in place of 1/sqrt(d_head), or with the key and
    value scales swapped, or an FFN residual with gamma on the function branch
    instead of the residual input, fails them on the oracle's values."""
    blob = MODELS[name]()
    om, ref = oracle.Model(blob), FakeQuantModel(blob)
    src = np.random.default_rng(8).integers(4, ref.V, 11).astype(np.int32)
    tr = om.encode_trace(src)
    d = ref.d
    s_out = ref.vec("enc.0.sa.qkv.sout")
    s_ctx = ref.scalar("enc.0.sa.o.sin")
    q, k, v = tr["pj"][0][:, :d], tr["pj"][0][:, d:2 * d], tr["pj"][0][:, 2 * d:3 * d]
    check_codes(tr["ctx"][0], ref.attention(q, k, v, s_out[0], s_out[1], s_out[2], s_ctx), "context", Stats())
    # 1/sqrt(d) in place of 1/sqrt(d_head): the query scale times sqrt(d_head / d)
    wrong_scale = ref.attention(q, k, v, s_out[0] * np.sqrt(ref.dh / d), s_out[1], s_out[2], s_ctx)
    swapped = ref.attention(q, k, v, s_out[0], s_out[2], s_out[1], s_ctx)
    for what, bad in (("1/sqrt(d)", wrong_scale), ("swapped key/value scales", swapped)):
        with pytest.raises(AssertionError):
            check_codes(tr["ctx"][0], bad, what, Stats())
    x = tr["x"][1].astype(np.float64)
    g = ref.scalar("enc.0.ff.gamma")
    s_h = ref.scalar("enc.0.ff.w1.sout")
    upd = ref.linear(tr["pj"][1][:, : ref.F], s_h, "enc.0.ff.w2")
    assert abs(g - 1.0) > 0.05
    with pytest.raises(AssertionError):
        check_f32(tr["x"][2], x + g * upd, "gamma on the function branch")


@pytest.mark.parametrize("name", ["varied_256", "mobile"])
def test_int8_argmax_agrees_with_float_model(name):
    """Sanity check of the whole int8 model: teacher-forced on the oracle's
    own greedy output, its arg-max agrees with the arg-max of the same model
    run in float64 with real-valued weights and no activation quantization on
    most steps (8-bit activations perturb, they do not scramble, the logits)."""
    blob = MODELS[name]()
    om, ref = oracle.Model(blob), FakeQuantModel(blob)
    agree = total = 0
    for s in range(3):
        src, lens = G.make_sources(ref.V, 1, [20 + 5 * s], seed=60 + s)
        out, _, z = om.greedy(src, lens, 12, want_logits=True)
        zf = ref.float_logits(src[0, : lens[0]], out[0])
        agree += int((zf.argmax(axis=1) == z[0].argmax(axis=1)).sum())
        total += 12
        # the int8 logits track the float ones closely in correlation
        for t in range(12):
            c = np.corrcoef(zf[t], z[0, t])[0, 1]
            assert c > 0.98, f"step {t}: correlation {c:.4f}"
    assert agree >= 0.75 * total, f"{agree}/{total} arg-max agreements"
