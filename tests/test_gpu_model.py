"""End-to-end GPU parity against the oracle: encoder output codes and cross
keys/values bit-exact, decode-step logits (bar: 1e-3 relative; bit-exact
expected), greedy token sequences identical on the tiny and mobile workloads,
hipGraph replay identical to eager launches, beam search identical on small
models and on sampled sentences of the batched beam workloads."""
import dataclasses

import numpy as np
import pytest

import oracle
from synth import generate as G

from .conftest import model_blob

pytestmark = pytest.mark.gpu
RTOL = 1e-3

SMALL_PRE = G.ModelConfig("small-preln", 64, 4, 128, 2, 2, 500, ln_post=0, seed=77, random_gamma=True)
SMALL_POST = G.ModelConfig("small-postln", 64, 2, 128, 2, 2, 300, ln_post=1, seed=78, random_gamma=True,
                           weight_std=0.1)
DIVERSE = G.ModelConfig("diverse-preln", 128, 2, 256, 3, 2, 700, ln_post=0, seed=81, random_gamma=True,
                        weight_std=0.1)


@pytest.fixture(scope="module")
def torch_dev():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    return torch, torch.device("cuda:0")


_models = {}


def _pair(name_or_cfg, flags=0):
    """(oracle model, GPU model) for a named workload model or a ModelConfig
    (flags: the GPU model's load flags)."""
    from paper_2306_04235_amd import mnmt

    key = (name_or_cfg if isinstance(name_or_cfg, str) else name_or_cfg.name, flags)
    if key not in _models:
        blob = model_blob(name_or_cfg) if isinstance(name_or_cfg, str) else G.build_model(name_or_cfg)
        _models[key] = (oracle.Model(blob), mnmt.Model(blob, flags=flags))
    return _models[key]


def _t(torch, dev, a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def _greedy_check(torch, dev, cfg, src, lens, steps, stop_at_eos=False, check_logits=True, flags=0):
    from paper_2306_04235_amd import mnmt

    om, gm = _pair(cfg, flags)
    B, S = src.shape
    print(f"greedy {cfg if isinstance(cfg, str) else cfg.name} B={B} S={S} steps={steps}", flush=True)
    sess = mnmt.Session(gm, B, S, steps, 1)
    ts, tl = _t(torch, dev, src), _t(torch, dev, lens)
    o_out, o_len, o_logits = om.greedy(src, lens, steps, stop_at_eos=stop_at_eos, want_logits=True)
    # encoder output and cross keys/values, bit-exact on valid rows
    sess.encode(ts, tl)
    torch.cuda.synchronize()
    enc = sess.tensor("enc_out", torch.int8, (B, S, gm.info.d_model)).cpu().numpy()
    o_enc = om.encode(src, lens)
    for b in range(B):
        assert np.array_equal(enc[b, : lens[b]], o_enc[b, : lens[b]]), f"encoder output, sentence {b}"
    for l in range(gm.info.n_dec):
        kv = sess.tensor(f"cross_kv.{l}", torch.int8, (B, S, 2 * gm.info.d_model)).cpu().numpy()
        o_kv = om.cross_kv(o_enc, lens, l)
        for b in range(B):
            assert np.array_equal(kv[b, : lens[b]], o_kv[b, : lens[b]]), f"cross kv layer {l} sentence {b}"
    # teacher-forced decode steps through the C ABI: logits and tokens
    if check_logits and not stop_at_eos:
        prev = None
        for t in range(steps):
            nxt, logits = sess.decode_step(prev, want_logits=True)
            z = logits.cpu().numpy()
            ref = o_logits[:, t]
            assert np.allclose(z, ref, rtol=RTOL, atol=RTOL * np.abs(ref).max()), f"logits step {t}"
            assert np.array_equal(z.view(np.uint32), ref.view(np.uint32)), f"logits bits step {t}"
            assert np.array_equal(nxt.cpu().numpy(), o_out[:, t]), f"tokens step {t}"
            prev = _t(torch, dev, o_out[:, t])
    # whole translation, eager and captured in a graph (replayed twice)
    for use_graph in (False, True, True):
        out, out_len, _ = sess.translate(ts, tl, beam=1, max_steps=steps, stop_at_eos=stop_at_eos,
                                         use_graph=use_graph)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy(), o_out), f"greedy tokens (graph={use_graph})"
        assert np.array_equal(out_len.cpu().numpy(), o_len)
    # each step's winning arg-max key (recorded by the step that commits the
    # token): the high word is the order-preserving key of the maximum logit
    if not stop_at_eos:
        keys = sess.tensor("out_key", torch.int64, (steps, B)).cpu().numpy().view(np.uint64)
        assert np.array_equal(keys.T, _argmax_keys(o_logits)), "arg-max keys (maximum logit bits and index)"
    # no kernel of the translation chain gave up waiting for its predecessor
    assert int(sess.tensor("chain_err", torch.int32, (1,)).cpu().numpy()[0]) == 0
    sess.status()
    sess.close()
    return o_out


def _argmax_keys(z):
    """Packed arg-max keys of fp32 logits [..., V]: order-preserving 32-bit key of
    the maximum << 32 | (0xFFFFFFFF - index of its first occurrence)."""
    idx = z.argmax(axis=-1)
    m = np.take_along_axis(z, idx[..., None], axis=-1)[..., 0]
    u = m.astype(np.float32).view(np.uint32).astype(np.uint64)
    hi = np.where(u & 0x80000000, ~u & 0xFFFFFFFF, u | 0x80000000)
    return (hi << np.uint64(32)) | (np.uint64(0xFFFFFFFF) - idx.astype(np.uint64))


def test_tiny_postln_greedy(torch_dev):
    torch, dev = torch_dev
    src, lens = G.workload_inputs(G.WORKLOADS["tiny"])
    _greedy_check(torch, dev, "TINY", src, lens, 16)


def test_small_models_batched_greedy(torch_dev):
    torch, dev = torch_dev
    for cfg in (SMALL_PRE, SMALL_POST, DIVERSE):
        src, lens = G.make_sources(cfg.vocab, 5, [1, 7, 12, 3, 12], seed=21, s_max=12)
        _greedy_check(torch, dev, cfg, src, lens, 10)
        _greedy_check(torch, dev, cfg, src, lens, 10, stop_at_eos=True, check_logits=False)


def test_one_and_two_row_greedy(torch_dev):
    # 1 or 2 rows take the three-kernels-per-layer decoder step
    torch, dev = torch_dev
    for cfg in (SMALL_PRE, SMALL_POST, DIVERSE):
        for B in (1, 2):
            src, lens = G.make_sources(cfg.vocab, B, (3, 12), seed=24 + B, s_max=12)
            _greedy_check(torch, dev, cfg, src, lens, 10)
            _greedy_check(torch, dev, cfg, src, lens, 10, stop_at_eos=True, check_logits=False)


def test_two_row_greedy_longest_sequences(torch_dev):
    # 128 source positions and 128 target steps: the longest attention of the
    # 2-row step; one position more moves both lengths to the general path
    torch, dev = torch_dev
    src, lens = G.make_sources(SMALL_POST.vocab, 2, [128, 77], seed=26, s_max=128)
    _greedy_check(torch, dev, SMALL_POST, src, lens, 128)
    src, lens = G.make_sources(SMALL_POST.vocab, 2, [129, 5], seed=27, s_max=129)
    _greedy_check(torch, dev, SMALL_POST, src, lens, 129, check_logits=False)


def test_greedy_batch_above_gemv_limit(torch_dev):
    # 12 rows: the output projection runs on matrix cores, arg-max separately
    torch, dev = torch_dev
    src, lens = G.make_sources(DIVERSE.vocab, 12, (2, 20), seed=22, s_max=20)
    _greedy_check(torch, dev, DIVERSE, src, lens, 9)


def test_diverse_model_output_depends_on_the_source(torch_dev):
    # the higher-variance test model's translations differ between sources
    torch, dev = torch_dev
    src, lens = G.make_sources(DIVERSE.vocab, 3, (8, 14), seed=23, s_max=14)
    out = _greedy_check(torch, dev, DIVERSE, src, lens, 12, check_logits=False)
    assert len({tuple(r) for r in out}) > 1


def test_mobile_greedy_latency_workload(torch_dev):
    torch, dev = torch_dev
    src, lens = G.workload_inputs(G.WORKLOADS["mobile"])
    _greedy_check(torch, dev, "MOBILE", src, lens, 30)


def test_serial_steps_match_the_kernel_chain(torch_dev, monkeypatch):
    """The batch-1 steps run as a chain of kernels over two streams, each
    waiting on its predecessor's flags; with MNMT_SERIAL_STEPS=1 (read at
    session creation) they run in one stream.  Both give the oracle's tokens."""
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    om, gm = _pair("MOBILE")
    src, lens = G.workload_inputs(G.WORKLOADS["mobile"])
    o_out, o_len = om.greedy(src, lens, 30)[:2]
    ts, tl = _t(torch, dev, src), _t(torch, dev, lens)
    for serial in ("0", "1"):
        monkeypatch.setenv("MNMT_SERIAL_STEPS", serial)
        sess = mnmt.Session(gm, 1, src.shape[1], 30, 1)
        for use_graph in (False, True):
            out, out_len, _ = sess.translate(ts, tl, beam=1, max_steps=30, use_graph=use_graph)
            torch.cuda.synchronize()
            assert np.array_equal(out.cpu().numpy(), o_out), f"serial={serial} graph={use_graph}"
            assert np.array_equal(out_len.cpu().numpy(), o_len)
        assert int(sess.tensor("chain_err", torch.int32, (1,)).cpu().numpy()[0]) == 0
        sess.close()


def test_kernel_chain_many_sentences(torch_dev, monkeypatch):
    """Two dozen different batch-1 sentences (10-30 source tokens) through the
    kernel chain, in graph replays as the benchmark runs them, against the
    one-stream steps of the same kernels (about 5,000 flag hand-offs, each
    consumer reading what its predecessors wrote on other compute units),
    and the first four against the oracle."""
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    om, gm = _pair("MOBILE")
    rng = np.random.default_rng(2024)
    lens_all = rng.integers(10, 31, 24)
    outs = {}
    for serial in ("1", "0"):
        monkeypatch.setenv("MNMT_SERIAL_STEPS", serial)
        sess = mnmt.Session(gm, 1, 30, 30, 1)
        got = []
        for k, n in enumerate(lens_all):
            src, lens = G.make_sources(G.MOBILE.vocab, 1, [int(n)], seed=500 + k, s_max=30)
            out, out_len, _ = sess.translate(_t(torch, dev, src), _t(torch, dev, lens), beam=1, max_steps=30,
                                             use_graph=True)
            torch.cuda.synchronize()
            got.append((out.cpu().numpy().copy(), out_len.cpu().numpy().copy()))
            if serial == "0" and k < 4:
                o_out, o_len = om.greedy(src, lens, 30)[:2]
                assert np.array_equal(got[-1][0], o_out) and np.array_equal(got[-1][1], o_len), f"sentence {k}"
        assert int(sess.tensor("chain_err", torch.int32, (1,)).cpu().numpy()[0]) == 0
        sess.close()
        outs[serial] = got
    for k, (a, b) in enumerate(zip(outs["0"], outs["1"])):
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]), f"sentence {k}"


LAUNCH_FORMS = {"step": {"MNMT_STEP_LAUNCH": "1"}, "layer": {}, "three": {"MNMT_MERGED_LAYERS": "0"}}


@pytest.mark.parametrize("form", list(LAUNCH_FORMS))
def test_layer_launch_forms(torch_dev, monkeypatch, form):
    """The batch-1 translation's decode step in one launch (two-layer models
    of width 256 with a 32000-word vocabulary: both layers' self-
    attention, cross-attention and FFN blocks and the logits blocks, handing
    off through the counted words and flags inside it; MNMT_STEP_LAUNCH=1),
    one launch per decoder layer and one for the logits (the default), or
    with MNMT_MERGED_LAYERS=0 three launches per layer (read at session
    creation).  Per-step logits bits and tokens equal the oracle's at one and
    two rows, pre- and post-LN, with 4-bit weights, shared layers and widths
    64-512, eager and in graph replays."""
    import dataclasses

    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    for k, v in LAUNCH_FORMS[form].items():
        monkeypatch.setenv(k, v)
    src, lens = G.workload_inputs(G.WORKLOADS["mobile"])
    _greedy_check(torch, dev, "MOBILE", src, lens, 30)
    mob4 = dataclasses.replace(G.MOBILE, name="mobile-w4", w_bits=4)
    _greedy_check(torch, dev, mob4, src, lens, 30, flags=mnmt.LOAD_PACKED_4BIT_ONLY)
    for cfg, B, n, seed in ((SMALL_POST, 2, [9, 4], 121), (DIVERSE, 2, [14, 11], 122), (SHARED, 1, [12], 123),
                            (WIDE512, 1, [20], 124), (WIDE384, 2, [25, 19], 125), (VARIED, 2, [30, 21], 126)):
        src, lens = G.make_sources(cfg.vocab, B, n, seed=seed, s_max=max(n))
        _greedy_check(torch, dev, cfg, src, lens, 12)


def test_merged_layers_many_sentences(torch_dev, monkeypatch):
    """Two dozen batch-1 sentences in graph replays through the one-launch
    step against the per-layer launches and the three-kernel layers (all on
    the counted hand-off), the first four also against the oracle."""
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    om, gm = _pair("MOBILE")
    rng = np.random.default_rng(2025)
    lens_all = rng.integers(10, 31, 24)
    outs = {}
    for form, env in LAUNCH_FORMS.items():
        monkeypatch.setenv("MNMT_STEP_LAUNCH", env.get("MNMT_STEP_LAUNCH", "0"))
        monkeypatch.setenv("MNMT_MERGED_LAYERS", env.get("MNMT_MERGED_LAYERS", "1"))
        sess = mnmt.Session(gm, 1, 30, 30, 1)
        got = []
        for k, n in enumerate(lens_all):
            src, lens = G.make_sources(G.MOBILE.vocab, 1, [int(n)], seed=700 + k, s_max=30)
            out, out_len, _ = sess.translate(_t(torch, dev, src), _t(torch, dev, lens), beam=1, max_steps=30,
                                             use_graph=True)
            torch.cuda.synchronize()
            got.append((out.cpu().numpy().copy(), out_len.cpu().numpy().copy()))
            if form == "step" and k < 4:
                o_out, o_len = om.greedy(src, lens, 30)[:2]
                assert np.array_equal(got[-1][0], o_out) and np.array_equal(got[-1][1], o_len), f"sentence {k}"
        assert int(sess.tensor("chain_err", torch.int32, (1,)).cpu().numpy()[0]) == 0
        sess.close()
        outs[form] = got
    for other in ("layer", "three"):
        for k, (a, b) in enumerate(zip(outs[other], outs["step"])):
            assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]), f"{other}: sentence {k}"


@pytest.mark.parametrize("form", ["step", "layer"])
def test_many_translations_in_one_session(torch_dev, monkeypatch, form):
    """130 batch-1 translations of one sentence in one session, each alone
    in a graph replay: the tags that the chained step kernels hand off by
    (translation counter, step) wrap around more than once, and every
    translation must still equal the oracle's with no chain wait giving up
    (a tag that once coincided with that of the cleared slots derailed every
    64th translation)."""
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    for k, v in LAUNCH_FORMS[form].items():
        monkeypatch.setenv(k, v)
    om, gm = _pair("MOBILE")
    src, lens = G.workload_inputs(G.WORKLOADS["mobile"])
    o_out, o_len = om.greedy(src, lens, 30)[:2]
    sess = mnmt.Session(gm, 1, 30, 30, 1)
    ts, tl = _t(torch, dev, src), _t(torch, dev, lens)
    err = sess.tensor("chain_err", torch.int32, (1,))
    for k in range(130):
        out, out_len, _ = sess.translate(ts, tl, beam=1, max_steps=30, use_graph=True)
        torch.cuda.synchronize()
        assert int(err.cpu().numpy()[0]) == 0, f"translation {k}: a chained wait gave up"
        assert np.array_equal(out.cpu().numpy(), o_out) and np.array_equal(out_len.cpu().numpy(), o_len), k
    sess.status()
    sess.close()


WIDE384 = G.ModelConfig("wide-384", 384, 6, 768, 2, 1, 600, ln_post=0, seed=83, random_gamma=True, weight_std=0.05)
WIDE512 = G.ModelConfig("wide-512", 512, 8, 1024, 2, 1, 600, ln_post=0, seed=84, random_gamma=True, weight_std=0.05)


def test_small_encoder_wide_models(torch_dev):
    """The batch-1 encoder kernels at widths 384 (two sentences, 50 rows: 8 rows
    per wave, attention within each sentence) and 512 (one sentence of 20)."""
    torch, dev = torch_dev
    src, lens = G.make_sources(WIDE384.vocab, 2, [25, 19], seed=41, s_max=25)
    _greedy_check(torch, dev, WIDE384, src, lens, 8)
    src, lens = G.make_sources(WIDE512.vocab, 1, [20], seed=42, s_max=20)
    _greedy_check(torch, dev, WIDE512, src, lens, 8)


@pytest.mark.parametrize("cfg", [G.PAPER_10MB, G.PAPER_20MB], ids=lambda c: c.name)
def test_paper_model_shapes_greedy(torch_dev, cfg):
    """The paper's MobileNMT-10MB / 20MB settings (vocabulary 8000, width 256 /
    384, 4 / 6 heads of 64, FFN 512 / 768, 12 + 2 layers): batch 1, 30 source
    tokens, 30 greedy steps, tokens and logits against the oracle."""
    torch, dev = torch_dev
    src, lens = G.make_sources(cfg.vocab, 1, [30], seed=2010 + cfg.d_model, s_max=30)
    _greedy_check(torch, dev, cfg, src, lens, 30)


def _beam_check(torch, dev, cfg, src, lens, W, steps, alpha, sample=None, parallel=False, flags=0):
    from paper_2306_04235_amd import mnmt

    from .oracle_pool import beam_many

    om, gm = _pair(cfg, flags)
    B, S = src.shape
    print(f"beam {cfg if isinstance(cfg, str) else cfg.name} B={B} S={S} W={W} T={steps}", flush=True)
    sess = mnmt.Session(gm, B, S, steps, W)
    ts, tl = _t(torch, dev, src), _t(torch, dev, lens)
    results = []
    for use_graph in (False, True):
        out, out_len, score = sess.translate(ts, tl, beam=W, max_steps=steps, alpha=alpha, use_graph=use_graph)
        torch.cuda.synchronize()
        results.append((out.cpu().numpy(), out_len.cpu().numpy(), score.cpu().numpy()))
    assert all(np.array_equal(results[0][i], results[1][i]) for i in range(3)), "graph replay differs from eager"
    out, out_len, score = results[0]
    idx = np.arange(B) if sample is None else np.asarray(sample)
    if parallel:  # one oracle process per sentence, up to 16 at a time
        mcfg = getattr(G, cfg) if isinstance(cfg, str) else cfg
        o_out, o_len, o_score = beam_many(mcfg, src, lens, idx, W, steps, alpha)
    else:
        o_out, o_len, o_score = om.beam(src[idx], lens[idx], W, steps, alpha)
    assert np.array_equal(out_len[idx], o_len)
    assert np.array_equal(out[idx], o_out)
    assert np.array_equal(score[idx].view(np.uint32), o_score.view(np.uint32))
    sess.close()


VARIED_BEAM = G.ModelConfig("varied-256-beam", 256, 4, 1024, 2, 2, 2000, ln_post=0, seed=1104, random_gamma=True,
                            weight_std=0.2)


# a long feed-forward (K 2048): W2's split partial sums are added by the next
# layer's fused self-attention prologue, which stores the updated rows into
# the second residual buffer
SPLIT_BEAM = G.ModelConfig("split-preln-beam", 128, 4, 2048, 2, 3, 700, ln_post=0, seed=94, random_gamma=True,
                           weight_std=0.1)


@pytest.mark.parametrize("cfg", [DIVERSE, VARIED_BEAM, SPLIT_BEAM], ids=lambda c: c.name)
def test_batched_layernorm_forms(torch_dev, monkeypatch, cfg):
    """Pre-LN beam search above 64 rows (19 sentences of beam 4: 76 rows, a
    ragged last tile of 16 rows): the LayerNorms in the prologue of the
    kernels they feed (each block of the one-round-trip GEMM normalizes its
    rows) and, with MNMT_LN_FUSED=0 (read at session creation), as kernels of
    their own; the self-attention computing its rows' Q/K/V and, with
    MNMT_QKV_FUSED=0, the projection as a GEMM; the fused self-attention's
    128- and 256-position classes over 100 and 200 steps; every sentence
    against the oracle."""
    torch, dev = torch_dev
    src, lens = G.make_sources(cfg.vocab, 19, (2, 24), seed=97, s_max=24)
    for fused in ("1", "0"):
        monkeypatch.setenv("MNMT_LN_FUSED", fused)
        _beam_check(torch, dev, cfg, src, lens, 4, 12, 0.6, parallel=True)
    monkeypatch.setenv("MNMT_LN_FUSED", "1")
    monkeypatch.setenv("MNMT_QKV_FUSED", "0")
    _beam_check(torch, dev, cfg, src, lens, 4, 12, 0.6, parallel=True)
    monkeypatch.setenv("MNMT_QKV_FUSED", "1")
    # eight hypotheses per sentence (two rows per wave in the fused
    # self-attention, the K > 8 bound of the top-k), 9 sentences (72 rows)
    src8, lens8 = G.make_sources(cfg.vocab, 9, (2, 24), seed=96, s_max=24)
    _beam_check(torch, dev, cfg, src8, lens8, 8, 12, 0.6, parallel=True)
    # two and six hypotheses per sentence above 64 rows (40 and 12 sentences)
    src2, lens2 = G.make_sources(cfg.vocab, 40, (2, 24), seed=95, s_max=24)
    _beam_check(torch, dev, cfg, src2, lens2, 2, 12, 0.6, parallel=True)
    src6, lens6 = G.make_sources(cfg.vocab, 12, (2, 24), seed=94, s_max=24)
    _beam_check(torch, dev, cfg, src6, lens6, 6, 12, 0.6, parallel=True)
    # the longer key-length classes of the fused self-attention (up to 128 and
    # 256 target positions), 17 sentences (68 rows)
    src, lens = G.make_sources(cfg.vocab, 17, (1, 40), seed=98, s_max=40)
    for steps in (100, 200):
        _beam_check(torch, dev, cfg, src, lens, 4, steps, 0.6, parallel=True)


# models whose EOS row of the embedding is drawn larger, so that hypotheses
# and greedy sentences end at varied steps (the search's end-of-sentence
# rules: finished hypotheses, length penalty, finished sentences skipped)
VARIED_EOS = dataclasses.replace(VARIED_BEAM, name="varied-256-eos", eos_gain=3.0)
DIVERSE_EOS = dataclasses.replace(DIVERSE, name="diverse-eos", eos_gain=4.0)


def test_end_of_sentence_search(torch_dev):
    """Beam search and greedy search with stop_at_eos on models that emit EOS
    at varied steps (the oracle's lengths range from 1 to the maximum):
    batched beam above and below 64 rows (the fused and the general batched
    decoder), small-model beam at widths 2, 4, 6, and greedy at 1, 2 and 5
    rows (the chained batch-1 step, the 2-row and the 3-8-row paths)."""
    torch, dev = torch_dev
    src, lens = G.make_sources(VARIED_EOS.vocab, 19, (2, 24), seed=97, s_max=24)
    for W in (4, 2):
        _beam_check(torch, dev, VARIED_EOS, src, lens, W, 20, 0.6, parallel=True)
    src, lens = G.make_sources(DIVERSE_EOS.vocab, 4, [5, 1, 9, 9], seed=31, s_max=9)
    for W in (2, 4, 6):
        _beam_check(torch, dev, DIVERSE_EOS, src, lens, W, 16, 0.6)
    for B, seed in ((1, 45), (1, 48), (2, 42), (5, 45)):
        src, lens = G.make_sources(VARIED_EOS.vocab, B, (3, 30), seed=seed, s_max=30)
        _greedy_check(torch, dev, VARIED_EOS, src, lens, 20, stop_at_eos=True, check_logits=False)
    # the oracle's lengths do vary (the test exercises the end-of-sentence rules)
    om, _ = _pair(VARIED_EOS)
    src, lens = G.make_sources(VARIED_EOS.vocab, 19, (2, 24), seed=97, s_max=24)
    _, o_len, _ = om.beam(src[:6], lens[:6], 4, 20, 0.6)
    assert o_len.min() < 20 and o_len.max() > 1


HEAD16 = G.ModelConfig("head-16", 128, 8, 256, 1, 1, 600, ln_post=0, seed=88, random_gamma=True, weight_std=0.1)
HEAD128 = G.ModelConfig("head-128", 256, 2, 512, 1, 1, 600, ln_post=1, seed=89, random_gamma=True, weight_std=0.08)


@pytest.mark.parametrize("cfg", [HEAD16, HEAD128], ids=lambda c: c.name)
def test_attention_length_and_head_classes(torch_dev, cfg):
    """The batched attention kernels' length classes (64, 128, 256 keys) and
    head-width classes (16-64 and 128) against the oracle, up to the maximum
    lengths (256 source tokens, 256 target positions): greedy at 3 rows
    (batched encoder, 3-8-row decoder) and beam search at 8 rows, with a
    one-token source among long ones."""
    torch, dev = torch_dev
    src, lens = G.make_sources(cfg.vocab, 3, [256, 131, 1], seed=90, s_max=256)
    _greedy_check(torch, dev, cfg, src, lens, 200, check_logits=False)
    src, lens = G.make_sources(cfg.vocab, 3, [100, 65, 7], seed=91, s_max=100)
    _greedy_check(torch, dev, cfg, src, lens, 100)
    src, lens = G.make_sources(cfg.vocab, 2, [150, 1], seed=92, s_max=150)
    _beam_check(torch, dev, cfg, src, lens, 4, 140, 0.6)


def test_postln_beam_above_64_rows(torch_dev):
    """Post-LN beam search above 64 rows (the normalized rows replace the
    residual stream, so the batched decoder keeps its LayerNorm kernels):
    76 rows of a d-64 model on the one-wave 16x16 GEMM blocks, and 68 rows
    of a d-256 model with 128-wide heads, whose cross-attention computes its
    query rows itself, against the oracle on every sentence."""
    torch, dev = torch_dev
    src, lens = G.make_sources(SMALL_POST.vocab, 19, (2, 24), seed=99, s_max=24)
    _beam_check(torch, dev, SMALL_POST, src, lens, 4, 12, 0.6, parallel=True)
    src, lens = G.make_sources(HEAD128.vocab, 17, (2, 40), seed=100, s_max=40)
    _beam_check(torch, dev, HEAD128, src, lens, 4, 12, 0.6, parallel=True)


ODD_VOCAB = G.ModelConfig("odd-vocab", 64, 4, 128, 1, 1, 501, ln_post=0, seed=79, random_gamma=True, weight_std=0.1)


def test_small_models_beam(torch_dev):
    torch, dev = torch_dev
    for cfg in (SMALL_PRE, SMALL_POST, DIVERSE, ODD_VOCAB):  # odd vocabulary: the one-wave-per-row top-k
        src, lens = G.make_sources(cfg.vocab, 4, [5, 1, 9, 9], seed=31, s_max=9)
        for W in (2, 4, 6):
            _beam_check(torch, dev, cfg, src, lens, W, 8, 0.6)


TIES3 = G.ModelConfig("ties-3", 64, 4, 128, 1, 1, 3000, ln_post=0, seed=86, emb_distinct=3)
TIES1 = G.ModelConfig("ties-1", 64, 4, 128, 1, 1, 2048, ln_post=0, seed=87, emb_distinct=1)


def test_beam_tied_logits(torch_dev):
    """Embedding rows repeated so the logits come in groups of equal values:
    1000 equal best scores per row (the filtered top-k list near its 1024
    capacity) and 2048 (every score equal: the overflow path).  Ties go to the
    lower flat index on both sides."""
    torch, dev = torch_dev
    for cfg in (TIES3, TIES1):
        src, lens = G.make_sources(cfg.vocab, 3, [6, 2, 7], seed=33, s_max=7)
        for W in (2, 4, 8):
            _beam_check(torch, dev, cfg, src, lens, W, 6, 0.6)


def test_4bit_weight_models(torch_dev):
    """The paper's W-E-A 4-8-8 setting (4-bit linear weights, 8-bit embedding
    and activations): batch-1 greedy on the mobile shape and on a small model,
    batched greedy and beam search on the small one, all against the oracle."""
    import dataclasses

    torch, dev = torch_dev
    mob4 = dataclasses.replace(G.MOBILE, name="mobile-w4", w_bits=4)
    src, lens = G.workload_inputs(G.WORKLOADS["mobile"])
    _greedy_check(torch, dev, mob4, src, lens, 30)
    div4 = dataclasses.replace(DIVERSE, name="diverse-w4", w_bits=4)
    src, lens = G.make_sources(div4.vocab, 1, [9], seed=31, s_max=9)
    _greedy_check(torch, dev, div4, src, lens, 10)
    src, lens = G.make_sources(div4.vocab, 3, [9, 5, 7], seed=31, s_max=9)
    _greedy_check(torch, dev, div4, src, lens, 10)
    _beam_check(torch, dev, div4, src, lens, 2, 8, 0.6)


def test_4bit_packed_only_models(torch_dev):
    """MNMT_LOAD_PACKED_4BIT_ONLY: the 4-bit weights stay packed on the device
    (half the int8 model's linear-weight bytes) and the batch-1 decoder and
    small-batch encoder kernels widen them in registers: per-step logits and
    tokens equal the oracle's on the mobile shape and on the varied model at
    one and two rows."""
    import dataclasses

    from paper_2306_04235_amd import mnmt

    torch, dev = torch_dev
    mob4 = dataclasses.replace(G.MOBILE, name="mobile-w4", w_bits=4)
    _, gm_full = _pair(mob4)
    _, gm = _pair(mob4, mnmt.LOAD_PACKED_4BIT_ONLY)
    _, gm8 = _pair("MOBILE")
    assert gm.arena.numel() < gm8.arena.numel() < gm_full.arena.numel()
    src, lens = G.workload_inputs(G.WORKLOADS["mobile"])
    _greedy_check(torch, dev, mob4, src, lens, 30, flags=mnmt.LOAD_PACKED_4BIT_ONLY)
    var4 = dataclasses.replace(VARIED, name="varied-w4", w_bits=4)
    for B in (1, 2):
        src, lens = G.make_sources(var4.vocab, B, [30, 21][:B], seed=95 + B, s_max=30)
        out = _greedy_check(torch, dev, var4, src, lens, 30, flags=mnmt.LOAD_PACKED_4BIT_ONLY)
        assert len(set(out[0].tolist())) >= 3


def test_4bit_packed_only_batched_paths(torch_dev):
    """Packed-only 4-bit models on the batched paths, which then read the
    packed rows too: 3-row greedy steps (the fused GEMV), beam search on a
    small model, and the mobile beam workload (64 sentences of 10-60 tokens:
    the encoder's 3840-row projections on the tiled GEMM, the 256-row beam
    decoder on the one-wave matrix-core blocks), a dozen sentences of it
    against the oracle, shortest and longest included."""
    from paper_2306_04235_amd import mnmt

    torch, dev = torch_dev
    flags = mnmt.LOAD_PACKED_4BIT_ONLY
    div4 = dataclasses.replace(DIVERSE, name="diverse-w4", w_bits=4)
    src, lens = G.make_sources(div4.vocab, 3, [9, 5, 7], seed=31, s_max=9)
    _greedy_check(torch, dev, div4, src, lens, 10, flags=flags)
    _beam_check(torch, dev, div4, src, lens, 2, 8, 0.6, flags=flags)
    src, lens = G.make_sources(div4.vocab, 12, [9, 5, 7, 16, 3, 11, 8, 8, 2, 16, 12, 6], seed=32, s_max=16)
    _greedy_check(torch, dev, div4, src, lens, 6, flags=flags)
    # above 64 rows at d 128: the fused self-attention on packed W_qkv rows
    src, lens = G.make_sources(div4.vocab, 19, (2, 16), seed=34, s_max=16)
    _beam_check(torch, dev, div4, src, lens, 4, 10, 0.6, parallel=True, flags=flags)
    mob4 = dataclasses.replace(G.MOBILE, name="mobile-w4", w_bits=4)
    w = G.WORKLOADS["mobile_beam"]
    src, lens = G.workload_inputs(w)
    order = np.argsort(lens, kind="stable")
    idx = sorted({int(order[0]), int(order[-1]), *range(0, 64, 6)})
    _beam_check(torch, dev, mob4, src, lens, w.beam, w.steps, w.alpha, sample=idx, parallel=True, flags=flags)


SPLIT_PRE = G.ModelConfig("split-preln", 128, 4, 2048, 2, 2, 700, ln_post=0, seed=91, random_gamma=True,
                          weight_std=0.1)
SPLIT_POST = G.ModelConfig("split-postln", 64, 2, 1536, 1, 2, 500, ln_post=1, seed=92, random_gamma=True,
                           weight_std=0.1)


@pytest.mark.parametrize("cfg", [SPLIT_PRE, SPLIT_POST], ids=lambda c: c.name)
def test_split_k_feed_forward(torch_dev, cfg):
    """Feed-forward widths of 1536 and 2048 in the batched decoder: W2's K is
    split over blocks whose int32 partial sums the next LayerNorm kernel adds
    before the residual update (pre-LN with gamma != 1: the updated rows are
    stored, post-LN: the normalized rows replace them; the final LayerNorm
    too).  Batched greedy (12 rows) and beam search against the oracle, and
    the same with packed 4-bit weights."""
    from paper_2306_04235_amd import mnmt

    torch, dev = torch_dev
    src, lens = G.make_sources(cfg.vocab, 12, [9, 5, 7, 16, 3, 11, 8, 8, 2, 16, 12, 6], seed=93, s_max=16)
    _greedy_check(torch, dev, cfg, src, lens, 8)
    _beam_check(torch, dev, cfg, src[:5], lens[:5], 4, 8, 0.6)
    c4 = dataclasses.replace(cfg, name=cfg.name + "-w4", w_bits=4)
    _beam_check(torch, dev, c4, src[:5], lens[:5], 4, 8, 0.6, flags=mnmt.LOAD_PACKED_4BIT_ONLY)


SHARED = G.ModelConfig("shared-preln", 64, 4, 128, 4, 3, 500, ln_post=0, seed=82, random_gamma=True,
                       weight_std=0.1, share_every=1)
SHARED_256 = G.ModelConfig("shared-256", 256, 4, 1024, 6, 2, 32000, ln_post=0, seed=1103, random_gamma=True,
                           weight_std=0.2, share_every=2)


def test_cross_layer_sharing_models(torch_dev):
    """Cross-layer parameter sharing (Section 2.2): layers that reuse another
    layer's parameters (aliased device pointers, stored once) on every path --
    the batch-1 chained step and encoder, the 3-8 row and matrix-core paths,
    beam search -- against the oracle."""
    torch, dev = torch_dev
    for B in (1, 2, 5, 12):
        src, lens = G.make_sources(SHARED.vocab, B, (3, 12), seed=60 + B, s_max=12)
        _greedy_check(torch, dev, SHARED, src, lens, 9)
    src, lens = G.make_sources(SHARED.vocab, 4, [5, 1, 9, 9], seed=31, s_max=9)
    _beam_check(torch, dev, SHARED, src, lens, 4, 8, 0.6)
    src, lens = G.make_sources(SHARED_256.vocab, 1, [30], seed=64, s_max=30)
    _greedy_check(torch, dev, SHARED_256, src, lens, 30)


FACTOR = G.ModelConfig("factorized-256", 256, 4, 512, 2, 2, 2000, ln_post=0, seed=83, random_gamma=True,
                       weight_std=0.2, emb_dim=128)
FACTOR_POST = G.ModelConfig("factorized-post", 128, 2, 256, 2, 1, 700, ln_post=1, seed=84, weight_std=0.1,
                            emb_dim=64)


def test_factorized_embedding_models(torch_dev):
    """Embedding factorization (Section 2.1): rows of width E projected to the
    model width on the way in (k_embed_proj) and the final rows projected back
    (an int8 linear layer over the transposed matrix) before the tied logits,
    on the general greedy path at 1, 5 and 12 rows (per-step logits bits via
    mnmt_decode_step) and in beam search, against the oracle."""
    torch, dev = torch_dev
    for cfg in (FACTOR, FACTOR_POST):
        om, gm = _pair(cfg)
        assert gm.info.emb_dim == cfg.emb_dim and om.emb_dim == cfg.emb_dim
        for B in (1, 5, 12):
            src, lens = G.make_sources(cfg.vocab, B, (3, 16), seed=70 + B, s_max=16)
            _greedy_check(torch, dev, cfg, src, lens, 10)
        src, lens = G.make_sources(cfg.vocab, 4, [5, 1, 9, 9], seed=31, s_max=9)
        _beam_check(torch, dev, cfg, src, lens, 4, 8, 0.6)


def test_mobile_beam_workload_all_sentences(torch_dev):
    """The batched beam workload on the mobile model: all 64 sentences (10-60
    source tokens, beam 4, 64 steps) against the oracle, run one sentence per
    host process."""
    torch, dev = torch_dev
    w = G.WORKLOADS["mobile_beam"]
    src, lens = G.workload_inputs(w)
    _beam_check(torch, dev, "MOBILE", src, lens, w.beam, w.steps, w.alpha, parallel=True)


def test_base_beam_workload_sentences(torch_dev):
    """The base-model beam workload (128 sentences of 20-64 tokens, beam 4, 80
    steps): the shortest and longest sources and 22 more spread over the
    batch, against the oracle in host processes."""
    torch, dev = torch_dev
    w = G.WORKLOADS["base_beam"]
    src, lens = G.workload_inputs(w)
    order = np.argsort(lens, kind="stable")
    idx = sorted({int(order[0]), int(order[-1]), *range(0, 128, 6)})
    assert len(idx) >= 16
    _beam_check(torch, dev, "BASE", src, lens, w.beam, w.steps, w.alpha, sample=idx, parallel=True)


VARIED = G.ModelConfig("varied-256", 256, 4, 1024, 2, 2, 32000, ln_post=0, seed=1102, random_gamma=True,
                       weight_std=0.2)


@pytest.mark.parametrize("B", [1, 2])
def test_varied_output_chained_translate(torch_dev, B):
    """The path the latency benchmark times -- width 256, vocabulary 32000, two
    decoder layers: the two-stream kernel chain, the commit folded into the
    next step and the 4-tile logits kernel of the chain, replayed from a graph
    -- on a model whose greedy outputs vary from step to step (the workload
    model repeats its input token), against the oracle's tokens and the bits
    of every step's maximum logit."""
    torch, dev = torch_dev
    src, lens = G.make_sources(VARIED.vocab, B, [30, 17][:B], seed=90 + B, s_max=30)
    out = _greedy_check(torch, dev, VARIED, src, lens, 30)
    for b in range(B):
        assert len(set(out[b].tolist())) >= 4, "the varied model should not repeat one token"


def test_beam_session_rejects_decode_step(torch_dev):
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    _, gm = _pair("TINY")
    sess = mnmt.Session(gm, 2, 8, 4, 2)
    src = torch.full((2, 8), 5, dtype=torch.int32, device=dev)
    lens = torch.full((2,), 8, dtype=torch.int32, device=dev)
    sess.encode(src, lens)
    with pytest.raises(mnmt.MnmtError) as e:
        sess.decode_step()
    assert e.value.status == mnmt.E_UNSUPPORTED
    sess.close()


def test_chain_error_word_marks_outputs(torch_dev):
    """A chained kernel whose bounded wait gives up sets the session's error
    word; here the host sets that word itself (no kernel waits in vain).  The
    next translations report length -1 until mnmt_session_status raises
    E_TIMEOUT and clears it."""
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    om, gm = _pair("TINY")
    src, lens = G.workload_inputs(G.WORKLOADS["tiny"])
    o_out, o_len = om.greedy(src, lens, 16)
    sess = mnmt.Session(gm, 1, src.shape[1], 16, 1)
    ts, tl = _t(torch, dev, src), _t(torch, dev, lens)
    sess.status()
    err = sess.tensor("chain_err", torch.int32, (1,))
    err.fill_(1)
    torch.cuda.synchronize()
    for use_graph in (False, True):
        out, out_len, _ = sess.translate(ts, tl, beam=1, max_steps=16, use_graph=use_graph)
        torch.cuda.synchronize()
        assert int(out_len.cpu()[0]) == -1
    with pytest.raises(mnmt.MnmtError) as e:
        sess.status()
    assert e.value.status == mnmt.E_TIMEOUT
    out, out_len, _ = sess.translate(ts, tl, beam=1, max_steps=16, use_graph=True)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy(), o_out) and np.array_equal(out_len.cpu().numpy(), o_len)
    sess.status()
    sess.close()


def test_session_capacity_errors(torch_dev):
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    _, gm = _pair("TINY")
    sess = mnmt.Session(gm, 2, 8, 4, 1)
    src = torch.full((3, 8), 5, dtype=torch.int32, device=dev)
    lens = torch.full((3,), 8, dtype=torch.int32, device=dev)
    with pytest.raises(mnmt.MnmtError) as e:
        sess.translate(src, lens, max_steps=4)
    assert e.value.status == mnmt.E_CAPACITY
    with pytest.raises(mnmt.MnmtError) as e:
        sess.translate(src[:2], lens[:2], max_steps=5)
    assert e.value.status == mnmt.E_CAPACITY
    with pytest.raises(mnmt.MnmtError) as e:
        mnmt.Session(gm, 1, 8, 4, 9)  # beam above the supported width
    assert e.value.status == mnmt.E_INVALID_ARG
    sess.encode(src[:1], lens[:1])
    for _ in range(4):
        sess.decode_step()
    with pytest.raises(mnmt.MnmtError) as e:
        sess.decode_step()
    assert e.value.status == mnmt.E_CAPACITY
    sess.close()
