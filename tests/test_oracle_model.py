"""Model-level pins for the oracle: cache vs cache-free decoding, batch
invariance, beam search against greedy and against exhaustive search, the
paper's closed-form sizes, model-file validation and input statistics."""
import dataclasses
import itertools
import os

import numpy as np
import pytest

import oracle
from paper_2306_04235_amd import workload as W
from synth import generate as G
from synth.modelfile import read_model, write_model

from .conftest import model_blob

# A pre-LN model small enough for exhaustive checks, with gamma != 1.
SMALL_PRE = G.ModelConfig("small-preln", 64, 4, 128, 2, 2, 500, ln_post=0, seed=77, random_gamma=True)
SMALL_POST = G.ModelConfig("small-postln", 64, 2, 128, 2, 2, 300, ln_post=1, seed=78, random_gamma=True,
                           weight_std=0.1)
MICRO = G.ModelConfig("micro-v6", 16, 2, 32, 1, 1, 6, ln_post=0, seed=79, weight_std=0.3, emb_std=0.3)


@pytest.fixture(scope="module")
def small_pre():
    return oracle.Model(G.build_model(SMALL_PRE))


@pytest.fixture(scope="module")
def small_post():
    return oracle.Model(G.build_model(SMALL_POST))


@pytest.mark.parametrize("which", ["small_pre", "small_post"])
def test_cached_decoding_equals_cache_free_causal_block(which, request):
    m = request.getfixturevalue(which)
    src, lens = G.make_sources(m.V, 3, (4, 12), seed=5)
    rng = np.random.default_rng(1)
    for b in range(3):
        toks = rng.integers(0, m.V, size=9).astype(np.int32)
        row = src[b, : lens[b]]
        z_inc = m.decoder_logits(row, toks)
        z_full = m.decoder_logits_full(row, toks)
        assert np.array_equal(z_inc, z_full)


def test_tiny_cached_equals_cache_free():
    m = oracle.Model(model_blob("TINY"))
    src, lens = G.workload_inputs(G.WORKLOADS["tiny"])
    toks = np.arange(4, 20, dtype=np.int32)
    assert np.array_equal(m.decoder_logits(src[0], toks), m.decoder_logits_full(src[0], toks))


def test_greedy_follows_its_own_logits(small_pre):
    m = small_pre
    src, lens = G.make_sources(m.V, 2, (5, 9), seed=6)
    out, out_len, logits = m.greedy(src, lens, 10, want_logits=True)
    for b in range(2):
        for t in range(10):
            z = logits[b, t]
            assert out[b, t] == int(np.argmax(z))  # numpy argmax: first maximum
        # teacher forcing with the greedy output reproduces the same logits
        z_tf = m.decoder_logits(src[b, : lens[b]], out[b])
        assert np.array_equal(z_tf, logits[b])


def test_batch_invariance_and_padding(small_pre):
    m = small_pre
    src, lens = G.make_sources(m.V, 4, [3, 9, 1, 6], seed=7, s_max=12)
    enc = m.encode(src, lens)
    out, out_len = m.greedy(src, lens, 8)
    bo, bl, bs = m.beam(src, lens, 3, 8)
    for b in range(4):
        one = src[b: b + 1, : lens[b]]
        e1 = m.encode(one, lens[b: b + 1])
        assert np.array_equal(enc[b, : lens[b]], e1[0])
        assert not enc[b, lens[b]:].any()
        o1, _ = m.greedy(one, lens[b: b + 1], 8)
        assert np.array_equal(out[b], o1[0])
        p1, l1, s1 = m.beam(one, lens[b: b + 1], 3, 8)
        assert np.array_equal(bo[b], p1[0]) and bl[b] == l1[0] and bs[b] == s1[0]


def test_beam_width_one_is_greedy(small_post):
    m = small_post
    src, lens = G.make_sources(m.V, 4, (3, 10), seed=8)
    g, gl = m.greedy(src, lens, 12, stop_at_eos=True)
    b, bl, _ = m.beam(src, lens, 1, 12)
    assert np.array_equal(gl, bl)
    for i in range(4):
        assert np.array_equal(g[i, : gl[i]], b[i, : bl[i]])


def _seq_score(m, row, seq, alpha):
    """Teacher-forced fp32 score of a token sequence, accumulated as the
    search does: s = s + (z[v] - lse) per step, then s / lp(len)."""
    z = m.decoder_logits(row, np.asarray(seq, np.int32))
    s = np.float32(0.0)
    for t, v in enumerate(seq):
        _, lse = oracle.log_softmax_stats(z[t])
        s = np.float32(s + np.float32(z[t, v] - lse))
    return np.float32(s / oracle.length_penalty(len(seq), alpha))


def test_beam_equals_exhaustive_search_on_micro_model():
    m = oracle.Model(G.build_model(MICRO))
    assert m.V == 6
    T, alpha = 3, 0.6
    non_eos = [v for v in range(m.V) if v != m.eos_id]
    src, lens = G.make_sources(m.V, 2, (2, 4), seed=9)
    for b in range(2):
        row = src[b, : lens[b]]
        cands = []
        for L in range(1, T + 1):  # EOS-terminated hypotheses of every length
            for pre in itertools.product(non_eos, repeat=L - 1):
                cands.append(list(pre) + [m.eos_id])
        for full in itertools.product(non_eos, repeat=T):  # unfinished at the last step
            cands.append(list(full))
        scores = np.array([_seq_score(m, row, c, alpha) for c in cands], np.float32)
        best = int(np.argmax(scores))
        assert (scores == scores[best]).sum() == 1
        out, out_len, score = m.beam(src[b: b + 1, : lens[b]], lens[b: b + 1], 150, T, alpha)
        assert list(out[0, : out_len[0]]) == cands[best]
        assert score[0] == scores[best]


def test_beam_scores_are_normalized_sequence_scores(small_pre):
    m = small_pre
    src, lens = G.make_sources(m.V, 3, (4, 9), seed=10)
    out, out_len, score = m.beam(src, lens, 4, 10, 0.6)
    for b in range(3):
        seq = out[b, : out_len[b]]
        assert score[b] == _seq_score(m, src[b, : lens[b]], seq, 0.6)
        assert np.all(out[b, out_len[b]:] == m.pad_id)


def _paper_rows():
    path = os.path.join(os.path.dirname(__file__), "golden", "paper_sizes.txt")
    with open(path) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


@pytest.mark.parametrize("row", _paper_rows(), ids=lambda r: r[0])
def test_paper_parameter_and_mac_counts(row):
    name, d, h, F, le, ld, V, p_m, p_wo_m, flops_g, tol_m, tol_g = row
    d, h, F, le, ld, V = map(int, (d, h, F, le, ld, V))
    dims = W.Dims(d, h, F, le, ld, V)
    with_e, without_e = W.param_counts(dims)
    assert abs(with_e / 1e6 - float(p_m)) <= float(tol_m)
    assert abs(without_e / 1e6 - float(p_wo_m)) <= float(tol_m)
    assert abs(W.sentence_macs(dims, 30, 30) / 1e9 - float(flops_g)) <= float(tol_g)
    # the model files the engine loads hold exactly these weight matrices
    cfg = G.ModelConfig(name, d, h, F, le, ld, V, ln_post=0, seed=3)
    _, t = read_model(G.build_model(cfg))
    n_w = sum(a.size for k, a in t.items() if k.endswith(".w") and a.dtype == np.int8)
    assert n_w == with_e
    assert n_w - t["emb.w"].size == without_e


def test_model_file_validation():
    blob = model_blob("TINY")
    oracle.Model(blob)  # loads
    bad = bytearray(blob)
    bad[0:4] = b"XXXX"
    with pytest.raises(RuntimeError):
        oracle.Model(bytes(bad))
    with pytest.raises(RuntimeError):
        oracle.Model(blob[: len(blob) // 2])  # truncated payload
    hdr, t = read_model(blob)
    t = dict(t)
    del t["dec.0.ca.kv.sout"]
    with pytest.raises(RuntimeError):
        oracle.Model(write_model(hdr, t))
    hdr2, t2 = read_model(blob)
    t2 = dict(t2)
    t2["enc.0.sa.qkv.sin"] = np.array([-1.0], np.float32)  # non-positive scale
    with pytest.raises(RuntimeError):
        oracle.Model(write_model(hdr2, t2))


def test_generator_is_deterministic():
    assert G.build_model(G.TINY) == model_blob("TINY")
    a = G.workload_inputs(G.WORKLOADS["mobile_beam"])
    b = G.workload_inputs(G.WORKLOADS["mobile_beam"])
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert a[1].min() >= 10 and a[1].max() <= 60
    assert a[0][a[0] > 0].min() >= 4


def test_activation_statistics_are_not_degenerate():
    for name, wl in (("TINY", "tiny"), ("MOBILE", "mobile")):
        m = oracle.Model(model_blob(name))
        src, lens = G.make_sources(m.V, 2, 20, seed=11)
        enc = m.encode(src, lens)
        kv = m.cross_kv(enc, lens, 0)
        for codes in (enc, kv):
            assert (np.abs(codes) == 127).mean() < 0.01
            assert (codes == 0).mean() < 0.5
            assert codes.std() > 5


def test_4bit_weights_quantizer_and_packing():
    """The paper's W-E-A 4-8-8 setting: per-row symmetric 4-bit codes in
    [-7, 7] with s = max|w| / 7, stored packed two codes per byte.  The
    quantizer reproduces each weight within half a step, the extreme of every
    row maps to +-7, and the packing round-trips."""
    from synth.generate import _quantize_rows
    from synth.modelfile import pack_int4, unpack_int4

    rng = np.random.default_rng(41)
    w = rng.normal(0.0, 0.02, size=(48, 64))
    codes, s = _quantize_rows(w, 7)
    assert codes.min() >= -7 and codes.max() <= 7
    assert np.all(np.abs(codes).max(axis=1) == 7)
    assert np.all(np.abs(codes * s[:, None].astype(np.float64) - w) <= s[:, None] / 2 * (1 + 1e-6))
    assert np.array_equal(unpack_int4(pack_int4(codes), 48, 64), codes)
    # the byte layout: byte i of a 16-code group holds codes i and i + 8, plus 8
    one = np.arange(-7, 9, dtype=np.int8)[None, :16].clip(-7, 7)
    packed = np.frombuffer(pack_int4(one), np.uint8)
    assert [int(b) for b in packed] == [int(one[0, i] + 8) | (int(one[0, i + 8] + 8) << 4) for i in range(8)]


def test_4bit_model_equals_its_int8_form():
    """A model stored with 4-bit weights translates exactly as the same codes
    stored as int8 (the oracle unpacks; nothing after the GEMM changes)."""
    import dataclasses

    from synth.modelfile import read_model, write_model

    cfg = dataclasses.replace(G.TINY, name="tiny-w4", w_bits=4, seed=1101)
    blob4 = G.build_model(cfg)
    hdr, t = read_model(blob4)
    blob8 = write_model(hdr, {k: np.ascontiguousarray(v) for k, v in t.items()})
    src, lens = G.make_sources(cfg.vocab, 2, [9, 5], seed=7, s_max=9)
    a = oracle.Model(blob4).greedy(src, lens, 10, want_logits=True)
    b = oracle.Model(blob8).greedy(src, lens, 10, want_logits=True)
    assert np.array_equal(a[0], b[0])
    assert np.array_equal(a[2].view(np.uint32), b[2].view(np.uint32))


SHARED = G.ModelConfig("shared-preln", 64, 4, 128, 4, 3, 500, ln_post=0, seed=82, random_gamma=True,
                       weight_std=0.1, share_every=1)


def _unshare(blob):
    """The same model with every shared layer's tensors written out in full."""
    hdr, t = read_model(blob)
    out = {k: np.ascontiguousarray(v) for k, v in t.items() if not k.endswith(".share")}
    for k, v in t.items():
        if not k.endswith(".share"):
            continue
        side, l = k.split(".")[:2]
        src = f"{side}.{int(v[0])}."
        for name, arr in t.items():
            if name.startswith(src) and not name.endswith(".share"):
                out[f"{side}.{l}." + name[len(src):]] = np.ascontiguousarray(arr)
    return write_model(hdr, out)


def test_cross_layer_sharing_equals_written_out_layers():
    """Cross-layer parameter sharing (Section 2.2, Encoder/Decoder Compression)
    is a storage form: a file whose layers 1.. reuse layer 0 translates bit for
    bit like the file with those parameters copied into every layer."""
    blob = G.build_model(SHARED)
    full = _unshare(blob)
    assert len(full) > len(blob)
    a, b = oracle.Model(blob), oracle.Model(full)
    src, lens = G.make_sources(SHARED.vocab, 3, [7, 3, 11], seed=4, s_max=11)
    ga, gb = a.greedy(src, lens, 9, want_logits=True), b.greedy(src, lens, 9, want_logits=True)
    assert np.array_equal(ga[0], gb[0]) and np.array_equal(ga[2].view(np.uint32), gb[2].view(np.uint32))
    ba, bb = a.beam(src, lens, 3, 8), b.beam(src, lens, 3, 8)
    assert all(np.array_equal(x, y) for x, y in zip(ba[:2], bb[:2]))
    assert np.array_equal(ba[2].view(np.uint32), bb[2].view(np.uint32))
    # the shared layers really are the same function: sharing changes the output
    # compared with the unshared model drawn from the same seed
    c = oracle.Model(G.build_model(dataclasses.replace(SHARED, share_every=0)))
    assert not np.array_equal(c.greedy(src, lens, 9, want_logits=True)[2], ga[2])


def test_cross_layer_sharing_rejects_forward_references():
    hdr, t = read_model(G.build_model(SHARED))
    for bad in (2, 5, -1):  # layer 2 may only name layers 0 and 1
        t2 = {k: np.ascontiguousarray(v) for k, v in t.items()}
        t2["enc.2.share"] = np.array([bad], np.int8)
        with pytest.raises(RuntimeError):
            oracle.Model(write_model(hdr, t2))
