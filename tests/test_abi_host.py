"""Host-side checks of the C ABI library that need no GPU: it loads, exports
every entry point declared in include/mnmt.h, and its host-only functions
(model validation, constant folding, status strings) behave."""
import os
import re

import numpy as np
import pytest

import oracle
from paper_2306_04235_amd import mnmt
from synth import generate as G
from synth.modelfile import read_model, write_model

from .conftest import ROOT, model_blob


def _declared():
    with open(os.path.join(ROOT, "include", "mnmt.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(mnmt_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = mnmt.lib()
    declared = _declared()
    assert set(declared) == set(mnmt.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name


def test_status_strings():
    L = mnmt.lib()
    assert L.mnmt_status_str(0) == b"ok"
    assert L.mnmt_status_str(mnmt.E_BAD_MODEL) == b"bad model file"
    assert L.mnmt_status_str(12345) == b"unknown status"


def test_model_bytes_accepts_the_generated_models():
    for name in ("TINY", "MOBILE"):
        blob = model_blob(name)
        n = mnmt.mnmt_model_bytes(blob)
        _, t = read_model(blob)
        weights = sum(a.size for k, a in t.items() if k.endswith(".w"))
        assert weights < n < 2 * len(blob)


def test_model_bytes_of_4bit_weights():
    """4-bit weights (the paper's W-E-A 4-8-8 setting): by default the arena
    holds their packed rows (read by the batch-1 decoder and small-batch
    encoder kernels) and their int8 codes (read by the batched kernels); with
    MNMT_LOAD_PACKED_4BIT_ONLY only the packed rows, half the bytes of the
    int8 model's linear weights.  An int8 model cannot be loaded that way."""
    import dataclasses

    from synth import generate as G

    blob4 = G.build_model(dataclasses.replace(G.TINY, name="tiny-w4", w_bits=4))
    hdr, t = read_model(blob4)
    blob8 = write_model(hdr, {k: np.ascontiguousarray(v) for k, v in t.items()})
    assert len(blob4) < len(blob8)
    lin = sum(v.size for k, v in t.items() if k.endswith(".w") and k != "emb.w")
    assert all((v.size // 2) % 256 == 0 for k, v in t.items() if k.endswith(".w") and k != "emb.w")
    b8 = mnmt.mnmt_model_bytes(blob8)
    assert mnmt.mnmt_model_bytes(blob4) == b8 + lin // 2
    assert mnmt.mnmt_model_bytes(blob4, mnmt.LOAD_PACKED_4BIT_ONLY) == b8 - lin // 2
    with pytest.raises(mnmt.MnmtError) as e:
        mnmt.mnmt_model_bytes(blob8, mnmt.LOAD_PACKED_4BIT_ONLY)
    assert e.value.status == mnmt.E_UNSUPPORTED
    with pytest.raises(mnmt.MnmtError) as e:
        mnmt.mnmt_model_bytes(blob4, 2)
    assert e.value.status == mnmt.E_INVALID_ARG


def test_model_bytes_rejects_bad_files():
    blob = model_blob("TINY")
    with pytest.raises(mnmt.MnmtError) as e:
        mnmt.mnmt_model_bytes(b"XXXX" + blob[4:])
    assert e.value.status == mnmt.E_BAD_MODEL
    with pytest.raises(mnmt.MnmtError) as e:
        mnmt.mnmt_model_bytes(blob[:1000])
    assert e.value.status == mnmt.E_BAD_MODEL
    hdr, t = read_model(blob)
    t = dict(t)
    t["dec.0.ff.w2.b"] = np.full(t["dec.0.ff.w2.b"].shape, np.nan, np.float32)
    with pytest.raises(mnmt.MnmtError) as e:
        mnmt.mnmt_model_bytes(write_model(hdr, t))
    assert e.value.status == mnmt.E_BAD_MODEL
    hdr.d_model = 48  # not a multiple of 64: shapes the kernels do not support
    with pytest.raises(mnmt.MnmtError) as e:
        mnmt.mnmt_model_bytes(write_model(hdr, dict(read_model(blob)[1])))
    assert e.value.status in (mnmt.E_UNSUPPORTED, mnmt.E_BAD_MODEL)


def test_fold_requant_matches_oracle_bitwise():
    rng = np.random.default_rng(4)
    for _ in range(5):
        s_w = rng.uniform(1e-5, 1e-2, 1000).astype(np.float32)
        b = rng.normal(0, 0.05, 1000).astype(np.float32)
        s_in, s_out = np.float32(rng.uniform(0.01, 0.05)), np.float32(rng.uniform(0.01, 0.2))
        a = mnmt.mnmt_fold_requant(s_in, s_w, b, s_out)
        r = oracle.fold_requant(s_in, s_w, b, s_out)
        assert np.array_equal(a[0].view(np.uint32), r[0].view(np.uint32))
        assert np.array_equal(a[1].view(np.uint32), r[1].view(np.uint32))


def test_packed_bytes_sizes():
    """The fragment-order copy of an int8 [N, K] weight takes whole 16-row
    tiles; sizes that cannot be packed give 0."""
    L = mnmt.lib()
    assert L.mnmt_packed_bytes(32000, 256) == 32000 * 256
    assert L.mnmt_packed_bytes(33, 64) == 48 * 64
    assert L.mnmt_packed_bytes(1, 512) == 16 * 512
    for N, K in ((0, 64), (-1, 64), (16, 0), (16, 100), (16, -64)):
        assert L.mnmt_packed_bytes(N, K) == 0


def test_model_arena_holds_the_packed_embedding():
    """The arena holds every weight plus the fragment-order copy of the tied
    embedding that the batch-1 logits kernel reads."""
    blob = model_blob("MOBILE")
    hdr, t = read_model(blob)
    V, d = np.asarray(t["emb.w"]).shape
    weights = sum(np.asarray(a).size for k, a in t.items() if k.endswith(".w"))
    assert mnmt.mnmt_model_bytes(blob) >= weights + mnmt.lib().mnmt_packed_bytes(V, d)


def test_shared_layers_are_stored_once():
    """Cross-layer parameter sharing: the arena holds a shared layer's
    parameters once; the loader rejects a layer that names itself or a later
    layer."""
    from tests.test_oracle_model import SHARED, _unshare

    blob = G.build_model(SHARED)
    full = _unshare(blob)
    per_layer_enc = 4 * 64 * 64 + 2 * 64 * 128
    assert mnmt.mnmt_model_bytes(full) - mnmt.mnmt_model_bytes(blob) >= (3 + 2) * per_layer_enc
    hdr, t = read_model(blob)
    t2 = {k: np.ascontiguousarray(v) for k, v in t.items()}
    t2["dec.1.share"] = np.array([1], np.int8)
    with pytest.raises(mnmt.MnmtError) as e:
        mnmt.mnmt_model_bytes(write_model(hdr, t2))
    assert e.value.status == mnmt.E_BAD_MODEL


def test_factorized_embedding_arena_and_validation():
    """A factorized embedding (Section 2.1) stores E [V, emb_dim], the
    projection [d, emb_dim] and its transpose; a projection whose width is not
    a multiple of 64 or exceeds d is rejected."""
    import dataclasses

    from tests.test_oracle_assembly import FACTOR

    blob = G.build_model(FACTOR)
    plain = G.build_model(dataclasses.replace(FACTOR, emb_dim=0))
    d, V, E = FACTOR.d_model, FACTOR.vocab, FACTOR.emb_dim
    # smaller embedding, no fragment-order copy, plus P and its transpose with E scales and biases
    assert mnmt.mnmt_model_bytes(plain) - mnmt.mnmt_model_bytes(blob) >= 2 * V * (d - E) - 2 * d * E - 4096
    hdr, t = read_model(blob)
    for bad in (np.zeros((d, 96), np.int8), np.zeros((d, 512), np.int8)):
        t2 = {k: np.ascontiguousarray(v) for k, v in t.items()}
        t2["emb.proj.w"] = bad
        t2["emb.w"] = np.zeros((V, bad.shape[1]), np.int8)
        with pytest.raises(mnmt.MnmtError) as e:
            mnmt.mnmt_model_bytes(write_model(hdr, t2))
        assert e.value.status == mnmt.E_BAD_MODEL
