"""Seeded synthetic models and inputs.

The paper's trained weights and its WMT14 data are not available, so every
model and every source batch here is drawn from a seeded numpy PCG64 stream.
The recipe:

* weights N(0, 0.02), quantized offline per output channel, symmetric:
  s_w[n] = max|W[n, :]| / 127, code = rint(W / s_w) (this is model
  preparation, the output of training; inference consumes the codes);
* the shared embedding E[V, d] is drawn and quantized the same way (per row);
* biases N(0, 0.02), LayerNorm gains N(1, 0.02), shifts N(0, 0.02);
* residual weights gamma = 1 unless ``random_gamma`` (then U[0.5, 1.5]);
* optional: cross-layer parameter sharing (``share_every``) and a factorized
  embedding (``emb_dim``: E [V, emb_dim] rows N(0, emb_std) and a [d, emb_dim]
  projection N(0, 1 / emb_dim) with one per-tensor scale);
* static per-tensor activation scales "drawn from the seed": each is
  4 sigma / 127 times U[0.9, 1.1], where sigma is the standard deviation the
  activation has under this weight distribution (1 for LayerNorm outputs,
  0.02 sqrt(fan_in) for projections of unit-variance inputs); the context
  scale equals the value scale, so the context never saturates;
* sinusoidal position table (sin on even, cos on odd columns), in float64,
  rounded once to float32;
* source ids uniform in [4, V) (0..3 are PAD, BOS, EOS, UNK), lengths per
  workload, right padded with PAD.

This module holds no inference arithmetic: it draws numbers and serializes.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .modelfile import Header, Int4Rows, write_model

WEIGHT_STD = 0.02
SPECIAL = 4  # ids 0..3 are PAD, BOS, EOS, UNK
EOS = 2


@dataclass(frozen=True)
class ModelConfig:
    name: str
    d_model: int
    n_heads: int
    d_ffn: int
    n_enc: int
    n_dec: int
    vocab: int
    ln_post: int
    max_pos: int = 256
    seed: int = 0
    random_gamma: bool = False
    emb_std: float = WEIGHT_STD
    gamma_range: tuple = (0.5, 1.5)
    weight_std: float = WEIGHT_STD
    emb_distinct: int = 0  # > 0: embedding row v repeats drawn row v mod emb_distinct (groups of equal logits)
    w_bits: int = 8  # 4: linear weights as 4-bit codes (the paper's W-E-A 4-8-8; the embedding stays 8-bit)
    share_every: int = 0  # > 0: layer l >= share_every reuses the parameters of layer l % share_every (per stack)
    emb_dim: int = 0  # > 0: factorized embedding [V, emb_dim] with a [d_model, emb_dim] projection
    eos_gain: float = 1.0  # the EOS row of the embedding drawn this many times larger (its tied logit too)


# The model shapes of the five workloads.
TINY = ModelConfig("tiny-postln", 64, 4, 256, 1, 1, 1000, ln_post=1, seed=1001)
MOBILE = ModelConfig("mobile-12-2", 256, 4, 1024, 12, 2, 32000, ln_post=0, seed=1002)
BASE = ModelConfig("base-6-6", 512, 8, 2048, 6, 6, 32000, ln_post=0, seed=1005)
# The paper's own MobileNMT-10MB / 20MB shapes (model-settings table).
PAPER_10MB = ModelConfig("mobilenmt-10mb", 256, 4, 512, 12, 2, 8000, ln_post=0, seed=1010)
PAPER_20MB = ModelConfig("mobilenmt-20mb", 384, 6, 768, 12, 2, 8000, ln_post=0, seed=1020)


def _quantize_rows(w: np.ndarray, qmax: int = 127) -> tuple[np.ndarray, np.ndarray]:
    """Per-row symmetric codes in [-qmax, qmax] and float32 scales (offline
    preparation): 127 for 8-bit, 7 for 4-bit weights."""
    amax = np.abs(w).max(axis=1)
    s = np.where(amax > 0, amax / float(qmax), 1.0)
    codes = np.clip(np.rint(w / s[:, None]), -qmax, qmax).astype(np.int8)
    return codes, s.astype(np.float32)


def _act_scale(rng: np.random.Generator, sigma: float) -> np.float32:
    return np.float32(4.0 * sigma / 127.0 * rng.uniform(0.9, 1.1))


def positional_table(max_pos: int, d: int) -> np.ndarray:
    pos = np.arange(max_pos, dtype=np.float64)[:, None]
    i = np.arange(0, d, 2, dtype=np.float64)[None, :]
    ang = pos / np.power(10000.0, i / d)
    pe = np.zeros((max_pos, d), dtype=np.float64)
    pe[:, 0::2] = np.sin(ang)
    pe[:, 1::2] = np.cos(ang[:, : d // 2])
    return pe.astype(np.float32)


def build_model(cfg: ModelConfig) -> bytes:
    """Draw a model with the shapes of ``cfg`` and return the model-file bytes."""
    rng = np.random.Generator(np.random.PCG64(cfg.seed))
    d, F = cfg.d_model, cfg.d_ffn
    t: dict[str, np.ndarray] = {}
    wstd = cfg.weight_std
    sig_proj = wstd * np.sqrt(d)  # projection of a unit-variance d-vector
    sig_ffn = wstd * np.sqrt(d)

    def f32(a):
        return np.asarray(a, dtype=np.float32)

    def linear(pfx, n_out, n_in, s_in=None, s_out=None):
        w = rng.normal(0.0, wstd, size=(n_out, n_in))
        codes, sw = _quantize_rows(w, 7 if cfg.w_bits == 4 else 127)
        t[pfx + ".w"] = Int4Rows(codes) if cfg.w_bits == 4 else codes
        t[pfx + ".sw"] = sw
        t[pfx + ".b"] = f32(rng.normal(0.0, WEIGHT_STD, size=n_out))
        if s_in is not None:
            t[pfx + ".sin"] = f32([s_in])
        if s_out is not None:
            t[pfx + ".sout"] = f32(s_out)

    def ln(pfx):
        t[pfx + ".g"] = f32(rng.normal(1.0, WEIGHT_STD, size=d))
        t[pfx + ".b"] = f32(rng.normal(0.0, WEIGHT_STD, size=d))

    def gamma(name):
        t[name] = f32([rng.uniform(*cfg.gamma_range) if cfg.random_gamma else 1.0])

    ef = cfg.emb_dim or d
    e = rng.normal(0.0, cfg.emb_std, size=(cfg.emb_distinct or cfg.vocab, ef))
    if cfg.emb_distinct:
        e = e[np.arange(cfg.vocab) % cfg.emb_distinct]
    if cfg.eos_gain != 1.0:  # hypotheses that end at varied steps
        e = e.copy()
        e[EOS] = e[EOS] * cfg.eos_gain
    t["emb.w"], t["emb.s"] = _quantize_rows(e)
    if cfg.emb_dim:  # factorized: P [d, E] with entries N(0, 1/E), one per-tensor scale
        pw = rng.normal(0.0, 1.0 / np.sqrt(ef), size=(d, ef))
        s_p = float(np.abs(pw).max()) / 127.0
        t["emb.proj.w"] = np.clip(np.rint(pw / s_p), -127, 127).astype(np.int8)
        t["emb.proj.sw"] = f32([s_p])
        t["emb.proj.sout"] = f32([_act_scale(rng, np.sqrt(d / ef))])  # u = a P has variance d / E
    t["pe"] = positional_table(cfg.max_pos, d)
    s_enc = _act_scale(rng, 1.0)
    s_fin = _act_scale(rng, 1.0)
    t["enc.sout"] = f32([s_enc])
    t["dec.sout"] = f32([s_fin])
    for side, n_layers in (("enc", cfg.n_enc), ("dec", cfg.n_dec)):
        for l in range(n_layers):
            p = f"{side}.{l}"
            if cfg.share_every and l >= cfg.share_every:  # cross-layer parameter sharing
                t[p + ".share"] = np.array([l % cfg.share_every], np.int8)
                continue

            ln(p + ".sa.ln")
            s_qkv = [_act_scale(rng, sig_proj) for _ in range(3)]
            linear(p + ".sa.qkv", 3 * d, d, s_in=_act_scale(rng, 1.0), s_out=s_qkv)
            linear(p + ".sa.o", d, d, s_in=s_qkv[2])
            gamma(p + ".sa.gamma")
            if side == "dec":
                ln(p + ".ca.ln")
                s_q = _act_scale(rng, sig_proj)
                linear(p + ".ca.q", d, d, s_in=_act_scale(rng, 1.0), s_out=[s_q])
                s_kv = [_act_scale(rng, sig_proj) for _ in range(2)]
                linear(p + ".ca.kv", 2 * d, d, s_out=s_kv)
                linear(p + ".ca.o", d, d, s_in=s_kv[1])
                gamma(p + ".ca.gamma")
            ln(p + ".ff.ln")
            linear(p + ".ff.w1", F, d, s_in=_act_scale(rng, 1.0), s_out=[_act_scale(rng, sig_ffn)])
            linear(p + ".ff.w2", d, F)
            gamma(p + ".ff.gamma")
    if not cfg.ln_post:
        ln("enc.ln")
        ln("dec.ln")
    hdr = Header(d, cfg.n_heads, F, cfg.n_enc, cfg.n_dec, cfg.vocab, cfg.max_pos, cfg.ln_post)
    return write_model(hdr, t)


def make_sources(vocab: int, batch: int, lengths, seed: int, s_max: int | None = None):
    """Source ids [batch, s_max] int32 (right-padded with PAD=0) and lengths [batch].

    ``lengths`` is an int (every sentence), a (lo, hi) pair (uniform integer
    lengths in [lo, hi]) or a sequence of explicit lengths."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if isinstance(lengths, int):
        lens = np.full(batch, lengths, dtype=np.int32)
    elif isinstance(lengths, tuple) and len(lengths) == 2:
        lens = rng.integers(lengths[0], lengths[1] + 1, size=batch).astype(np.int32)
    else:
        lens = np.asarray(lengths, dtype=np.int32)
        assert lens.shape == (batch,)
    s_max = int(lens.max()) if s_max is None else s_max
    src = np.zeros((batch, s_max), dtype=np.int32)
    for b in range(batch):
        src[b, : lens[b]] = rng.integers(SPECIAL, vocab, size=lens[b])
    return src, lens


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelConfig
    batch: int
    lengths: object
    s_max: int
    beam: int
    steps: int
    alpha: float
    stop_at_eos: int
    seed: int


# The five workloads (the quantized-linear sweep has its own generator below).
WORKLOADS = {
    "tiny": Workload("tiny-postln-b1-greedy16", TINY, 1, 16, 16, 1, 16, 0.6, 0, 2001),
    "mobile": Workload("mobile-12-2-b1-s30-greedy30", MOBILE, 1, 30, 30, 1, 30, 0.6, 0, 2002),
    "mobile_beam": Workload("mobile-12-2-b64-s10to60-beam4-t64", MOBILE, 64, (10, 60), 60, 4, 64, 0.6, 1, 2003),
    "base_beam": Workload("base-6-6-b128-s20to64-beam4-t80", BASE, 128, (20, 64), 64, 4, 80, 0.6, 1, 2005),
}


def workload_inputs(w: Workload):
    return make_sources(w.model.vocab, w.batch, w.lengths, w.seed, s_max=w.s_max)


# Quantized-linear sweep: X [M, K], W [N, K] uniform in [-127, 127].
SWEEP_M = (1, 4, 64, 256, 4096)
SWEEP_KN = ((256, 1024), (1024, 256), (512, 2048), (256, 32000))


def sweep_case(M: int, K: int, N: int, seed: int = 2004):
    """Inputs of one sweep shape: X, W codes; folded per-channel requant scale
    (multiplier 127 / (4 * 5418.67 * sqrt(K)) * U[0.5, 1.5]) and bias
    (N(0, 8) output units).  5418.67 is the variance of U{-127..127}, so the
    requantized outputs span roughly +-32 codes."""
    rng = np.random.Generator(np.random.PCG64(seed + 7919 * M + 31 * K + N))
    X = rng.integers(-127, 128, size=(M, K), dtype=np.int64).astype(np.int8)
    W = rng.integers(-127, 128, size=(N, K), dtype=np.int64).astype(np.int8)
    mult = (127.0 / (4.0 * 5418.67 * np.sqrt(K)) * rng.uniform(0.5, 1.5, size=N)).astype(np.float32)
    bias = rng.normal(0.0, 8.0, size=N).astype(np.float32)
    return X, W, mult, bias
