"""Closed-form work counts for the INT8 encoder-decoder: parameters,
multiply-accumulates and the bytes one decode step must move.

These are the algorithmic figures the benchmark divides by measured time.  The
parameter and MAC formulas reproduce the paper's own figures (comparison table
with other efficient Transformers: MobileNMT-10MB 10M / 7.9M params and 0.3G
FLOPs at length 30, MobileNMT-20MB 20M / 17.7M and 0.6G, Transformer-base
65M / 44M and 1.9G; the paper's "FLOPs" are multiply-accumulates).
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass(frozen=True)
class Dims:
    d: int
    h: int
    F: int
    n_enc: int
    n_dec: int
    V: int


def param_counts(m: Dims) -> tuple[int, int]:
    """Weight-matrix elements (with, without the shared embedding)."""
    enc = m.n_enc * (4 * m.d * m.d + 2 * m.d * m.F)
    dec = m.n_dec * (8 * m.d * m.d + 2 * m.d * m.F)
    return m.V * m.d + enc + dec, enc + dec


def encoder_macs(m: Dims, S: int) -> int:
    """Encoder MACs for one sentence of S tokens: projections and FFN per token,
    attention scores and context per layer, plus every decoder layer's cross
    key/value projection (computed once per sentence)."""
    per_layer = S * (4 * m.d * m.d + 2 * m.d * m.F) + 2 * S * S * m.d
    return m.n_enc * per_layer + m.n_dec * 2 * m.d * m.d * S


def decoder_step_macs(m: Dims, t: int, S: int) -> int:
    """MACs of decode step t (0-based) for one hypothesis: self-attention
    projections, cross-attention query and output projections, FFN, attention
    over t + 1 cached and S source positions, and the logits over V."""
    per_layer = 6 * m.d * m.d + 2 * m.d * m.F + 2 * (t + 1) * m.d + 2 * S * m.d
    return m.n_dec * per_layer + m.V * m.d


def sentence_macs(m: Dims, S: int, T: int) -> int:
    return encoder_macs(m, S) + sum(decoder_step_macs(m, t, S) for t in range(T))


def decode_step_weight_bytes(m: Dims) -> int:
    """int8 weights plus the fp32 per-channel constants (scale and bias, 8 B per
    output channel; 4 B per vocabulary row for the logits) one decode step reads
    once whatever the batch: the decoder layers' self-attention QKV and O,
    cross-attention Q and O, FFN W1 and W2, and the tied output embedding.
    LayerNorm gains and shifts (8 B per element) are included."""
    d, F = m.d, m.F
    w = m.n_dec * (3 * d * d + d * d + d * d + d * d + F * d + d * F)
    chan = m.n_dec * (3 * d + d + d + d + F + d)
    ln = (3 * m.n_dec + 1) * 2 * d * 4
    return w + 8 * chan + m.V * d + 4 * m.V + ln


def decode_step_kv_bytes(m: Dims, t: int, S: int, rows: int = 1, beams_per_sentence: int = 1) -> int:
    """int8 cache bytes decode step t reads: the self-attention keys and values
    of positions 0..t for every row, and the cross-attention keys and values of
    the S source positions once per sentence."""
    self_kv = rows * m.n_dec * 2 * (t + 1) * m.d
    cross = (rows // beams_per_sentence) * m.n_dec * 2 * S * m.d
    return self_kv + cross


def logits_gemv_bytes(m: Dims) -> int:
    """Bytes the fused logits + arg-max kernel must read at batch 1: the int8
    embedding and its fp32 output scales."""
    return m.V * m.d + 4 * m.V


def encoder_weight_bytes(m: Dims) -> int:
    """Bytes of the encoder's weights and constants (read once per batch) plus
    every decoder layer's cross key/value projection."""
    d, F = m.d, m.F
    w = m.n_enc * (4 * d * d + 2 * d * F) + m.n_dec * 2 * d * d
    chan = m.n_enc * (3 * d + d + F + d) + m.n_dec * 2 * d
    ln = (2 * m.n_enc + 1) * 2 * d * 4
    return w + 8 * chan + ln


def greedy_sentence_bytes(m: Dims, S: int, T: int) -> int:
    """Algorithmic bytes of one batch-1 greedy translation: the encoder's and
    cross projections' weights once, then per decode step the decoder weights,
    the tied embedding and the step's key/value cache reads."""
    return encoder_weight_bytes(m) + sum(decode_step_weight_bytes(m) + decode_step_kv_bytes(m, t, S)
                                         for t in range(T))


def beam_roofline_s(m: Dims, src_lens, W: int, steps: int, peak_ops: float, bw: float) -> dict:
    """Composite roofline of a batched beam search that runs `steps` decode
    steps over sentences of lengths src_lens with W hypotheses each: the sum
    over phases of max(ops / peak_ops, bytes / bw), 2 ops per MAC.
    Phases: encoder linear layers (with the cross key/value projections) and
    encoder attention; per step the decoder linear layers, the logits, the
    self-attention over the key/value cache and the cross-attention.  Bytes
    are what each phase must move at least: weights once, int8 activations in
    and out, the caches read once per step (cross keys and values once per
    sentence), the logits' fp32 values not stored."""
    d, F, V, L = m.d, m.F, m.V, m.n_dec
    lens = [int(s) for s in src_lens]
    B, n_tok, n_sq = len(lens), sum(lens), sum(s * s for s in lens)
    R = B * W
    parts = {}

    def add(name, ops, nbytes):
        t = max(ops / peak_ops, nbytes / bw)
        p = parts.setdefault(name, [0.0, 0.0, 0.0])
        p[0] += ops
        p[1] += nbytes
        p[2] += t

    enc_ops = 2 * n_tok * (m.n_enc * (4 * d * d + 2 * d * F) + L * 2 * d * d)
    enc_bytes = encoder_weight_bytes(m) + m.n_enc * n_tok * (d + 3 * d + d + d + F + F) + n_tok * (d + L * 2 * d)
    add("encoder_linear", enc_ops, enc_bytes)
    add("encoder_attention", m.n_enc * 2 * 2 * n_sq * d, m.n_enc * n_tok * 4 * d)
    lay_w = L * (6 * d * d + 2 * d * F) + 8 * L * (5 * d + F + d)
    for t in range(steps):
        add("decoder_linear", 2 * R * L * (6 * d * d + 2 * d * F), lay_w + R * L * (d + 3 * d + d + d + d + F + F))
        add("logits", 2 * R * V * d, V * d + 4 * V + R * d)
        add("self_attention", 2 * R * L * 2 * (t + 1) * d, R * L * 2 * (t + 1) * d + R * L * 2 * d)
        add("cross_attention", 2 * R * L * 2 * n_tok // B * d, L * 2 * n_tok * d + R * L * 2 * d)
    total = sum(p[2] for p in parts.values())
    return {"seconds": total, "parts": {k: {"ops": v[0], "bytes": v[1], "seconds": v[2]} for k, v in parts.items()}}
