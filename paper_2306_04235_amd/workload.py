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
