"""Python access to the CPU oracle (``mnmt_oracle.c``) through ctypes.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg call this.  The GPU library never imports or links it.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmnmt_oracle.so")

EPI_I32, EPI_I8, EPI_I8_RELU, EPI_F32, EPI_F32_RESID, EPI_LOGITS = range(6)

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _b
            _b.build()
        L = C.CDLL(LIB_PATH)
        f32, i32, vp, sz = C.c_float, C.c_int, C.c_void_p, C.c_size_t
        L.orc_exp.restype = f32
        L.orc_exp.argtypes = [f32]
        L.orc_log.restype = f32
        L.orc_log.argtypes = [f32]
        L.orc_canon_sum.restype = f32
        L.orc_canon_sum.argtypes = [vp, i32]
        L.orc_canon_sum_squares.restype = f32
        L.orc_canon_sum_squares.argtypes = [vp, i32]
        L.orc_canon_vocab_sum.restype = f32
        L.orc_canon_vocab_sum.argtypes = [vp, i32]
        L.orc_quantize.restype = C.c_int8
        L.orc_quantize.argtypes = [f32, f32]
        L.orc_length_penalty.restype = f32
        L.orc_length_penalty.argtypes = [i32, f32]
        L.orc_map.argtypes = [i32, vp, i32, vp]
        L.orc_qgemm_i32.argtypes = [vp, vp, i32, i32, i32, vp]
        L.orc_qlinear.argtypes = [vp, vp, i32, i32, i32, vp, vp, f32, i32, vp]
        L.orc_fold_requant.argtypes = [f32, vp, vp, f32, i32, vp, vp]
        L.orc_fold_dequant.argtypes = [f32, vp, i32, vp]
        L.orc_layernorm_quant.argtypes = [vp, i32, i32, vp, vp, f32, f32, vp, vp]
        L.orc_attend.argtypes = [vp, vp, vp, i32, i32, i32, f32, f32, vp]
        L.orc_log_softmax_stats.argtypes = [vp, i32, vp, vp]
        L.orc_model_load.argtypes = [C.c_char_p, sz, C.POINTER(vp)]
        L.orc_model_free.argtypes = [vp]
        L.orc_model_free.restype = None
        L.orc_model_dims.argtypes = [vp, vp]
        L.orc_model_constants.argtypes = [vp, C.c_char_p, vp, i32]
        L.orc_encode.argtypes = [vp, vp, vp, i32, i32, vp]
        L.orc_cross_kv.argtypes = [vp, vp, vp, i32, i32, i32, vp]
        L.orc_translate_greedy.argtypes = [vp, vp, vp, i32, i32, i32, i32, vp, vp, vp]
        L.orc_decoder_logits.argtypes = [vp, vp, i32, vp, i32, vp]
        L.orc_decoder_logits_full.argtypes = [vp, vp, i32, vp, i32, vp]
        L.orc_translate_beam.argtypes = [vp, vp, vp, i32, i32, i32, i32, f32, vp, vp, vp]
        L.orc_encode_trace.argtypes = [vp, vp, i32, vp, vp, vp, vp, vp]
        L.orc_decoder_trace.argtypes = [vp, vp, i32, vp, i32, vp, vp, vp, vp, vp, vp, vp]
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def _check(rc, what):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with status {rc}")


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ---- canonical primitives ---------------------------------------------------
def exp(x: float) -> float:
    return lib().orc_exp(float(x))


def log(x: float) -> float:
    return lib().orc_log(float(x))


def exp_array(x):
    x = _c(x, np.float32)
    y = np.empty_like(x)
    _check(lib().orc_map(0, _p(x), x.size, _p(y)), "exp_array")
    return y


def log_array(x):
    x = _c(x, np.float32)
    y = np.empty_like(x)
    _check(lib().orc_map(1, _p(x), x.size, _p(y)), "log_array")
    return y


def canon_sum(x) -> np.float32:
    x = _c(x, np.float32)
    return np.float32(lib().orc_canon_sum(_p(x), x.size))


def canon_vocab_sum(x) -> np.float32:
    x = _c(x, np.float32)
    return np.float32(lib().orc_canon_vocab_sum(_p(x), x.size))


def canon_sum_squares(x) -> np.float32:
    x = _c(x, np.float32)
    return np.float32(lib().orc_canon_sum_squares(_p(x), x.size))


def fold_dequant(s_in, s_w):
    s_w = _c(s_w, np.float32)
    out = np.empty_like(s_w)
    lib().orc_fold_dequant(float(s_in), _p(s_w), s_w.size, _p(out))
    return out


def quantize(y: float, inv_s: float) -> int:
    return int(lib().orc_quantize(float(y), float(inv_s)))


def length_penalty(L: int, alpha: float) -> np.float32:
    return np.float32(lib().orc_length_penalty(int(L), float(alpha)))


# ---- stages -----------------------------------------------------------------
def qgemm_i32(X, W):
    X, W = _c(X, np.int8), _c(W, np.int8)
    M, K = X.shape
    N = W.shape[0]
    Y = np.empty((M, N), np.int32)
    _check(lib().orc_qgemm_i32(_p(X), _p(W), M, K, N, _p(Y)), "qgemm")
    return Y


def qlinear(X, W, scale, bias, epilogue, gamma=1.0, resid=None):
    X, W = _c(X, np.int8), _c(W, np.int8)
    M, K = X.shape
    N = W.shape[0]
    scale = _c(scale, np.float32)
    bias = None if bias is None else _c(bias, np.float32)
    if epilogue == EPI_I32:
        Y = np.empty((M, N), np.int32)
    elif epilogue in (EPI_I8, EPI_I8_RELU):
        Y = np.empty((M, N), np.int8)
    elif epilogue == EPI_F32_RESID:
        Y = np.array(resid, dtype=np.float32, copy=True).reshape(M, N)
    else:
        Y = np.empty((M, N), np.float32)
    _check(lib().orc_qlinear(_p(X), _p(W), M, K, N, _p(scale), _p(bias), float(gamma), epilogue, _p(Y)),
           "qlinear")
    return Y


def fold_requant(s_in, s_w, b, s_out):
    s_w, b = _c(s_w, np.float32), _c(b, np.float32)
    sc, bi = np.empty_like(s_w), np.empty_like(s_w)
    lib().orc_fold_requant(float(s_in), _p(s_w), _p(b), float(s_out), s_w.size, _p(sc), _p(bi))
    return sc, bi


def layernorm_quant(x, g, b, eps, inv_s, want_y=False):
    x = _c(x, np.float32)
    rows, d = x.shape
    q = np.empty((rows, d), np.int8)
    y = np.empty((rows, d), np.float32) if want_y else None
    _check(lib().orc_layernorm_quant(_p(x), rows, d, _p(_c(g, np.float32)), _p(_c(b, np.float32)), float(eps),
                                     float(inv_s), _p(q), _p(y)), "layernorm")
    return (q, y) if want_y else q


def attend(q, K, V, c_qk, c_pv):
    """One query row q[dh] against K[n, dh], V[n, dh] codes."""
    q, K, V = _c(q, np.int8), _c(K, np.int8), _c(V, np.int8)
    n, dh = K.shape
    out = np.empty(dh, np.int8)
    _check(lib().orc_attend(_p(q), _p(K), _p(V), n, dh, dh, float(c_qk), float(c_pv), _p(out)), "attend")
    return out


def log_softmax_stats(z):
    z = _c(z, np.float32)
    mx, lse = np.zeros(1, np.float32), np.zeros(1, np.float32)
    _check(lib().orc_log_softmax_stats(_p(z), z.size, _p(mx), _p(lse)), "lse")
    return mx[0], lse[0]


# ---- model ------------------------------------------------------------------
class Model:
    """A loaded model file; all methods run the scalar oracle."""

    def __init__(self, blob: bytes):
        self._blob = blob
        h = C.c_void_p()
        _check(lib().orc_model_load(blob, len(blob), C.byref(h)), "model_load")
        self._h = h
        dims = np.zeros(16, np.int32)
        lib().orc_model_dims(self._h, _p(dims))
        (self.d, self.h, self.F, self.n_enc, self.n_dec, self.V, self.max_pos, self.ln_post, self.pad_id,
         self.bos_id, self.eos_id, self.unk_id, self.emb_dim) = [int(v) for v in dims[:13]]

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.orc_model_free(self._h)
            self._h = None

    def constants(self, name: str, n: int):
        out = np.zeros(n, np.float32)
        _check(lib().orc_model_constants(self._h, name.encode(), _p(out), n), f"constants {name}")
        return out

    def encode(self, src, lens):
        src, lens = _c(src, np.int32), _c(lens, np.int32)
        B, S = src.shape
        enc = np.zeros((B, S, self.d), np.int8)
        _check(lib().orc_encode(self._h, _p(src), _p(lens), B, S, _p(enc)), "encode")
        return enc

    def cross_kv(self, enc, lens, layer):
        enc, lens = _c(enc, np.int8), _c(lens, np.int32)
        B, S, _ = enc.shape
        kv = np.zeros((B, S, 2 * self.d), np.int8)
        _check(lib().orc_cross_kv(self._h, _p(enc), _p(lens), B, S, layer, _p(kv)), "cross_kv")
        return kv

    def greedy(self, src, lens, steps, stop_at_eos=False, want_logits=False):
        src, lens = _c(src, np.int32), _c(lens, np.int32)
        B, S = src.shape
        out = np.zeros((B, steps), np.int32)
        out_len = np.zeros(B, np.int32)
        logits = np.zeros((B, steps, self.V), np.float32) if want_logits else None
        _check(lib().orc_translate_greedy(self._h, _p(src), _p(lens), B, S, steps, int(stop_at_eos), _p(out),
                                          _p(out_len), _p(logits)), "greedy")
        return (out, out_len, logits) if want_logits else (out, out_len)

    def decoder_logits(self, src_row, tokens):
        """Teacher-forced logits [n, V] for one sentence (inputs BOS, tokens[:-1])."""
        src_row, tokens = _c(src_row, np.int32), _c(tokens, np.int32)
        z = np.zeros((tokens.size, self.V), np.float32)
        _check(lib().orc_decoder_logits(self._h, _p(src_row), src_row.size, _p(tokens), tokens.size, _p(z)),
               "decoder_logits")
        return z

    def decoder_logits_full(self, src_row, tokens):
        """The same logits from the cache-free causal block computation."""
        src_row, tokens = _c(src_row, np.int32), _c(tokens, np.int32)
        z = np.zeros((tokens.size, self.V), np.float32)
        _check(lib().orc_decoder_logits_full(self._h, _p(src_row), src_row.size, _p(tokens), tokens.size,
                                             _p(z)), "decoder_logits_full")
        return z

    def encode_trace(self, src_row):
        """One sentence's encoder with its intermediate values: dict with x [U+1, S, d]
        fp32, a [U, S, d], pj [U, S, P], ctx [U, S, d] int8 (U = 2 n_enc,
        P = max(3d, F); FFN sublayers leave ctx zero) and enc [S, d]."""
        src_row = _c(src_row, np.int32)
        S, d, U = src_row.size, self.d, 2 * self.n_enc
        P = max(3 * d, self.F)
        t = dict(x=np.zeros((U + 1, S, d), np.float32), a=np.zeros((U, S, d), np.int8),
                 pj=np.zeros((U, S, P), np.int8), ctx=np.zeros((U, S, d), np.int8), enc=np.zeros((S, d), np.int8))
        _check(lib().orc_encode_trace(self._h, _p(src_row), S, _p(t["x"]), _p(t["a"]), _p(t["pj"]), _p(t["ctx"]),
                                      _p(t["enc"])), "encode_trace")
        return t

    def decoder_trace(self, src_row, tokens):
        """Teacher-forced decoding (inputs BOS, tokens[:-1]) with each step's
        intermediate values: x [U+1, n, d], a, pj, ctx as in encode_trace
        (U = 3 n_dec), fin [n, d] (int8 final rows), fin_u [n, emb_dim] (a
        factorized embedding's projection of them) and z [n, V] logits."""
        src_row, tokens = _c(src_row, np.int32), _c(tokens, np.int32)
        n, d, U = tokens.size, self.d, 3 * self.n_dec
        P = max(3 * d, self.F)
        t = dict(x=np.zeros((U + 1, n, d), np.float32), a=np.zeros((U, n, d), np.int8),
                 pj=np.zeros((U, n, P), np.int8), ctx=np.zeros((U, n, d), np.int8), fin=np.zeros((n, d), np.int8),
                 fin_u=np.zeros((n, max(self.emb_dim, 1)), np.int8), z=np.zeros((n, self.V), np.float32))
        _check(lib().orc_decoder_trace(self._h, _p(src_row), src_row.size, _p(tokens), n, _p(t["x"]), _p(t["a"]),
                                       _p(t["pj"]), _p(t["ctx"]), _p(t["fin"]), _p(t["fin_u"]), _p(t["z"])),
               "decoder_trace")
        return t

    def beam(self, src, lens, beam, max_steps, alpha=0.6):
        src, lens = _c(src, np.int32), _c(lens, np.int32)
        B, S = src.shape
        out = np.zeros((B, max_steps), np.int32)
        out_len = np.zeros(B, np.int32)
        score = np.zeros(B, np.float32)
        _check(lib().orc_translate_beam(self._h, _p(src), _p(lens), B, S, beam, max_steps, float(alpha), _p(out),
                                        _p(out_len), _p(score)), "beam")
        return out, out_len, score
