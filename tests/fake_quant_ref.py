"""Float64 fake-quantized reference of the INT8 model, written from the paper.

Test code, independent of the oracle: it reads the model file with its own
reader (``synth.modelfile``), uses the file's *unfolded* scales (s_in, s_w,
s_out, the embedding's row scales, the encoder-output and final scales, gamma)
and computes every stage in float64 straight from the paper's definitions:

* the self-weight and self-sum equations of Appendix A, with the multi-head
  scale 1/sqrt(d_head) and softmax in float64;
* the FFN equation of Appendix A, ReLU(X W1 + b1) W2 + b2;
* the quantizer figure of Section 3.2 for which edges are 8-bit: the input
  of every linear layer, Q, K, V and the attention context, the ReLU output;
  everything else (biases, residual stream, scaled scores, softmax output,
  logits) is full precision; gamma weights each sublayer's residual input;
* layer normalization at each sublayer input (pre-LN, Appendix D) or after
  each residual add (post-LN files), biased variance, the file's epsilon;
* one shared embedding for input and output (Appendix D), input rows scaled
  by sqrt(d) plus the stored position table, output projection tied;
* cross-layer parameter sharing (Section 2.2): a layer whose file entry
  "<side>.<l>.share" names layer j runs on layer j's parameters;
* embedding factorization (Section 2.1): embedding rows of width E times a
  transformation P [d, E] on the way in, the final rows times P on the way
  out (an int8 edge like every linear input), then the tied embedding.

Quantizer (the paper's rounding to the nearest integer, symmetric reading):
code = clamp(round(value / s), -127, 127).  The stage functions return the
float64 value in code units *before* rounding, so that a test can tell a
genuine mismatch from a value that lies on a rounding boundary.
"""
from __future__ import annotations

import numpy as np

from synth.modelfile import read_model

F64 = np.float64


class FakeQuantModel:
    def __init__(self, blob: bytes):
        h, t = read_model(blob)
        self.hdr = h
        self.t = t
        self.d, self.nh, self.F = h.d_model, h.n_heads, h.d_ffn
        self.dh = self.d // self.nh
        self.n_enc, self.n_dec, self.V = h.n_enc, h.n_dec, h.vocab
        self.post = bool(h.ln_post)
        self.eps = float(np.float32(h.ln_eps))

    # --- parameters ---------------------------------------------------------
    def layer(self, side: str, l: int) -> str:
        """Tensor-name prefix of layer l of a stack, following shared layers."""
        while f"{side}.{l}.share" in self.t:
            l = int(self.t[f"{side}.{l}.share"][0])
        return f"{side}.{l}"

    def scalar(self, name: str) -> float:
        return float(self.t[name][0])

    def vec(self, name: str) -> np.ndarray:
        return np.asarray(self.t[name], dtype=F64).reshape(-1)

    def weight(self, pfx: str) -> np.ndarray:
        """Real-valued weight [N, K] = s_w[n] * code[n, k]."""
        return self.t[pfx + ".w"].astype(F64) * self.vec(pfx + ".sw")[:, None]

    def linear(self, codes, s_in: float, pfx: str) -> np.ndarray:
        """x W^T + b with x = s_in * codes (the real value of an int8 input)."""
        return (np.asarray(codes, F64) * s_in) @ self.weight(pfx).T + self.vec(pfx + ".b")

    # --- building blocks ----------------------------------------------------
    def layer_norm(self, x, pfx: str) -> np.ndarray:
        x = np.asarray(x, F64)
        mu = x.mean(axis=-1, keepdims=True)
        var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
        return (x - mu) / np.sqrt(var + self.eps) * self.vec(pfx + ".g") + self.vec(pfx + ".b")

    @property
    def factorized(self) -> bool:
        return "emb.proj.w" in self.t

    def proj(self) -> np.ndarray:
        """Factorized embedding (Section 2.1): the real transformation P [d, E]."""
        return self.t["emb.proj.w"].astype(F64) * self.scalar("emb.proj.sw")

    def embed(self, tokens, positions) -> np.ndarray:
        E = self.t["emb.w"].astype(F64) * self.vec("emb.s")[:, None]
        pe = self.t["pe"].astype(F64)
        e = E[np.asarray(tokens)]
        if self.factorized:
            e = e @ self.proj().T
        return e * np.sqrt(self.d) + pe[np.asarray(positions)]

    def sublayer_input(self, x, ln_pfx: str, s_in: float) -> np.ndarray:
        """Code-unit value of the sublayer's int8 input: pre-LN normalizes the
        residual stream, post-LN quantizes it as it is (already normalized)."""
        y = np.asarray(x, F64) if self.post else self.layer_norm(x, ln_pfx)
        return y / s_in

    def residual(self, x, update, gamma: float, ln_pfx: str) -> np.ndarray:
        r = gamma * np.asarray(x, F64) + update
        return self.layer_norm(r, ln_pfx) if self.post else r

    def attention(self, q_codes, k_codes, v_codes, s_q, s_k, s_v, s_ctx) -> np.ndarray:
        """Context in code units of s_ctx: per head softmax(q k^T / sqrt(d_head)) v
        with q, k, v the real values of their codes; q [n_q, d], k and v [n_k, d]
        hold only the keys each query may attend to."""
        q = np.asarray(q_codes, F64) * s_q
        k = np.asarray(k_codes, F64) * s_k
        v = np.asarray(v_codes, F64) * s_v
        out = np.zeros((q.shape[0], self.d))
        for hd in range(self.nh):
            sl = slice(hd * self.dh, (hd + 1) * self.dh)
            s = q[:, sl] @ k[:, sl].T / np.sqrt(self.dh)
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            out[:, sl] = p @ v[:, sl]
        return out / s_ctx

    # --- sublayers: (code-unit values of the int8 results, next residual) --------
    def self_attention_sublayer(self, pfx, x, a_codes, qkv_codes, ctx_codes, key_rows):
        """pfx "enc.<l>" / "dec.<l>"; key_rows(i) -> indices of the keys row i sees.
        Returns the code-unit values of a, qkv and ctx and the next residual,
        each computed from the oracle's values of the stage before."""
        d = self.d
        s_in = self.scalar(pfx + ".sa.qkv.sin")
        s_out = self.vec(pfx + ".sa.qkv.sout")
        s_ctx = self.scalar(pfx + ".sa.o.sin")
        a_val = self.sublayer_input(x, pfx + ".sa.ln", s_in)
        y = self.linear(a_codes, s_in, pfx + ".sa.qkv")
        qkv_val = np.concatenate([y[:, i * d:(i + 1) * d] / s_out[i] for i in range(3)], axis=1)
        q, k, v = qkv_codes[:, :d], qkv_codes[:, d:2 * d], qkv_codes[:, 2 * d:3 * d]
        ctx_val = np.zeros((x.shape[0], d))
        for i in range(x.shape[0]):
            keys = key_rows(i)
            ctx_val[i] = self.attention(q[i:i + 1], k[keys], v[keys], s_out[0], s_out[1], s_out[2], s_ctx)[0]
        upd = self.linear(ctx_codes, s_ctx, pfx + ".sa.o")
        x_next = self.residual(x, upd, self.scalar(pfx + ".sa.gamma"), pfx + ".sa.ln")
        return a_val, qkv_val, ctx_val, x_next

    def cross_attention_sublayer(self, pfx, x, a_codes, q_codes, ctx_codes, kv_codes):
        d = self.d
        s_in = self.scalar(pfx + ".ca.q.sin")
        s_q = self.scalar(pfx + ".ca.q.sout")
        s_kv = self.vec(pfx + ".ca.kv.sout")
        s_ctx = self.scalar(pfx + ".ca.o.sin")
        a_val = self.sublayer_input(x, pfx + ".ca.ln", s_in)
        q_val = self.linear(a_codes, s_in, pfx + ".ca.q") / s_q
        ctx_val = self.attention(q_codes, kv_codes[:, :d], kv_codes[:, d:], s_q, s_kv[0], s_kv[1], s_ctx)
        upd = self.linear(ctx_codes, s_ctx, pfx + ".ca.o")
        x_next = self.residual(x, upd, self.scalar(pfx + ".ca.gamma"), pfx + ".ca.ln")
        return a_val, q_val, ctx_val, x_next

    def ffn_sublayer(self, pfx, x, a_codes, h_codes):
        s_in = self.scalar(pfx + ".ff.w1.sin")
        s_h = self.scalar(pfx + ".ff.w1.sout")  # the hidden layer's scale, W2's input scale
        a_val = self.sublayer_input(x, pfx + ".ff.ln", s_in)
        h_val = np.maximum(self.linear(a_codes, s_in, pfx + ".ff.w1"), 0.0) / s_h
        upd = self.linear(h_codes, s_h, pfx + ".ff.w2")
        x_next = self.residual(x, upd, self.scalar(pfx + ".ff.gamma"), pfx + ".ff.ln")
        return a_val, h_val, x_next

    def encoder_output(self, x) -> np.ndarray:
        s = self.scalar("enc.sout")
        return (np.asarray(x, F64) if self.post else self.layer_norm(x, "enc.ln")) / s

    def final_input(self, x) -> np.ndarray:
        s = self.scalar("dec.sout")
        return (np.asarray(x, F64) if self.post else self.layer_norm(x, "dec.ln")) / s

    def cross_kv(self, enc_codes, layer: int) -> np.ndarray:
        pfx = self.layer("dec", layer) + ".ca.kv"
        y = self.linear(enc_codes, self.scalar("enc.sout"), pfx)
        s = self.vec(pfx + ".sout")
        return np.concatenate([y[:, :self.d] / s[0], y[:, self.d:] / s[1]], axis=1)

    def proj_back(self, fin_codes) -> np.ndarray:
        """Factorized embedding: code-unit value of the final rows mapped back to
        the embedding width, u = (a P) / s_u."""
        return (np.asarray(fin_codes, F64) * self.scalar("dec.sout")) @ self.proj() / self.scalar("emb.proj.sout")

    def logits(self, fin_codes, u_codes=None) -> np.ndarray:
        """Tied output projection of the final rows (or, factorized, of their
        int8 projection u_codes)."""
        E = self.t["emb.w"].astype(F64) * self.vec("emb.s")[:, None]
        if self.factorized:
            return (np.asarray(u_codes, F64) * self.scalar("emb.proj.sout")) @ E.T
        return (np.asarray(fin_codes, F64) * self.scalar("dec.sout")) @ E.T

    # --- the whole model without activation quantization ------------------------
    def float_logits(self, src, tokens) -> np.ndarray:
        """Teacher-forced logits [n, V] of the model with real-valued weights and
        no activation quantization (inputs BOS, tokens[:-1]): the sanity
        reference for the int8 model's arg-max."""
        d = self.d
        S = len(src)
        x = self.embed(src, np.arange(S))
        for l in range(self.n_enc):
            p = self.layer("enc", l)
            a = x if self.post else self.layer_norm(x, p + ".sa.ln")
            y = (a @ self.weight(p + ".sa.qkv").T) + self.vec(p + ".sa.qkv.b")
            ctx = self.attention(y[:, :d], y[:, d:2 * d], y[:, 2 * d:], 1.0, 1.0, 1.0, 1.0)
            x = self.residual(x, ctx @ self.weight(p + ".sa.o").T + self.vec(p + ".sa.o.b"),
                              self.scalar(p + ".sa.gamma"), p + ".sa.ln")
            a = x if self.post else self.layer_norm(x, p + ".ff.ln")
            hid = np.maximum(a @ self.weight(p + ".ff.w1").T + self.vec(p + ".ff.w1.b"), 0.0)
            x = self.residual(x, hid @ self.weight(p + ".ff.w2").T + self.vec(p + ".ff.w2.b"),
                              self.scalar(p + ".ff.gamma"), p + ".ff.ln")
        enc = x if self.post else self.layer_norm(x, "enc.ln")
        bos = self.hdr.bos_id
        n = len(tokens)
        inp = np.concatenate([[bos], np.asarray(tokens[:-1])]).astype(np.int64)
        x = self.embed(inp, np.arange(n))
        for l in range(self.n_dec):
            p = self.layer("dec", l)
            a = x if self.post else self.layer_norm(x, p + ".sa.ln")
            y = (a @ self.weight(p + ".sa.qkv").T) + self.vec(p + ".sa.qkv.b")
            ctx = np.zeros((n, d))
            for i in range(n):
                ctx[i] = self.attention(y[i:i + 1, :d], y[: i + 1, d:2 * d], y[: i + 1, 2 * d:], 1.0, 1.0, 1.0,
                                        1.0)[0]
            x = self.residual(x, ctx @ self.weight(p + ".sa.o").T + self.vec(p + ".sa.o.b"),
                              self.scalar(p + ".sa.gamma"), p + ".sa.ln")
            a = x if self.post else self.layer_norm(x, p + ".ca.ln")
            q = a @ self.weight(p + ".ca.q").T + self.vec(p + ".ca.q.b")
            kv = enc @ self.weight(p + ".ca.kv").T + self.vec(p + ".ca.kv.b")
            ctx = self.attention(q, kv[:, :d], kv[:, d:], 1.0, 1.0, 1.0, 1.0)
            x = self.residual(x, ctx @ self.weight(p + ".ca.o").T + self.vec(p + ".ca.o.b"),
                              self.scalar(p + ".ca.gamma"), p + ".ca.ln")
            a = x if self.post else self.layer_norm(x, p + ".ff.ln")
            hid = np.maximum(a @ self.weight(p + ".ff.w1").T + self.vec(p + ".ff.w1.b"), 0.0)
            x = self.residual(x, hid @ self.weight(p + ".ff.w2").T + self.vec(p + ".ff.w2.b"),
                              self.scalar(p + ".ff.gamma"), p + ".ff.ln")
        fin = x if self.post else self.layer_norm(x, "dec.ln")
        E = self.t["emb.w"].astype(F64) * self.vec("emb.s")[:, None]
        if self.factorized:
            fin = fin @ self.proj()
        return fin @ E.T
