"""Thin Python binding of libmnmt (the C ABI in include/mnmt.h).

Argument marshalling only: every step of inference runs in the library's HIP
kernels.  PyTorch provides device memory (the model arena and the session
workspace are torch uint8 tensors) and streams.  There is no fallback: if the
library is not built, ``lib()`` raises.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmnmt.so")

OK, E_INVALID_ARG, E_BAD_MODEL, E_CAPACITY, E_HIP, E_UNSUPPORTED, E_TIMEOUT = 0, -1, -2, -3, -4, -5, -6
(EPI_I32, EPI_I8, EPI_I8_RELU, EPI_F32, EPI_F32_RESID, EPI_LOGITS, EPI_ARGMAX, EPI_ARGMAX_PARTIAL,
 EPI_ARGMAX_PARTIAL_PACKED) = range(9)

LOAD_PACKED_4BIT_ONLY = 1

EXPORTS = ("mnmt_model_bytes", "mnmt_model_load", "mnmt_model_bytes_ex", "mnmt_model_load_ex", "mnmt_model_get_info", "mnmt_model_free", "mnmt_session_bytes",
           "mnmt_session_create", "mnmt_session_free", "mnmt_encode", "mnmt_decode_step", "mnmt_translate",
           "mnmt_session_status", "mnmt_session_tensor", "mnmt_qlinear", "mnmt_qlinear_w4", "mnmt_qlinear_timed",
           "mnmt_argmax_partials", "mnmt_packed_bytes", "mnmt_pack_weights", "mnmt_logits_argmax_noalloc",
           "mnmt_fold_requant", "mnmt_debug_canon", "mnmt_debug_read", "mnmt_status_str", "mnmt_last_error")


class MnmtError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = lib().mnmt_last_error().decode(errors="replace")
        super().__init__(f"{where}: {lib().mnmt_status_str(status).decode()} ({status}): {msg}")
        self.status = status


class ModelInfo(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("d_model", "n_heads", "d_ffn", "n_enc", "n_dec", "vocab", "max_pos",
                                         "ln_post", "pad_id", "bos_id", "eos_id", "unk_id")] + [
        ("ln_eps", C.c_float), ("emb_dim", C.c_int32)]


class SessionCfg(C.Structure):
    _fields_ = [("max_batch", C.c_int32), ("max_src_len", C.c_int32), ("max_tgt_len", C.c_int32),
                ("beam", C.c_int32)]


class SearchCfg(C.Structure):
    _fields_ = [("beam", C.c_int32), ("max_steps", C.c_int32), ("len_penalty_alpha", C.c_float),
                ("stop_at_eos", C.c_int32), ("use_graph", C.c_int32)]


_lib = None


def lib():
    """Load libmnmt.so; raises if it has not been built (no fallback path)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "or python paper_2306_04235_amd/build.py")
        L = C.CDLL(LIB_PATH)
        vp, sz, i32, f32 = C.c_void_p, C.c_size_t, C.c_int, C.c_float
        L.mnmt_model_bytes.argtypes = [C.c_char_p, sz, C.POINTER(sz)]
        L.mnmt_model_load.argtypes = [C.c_char_p, sz, vp, sz, vp, C.POINTER(vp)]
        L.mnmt_model_bytes_ex.argtypes = [C.c_char_p, sz, C.c_uint, C.POINTER(sz)]
        L.mnmt_model_load_ex.argtypes = [C.c_char_p, sz, C.c_uint, vp, sz, vp, C.POINTER(vp)]
        L.mnmt_model_get_info.argtypes = [vp, C.POINTER(ModelInfo)]
        L.mnmt_model_free.argtypes = [vp]
        L.mnmt_model_free.restype = None
        L.mnmt_session_bytes.argtypes = [vp, C.POINTER(SessionCfg), C.POINTER(sz)]
        L.mnmt_session_create.argtypes = [vp, C.POINTER(SessionCfg), vp, sz, C.POINTER(vp)]
        L.mnmt_session_free.argtypes = [vp]
        L.mnmt_session_free.restype = None
        L.mnmt_encode.argtypes = [vp, vp, vp, i32, i32, vp]
        L.mnmt_decode_step.argtypes = [vp, vp, vp, vp, vp]
        L.mnmt_translate.argtypes = [vp, vp, vp, i32, i32, C.POINTER(SearchCfg), vp, vp, vp, vp]
        L.mnmt_session_tensor.argtypes = [vp, C.c_char_p, C.POINTER(vp), C.POINTER(sz)]
        L.mnmt_session_status.argtypes = [vp, vp]
        L.mnmt_qlinear.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, f32, vp, vp]
        L.mnmt_qlinear_w4.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, f32, vp, vp]
        L.mnmt_qlinear_timed.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, f32, vp, vp, vp, vp]
        L.mnmt_argmax_partials.argtypes = [i32]
        L.mnmt_packed_bytes.argtypes = [i32, i32]
        L.mnmt_packed_bytes.restype = sz
        L.mnmt_pack_weights.argtypes = [vp, i32, i32, vp, vp]
        L.mnmt_fold_requant.argtypes = [f32, vp, vp, f32, i32, vp, vp]
        L.mnmt_debug_canon.argtypes = [i32, vp, i32, vp, vp]
        L.mnmt_debug_read.argtypes = [vp, sz, i32, vp, vp]
        L.mnmt_logits_argmax_noalloc.argtypes = [vp, vp, vp, i32, i32, i32, vp, vp, vp]
        L.mnmt_status_str.argtypes = [i32]
        L.mnmt_status_str.restype = C.c_char_p
        L.mnmt_last_error.argtypes = []
        L.mnmt_last_error.restype = C.c_char_p
        _lib = L
    return _lib


def _check(rc: int, where: str):
    if rc != OK:
        raise MnmtError(rc, where)


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream=None):
    import torch

    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


# ---- host-only entry points ---------------------------------------------------
def mnmt_model_bytes(blob: bytes, flags: int = 0) -> int:
    n = C.c_size_t()
    _check(lib().mnmt_model_bytes_ex(blob, len(blob), flags, C.byref(n)), "mnmt_model_bytes_ex")
    return n.value


def mnmt_fold_requant(s_in, s_w, b, s_out):
    import numpy as np

    s_w = np.ascontiguousarray(s_w, np.float32)
    b = np.ascontiguousarray(b, np.float32)
    sc, bi = np.empty_like(s_w), np.empty_like(s_w)
    _check(lib().mnmt_fold_requant(float(s_in), s_w.ctypes.data, b.ctypes.data, float(s_out), s_w.size,
                                   sc.ctypes.data, bi.ctypes.data), "mnmt_fold_requant")
    return sc, bi


# ---- device entry points ---------------------------------------------------------
def mnmt_qlinear(X, W, scale, bias, epilogue, gamma=1.0, out=None, stream=None, n_out=None):
    """Y = epilogue(X W^T) for int8 CUDA tensors X [M, K], W [N, K] (for
    EPI_ARGMAX_PARTIAL_PACKED, W is mnmt_pack_weights' output and n_out = N)."""
    import torch

    M, K = X.shape
    N = W.shape[0] if n_out is None else int(n_out)
    if out is None and epilogue == EPI_ARGMAX:
        out = torch.zeros(M, dtype=torch.int64, device=X.device)  # packed (key, index) per row
    elif out is None and epilogue in (EPI_ARGMAX_PARTIAL, EPI_ARGMAX_PARTIAL_PACKED):
        out = torch.empty((M, argmax_partials(N)), dtype=torch.int64, device=X.device)
    elif out is None:
        dt = {EPI_I32: torch.int32, EPI_I8: torch.int8, EPI_I8_RELU: torch.int8}.get(epilogue, torch.float32)
        out = torch.empty((M, N), dtype=dt, device=X.device)
    _check(lib().mnmt_qlinear(_ptr(X), _ptr(W), _ptr(scale), _ptr(bias), M, K, N, epilogue, float(gamma),
                              _ptr(out), _stream(stream)), "mnmt_qlinear")
    return out


def mnmt_qlinear_w4(X, W4, scale, bias, epilogue, gamma=1.0, out=None, stream=None):
    """Y = epilogue(X W^T) for int8 CUDA tensor X [M, K] and W's packed 4-bit
    rows W4 uint8 [N, K / 2] (the model file's format)."""
    import torch

    M, K = X.shape
    N = W4.shape[0]
    if out is None:
        dt = {EPI_I32: torch.int32, EPI_I8: torch.int8, EPI_I8_RELU: torch.int8}.get(epilogue, torch.float32)
        out = torch.empty((M, N), dtype=dt, device=X.device)
    _check(lib().mnmt_qlinear_w4(_ptr(X), _ptr(W4), _ptr(scale), _ptr(bias), M, K, N, epilogue, float(gamma),
                                 _ptr(out), _stream(stream)), "mnmt_qlinear_w4")
    return out


def mnmt_qlinear_timed(X, W, scale, bias, epilogue, ev_start, ev_stop, gamma=1.0, out=None, stream=None,
                       n_out=None):
    """mnmt_qlinear bracketed by two torch.cuda.Event(enable_timing=True)
    (recorded once beforehand so that their HIP events exist)."""
    import torch

    M, K = X.shape
    N = W.shape[0] if n_out is None else int(n_out)
    if out is None:
        partial = epilogue in (EPI_ARGMAX_PARTIAL, EPI_ARGMAX_PARTIAL_PACKED)
        shape = (M, argmax_partials(N)) if partial else (M,)
        out = torch.zeros(shape, dtype=torch.int64, device=X.device)
    _check(lib().mnmt_qlinear_timed(_ptr(X), _ptr(W), _ptr(scale), _ptr(bias), M, K, N, epilogue, float(gamma),
                                    _ptr(out), _stream(stream), C.c_void_p(ev_start.cuda_event),
                                    C.c_void_p(ev_stop.cuda_event)), "mnmt_qlinear_timed")
    return out


def mnmt_pack_weights(W, stream=None):
    """Fragment-order copy of an int8 CUDA tensor W [N, K] (K a multiple of
    64): an int8 tensor [ceil(N / 16) * 16, K] whose bytes are in the order
    mnmt_pack_weights documents (not a row-major matrix)."""
    import torch

    N, K = W.shape
    if W.dtype != torch.int8 or not W.is_contiguous():
        raise ValueError("W must be a contiguous int8 tensor")
    nbytes = lib().mnmt_packed_bytes(int(N), int(K))
    if nbytes == 0:
        raise ValueError(f"cannot pack a [{N}, {K}] weight (K must be a positive multiple of 64)")
    out = torch.empty((nbytes // K, K), dtype=torch.int8, device=W.device)
    _check(lib().mnmt_pack_weights(_ptr(W), int(N), int(K), _ptr(out), _stream(stream)), "mnmt_pack_weights")
    return out


def argmax_partials(N: int) -> int:
    """Partial keys per row of an MNMT_EPI_ARGMAX_PARTIAL result for N outputs."""
    p = lib().mnmt_argmax_partials(int(N))
    if p < 1:
        raise ValueError(f"no arg-max partials for N={N}")
    return p


def argmax_index(packed):
    """Vocabulary index held in an MNMT_EPI_ARGMAX result (int64 tensor or array)."""
    import numpy as np

    low = np.asarray(packed.cpu() if hasattr(packed, "cpu") else packed).astype(np.int64) & 0xFFFFFFFF
    return (0xFFFFFFFF - low).astype(np.int64)


def mnmt_debug_canon(fn: int, x, stream=None):
    import torch

    y = torch.empty(x.numel() if fn != 2 else 1, dtype=torch.float32, device=x.device)
    _check(lib().mnmt_debug_canon(fn, _ptr(x), x.numel(), _ptr(y), _stream(stream)), "mnmt_debug_canon")
    return y


def mnmt_logits_argmax_noalloc(X, Wp, scale, N, key=None, tok=None, stream=None):
    """Per-row arg-max key (int64 view of the uint64) and index of X [M, K] against
    the packed weight Wp (mnmt_pack_weights), with no caller scratch."""
    import torch

    M, K = X.shape
    if key is None:
        key = torch.empty(M, dtype=torch.int64, device=X.device)
    if tok is None:
        tok = torch.empty(M, dtype=torch.int32, device=X.device)
    _check(lib().mnmt_logits_argmax_noalloc(_ptr(X), _ptr(Wp), _ptr(scale), M, K, N, _ptr(key), _ptr(tok),
                                            _stream(stream)), "mnmt_logits_argmax_noalloc")
    return key, tok


DEBUG_READ_BLOCKS = 2048


def mnmt_debug_read(x, sink, reps=1, stream=None):
    """Read every byte of the device tensor x `reps` times (bandwidth probe); sink: int32 [2048]."""
    if sink.numel() * sink.element_size() < 4 * DEBUG_READ_BLOCKS:
        raise ValueError("sink needs 2048 32-bit words")
    _check(lib().mnmt_debug_read(_ptr(x), x.numel() * x.element_size(), int(reps), _ptr(sink), _stream(stream)),
           "mnmt_debug_read")


class Model:
    """A model loaded into a torch-allocated device arena."""

    def __init__(self, blob: bytes, device="cuda", stream=None, flags: int = 0):
        import torch

        self.arena = torch.empty(mnmt_model_bytes(blob, flags), dtype=torch.uint8, device=device)
        h = C.c_void_p()
        _check(lib().mnmt_model_load_ex(blob, len(blob), flags, _ptr(self.arena), self.arena.numel(),
                                        _stream(stream), C.byref(h)), "mnmt_model_load_ex")
        self.handle = h
        info = ModelInfo()
        _check(lib().mnmt_model_get_info(h, C.byref(info)), "mnmt_model_get_info")
        self.info = info

    def close(self):
        if getattr(self, "handle", None):
            lib().mnmt_model_free(self.handle)
            self.handle = None

    def __del__(self):
        if _lib is not None:
            self.close()


class Session:
    """Decoding state of one model over a torch-allocated workspace."""

    def __init__(self, model: Model, max_batch: int, max_src_len: int, max_tgt_len: int, beam: int = 1):
        import torch

        self.model = model
        self.cfg = SessionCfg(max_batch, max_src_len, max_tgt_len, beam)
        n = C.c_size_t()
        _check(lib().mnmt_session_bytes(model.handle, C.byref(self.cfg), C.byref(n)), "mnmt_session_bytes")
        self.ws = torch.empty(n.value, dtype=torch.uint8, device=model.arena.device)
        h = C.c_void_p()
        _check(lib().mnmt_session_create(model.handle, C.byref(self.cfg), _ptr(self.ws), self.ws.numel(),
                                         C.byref(h)), "mnmt_session_create")
        self.handle = h

    def close(self):
        if getattr(self, "handle", None):
            lib().mnmt_session_free(self.handle)
            self.handle = None

    def __del__(self):
        if _lib is not None:
            self.close()

    def encode(self, src, lens, stream=None):
        B, S = src.shape
        _check(lib().mnmt_encode(self.handle, _ptr(src), _ptr(lens), B, S, _stream(stream)), "mnmt_encode")
        self._batch = B

    def decode_step(self, prev=None, want_logits=False, stream=None):
        import torch

        B = self._batch
        nxt = torch.empty(B, dtype=torch.int32, device=self.ws.device)
        logits = torch.empty((B, self.model.info.vocab), dtype=torch.float32,
                             device=self.ws.device) if want_logits else None
        _check(lib().mnmt_decode_step(self.handle, _ptr(prev), _ptr(nxt), _ptr(logits), _stream(stream)),
               "mnmt_decode_step")
        return nxt, logits

    def translate(self, src, lens, beam=1, max_steps=None, alpha=0.6, stop_at_eos=False, use_graph=True,
                  stream=None, out=None):
        import torch

        B, S = src.shape
        steps = max_steps or self.cfg.max_tgt_len
        if out is None:
            out = (torch.empty((B, steps), dtype=torch.int32, device=src.device),
                   torch.empty(B, dtype=torch.int32, device=src.device),
                   torch.empty(B, dtype=torch.float32, device=src.device))
        sc = SearchCfg(beam, steps, float(alpha), int(stop_at_eos), int(use_graph))
        _check(lib().mnmt_translate(self.handle, _ptr(src), _ptr(lens), B, S, C.byref(sc), _ptr(out[0]),
                                    _ptr(out[1]), _ptr(out[2]), _stream(stream)), "mnmt_translate")
        return out

    def status(self, stream=None):
        """Synchronize and raise MnmtError(E_TIMEOUT) if a chained kernel's wait gave up."""
        _check(lib().mnmt_session_status(self.handle, _stream(stream)), "mnmt_session_status")

    def tensor(self, name: str, dtype, shape):
        """A view of a session buffer (inside the workspace tensor)."""
        p, n = C.c_void_p(), C.c_size_t()
        _check(lib().mnmt_session_tensor(self.handle, name.encode(), C.byref(p), C.byref(n)), "mnmt_session_tensor")
        off = p.value - self.ws.data_ptr()
        return self.ws[off: off + n.value].view(dtype)[: _numel(shape)].view(shape)


def _numel(shape):
    n = 1
    for s in shape:
        n *= s
    return n
