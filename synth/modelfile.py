"""Writer and reader for the quantized model file (format version 1).

The format is plain data: a 64-byte header, a table of 64-byte tensor
entries and 256-byte-aligned tensor payloads.  It is described field by field
in ``include/mnmt.h``; this module only serializes, it performs none of the
inference arithmetic.

Header (little endian): magic "MNMT", u32 version=1, u32 d_model, n_heads,
d_ffn, n_enc, n_dec, vocab, max_pos, ln_post; i32 pad, bos, eos, unk;
f32 ln_eps; u32 n_tensors.
Entry: char name[40], u32 dtype (1 int8, 2 fp32, 3 packed 4-bit), u32 rank,
u32 dim0, u32 dim1, u64 offset.  A packed 4-bit tensor [dim0, dim1] (dim1 a
multiple of 16) holds codes in [-7, 7] as nibbles u = code + 8, dim0 * dim1 / 2
bytes: in each group of 16 codes of a row, byte i (i < 8) holds code i in its
low nibble and code i + 8 in its high nibble.
"""
from __future__ import annotations

import struct
from dataclasses import dataclass

import numpy as np

MAGIC = b"MNMT"
VERSION = 1
HEADER_FMT = "<4sIIIIIIIIIiiiifI"
ENTRY_FMT = "<40sIIIIQ"
ALIGN = 256

DT_I8 = 1
DT_F32 = 2
DT_I4 = 3


class Int4Rows:
    """int8 codes in [-7, 7] of a [rows, K] weight, to be stored packed (DT_I4)."""

    def __init__(self, codes: np.ndarray):
        codes = np.asarray(codes)
        if codes.ndim != 2 or codes.shape[1] % 16 or codes.min() < -7 or codes.max() > 7:
            raise ValueError("4-bit weights: [rows, K] codes in [-7, 7], K a multiple of 16")
        self.codes = codes.astype(np.int8)


def pack_int4(codes: np.ndarray) -> bytes:
    """The DT_I4 payload of codes [rows, K]."""
    u = (codes.astype(np.int16) + 8).astype(np.uint8).reshape(codes.shape[0], -1, 2, 8)
    return (u[:, :, 0, :] | (u[:, :, 1, :] << 4)).astype(np.uint8).tobytes()


def unpack_int4(data, rows: int, k: int) -> np.ndarray:
    """Codes [rows, k] (int8) of a DT_I4 payload."""
    b = np.frombuffer(data, dtype=np.uint8, count=rows * k // 2).reshape(rows, k // 16, 8)
    u = np.stack([b & 15, b >> 4], axis=2).reshape(rows, k).astype(np.int16)
    return (u - 8).astype(np.int8)


@dataclass
class Header:
    d_model: int
    n_heads: int
    d_ffn: int
    n_enc: int
    n_dec: int
    vocab: int
    max_pos: int
    ln_post: int
    pad_id: int = 0
    bos_id: int = 1
    eos_id: int = 2
    unk_id: int = 3
    ln_eps: float = 1e-5


def write_model(header: Header, tensors: dict[str, np.ndarray]) -> bytes:
    """Serialize ``tensors`` (name -> int8 or float32 array of rank 1 or 2)."""
    names = list(tensors)
    n = len(names)
    table_end = 64 + 64 * n
    off = (table_end + ALIGN - 1) // ALIGN * ALIGN
    entries = []
    payload = []
    for name in names:
        if isinstance(tensors[name], Int4Rows):
            codes = tensors[name].codes
            nb = name.encode()
            if len(nb) >= 40:
                raise ValueError(f"name too long: {name}")
            data = pack_int4(codes)
            entries.append(struct.pack(ENTRY_FMT, nb, DT_I4, 2, codes.shape[0], codes.shape[1], off))
            payload.append((off, data))
            off += (len(data) + ALIGN - 1) // ALIGN * ALIGN
            continue
        a = np.ascontiguousarray(tensors[name])
        if a.dtype == np.int8:
            dt = DT_I8
        elif a.dtype == np.float32:
            dt = DT_F32
        else:
            raise TypeError(f"{name}: dtype {a.dtype} not int8/float32")
        if a.ndim == 1:
            d0, d1 = a.shape[0], 1
        elif a.ndim == 2:
            d0, d1 = a.shape
        else:
            raise ValueError(f"{name}: rank {a.ndim}")
        nb = name.encode()
        if len(nb) >= 40:
            raise ValueError(f"name too long: {name}")
        entries.append(struct.pack(ENTRY_FMT, nb, dt, a.ndim, d0, d1, off))
        payload.append((off, a.tobytes()))
        off += (a.nbytes + ALIGN - 1) // ALIGN * ALIGN
    buf = bytearray(off)
    h = header
    struct.pack_into(HEADER_FMT, buf, 0, MAGIC, VERSION, h.d_model, h.n_heads, h.d_ffn, h.n_enc, h.n_dec,
                     h.vocab, h.max_pos, h.ln_post, h.pad_id, h.bos_id, h.eos_id, h.unk_id, h.ln_eps, n)
    for i, e in enumerate(entries):
        buf[64 + 64 * i: 128 + 64 * i] = e
    for o, data in payload:
        buf[o:o + len(data)] = data
    return bytes(buf)


def read_model(blob: bytes) -> tuple[Header, dict[str, np.ndarray]]:
    """Parse a model file back into a header and named arrays (views)."""
    f = struct.unpack_from(HEADER_FMT, blob, 0)
    if f[0] != MAGIC or f[1] != VERSION:
        raise ValueError("not a version-1 model file")
    h = Header(*f[2:10], pad_id=f[10], bos_id=f[11], eos_id=f[12], unk_id=f[13], ln_eps=f[14])
    out = {}
    for i in range(f[15]):
        name, dt, rank, d0, d1, off = struct.unpack_from(ENTRY_FMT, blob, 64 + 64 * i)
        name = name.rstrip(b"\0").decode()
        if dt == DT_I4:  # unpacked to int8 codes
            out[name] = unpack_int4(blob[off: off + d0 * d1 // 2], d0, d1)
            continue
        dtype = np.int8 if dt == DT_I8 else np.float32
        a = np.frombuffer(blob, dtype=dtype, count=d0 * d1, offset=off)
        out[name] = a.reshape(d0, d1) if rank == 2 else a
    return h, out
