"""Symbol ranking back end (Definition of Symbol Ranking; Experimental
Methodology: ranks written as byte-aligned variable-length integers, then
compressed by a general-purpose compressor).

Rank(s | W) = j iff s is the j-th symbol of the list ordered by
non-increasing probability.  Where the paper is silent: equal probabilities
are ordered by token id (the lower id first).  Ranks are computed from the
logits, whose order is the probability order (softmax is monotone); a caller
checking another implementation passes that implementation's logits so both
take the same comparisons.

varint: unsigned LEB128 -- 7 bits per byte, least significant group first,
the high bit set on every byte but the last.

Container-level compression: the concatenated chunk payloads are compressed as
one block ("none", "zlib" at a level, "lzma" xz at a preset, "zstd" at a
level).  zlib and lzma come from Python's standard modules; zstd from the
system's libzstd (ZSTD_compress / ZSTD_decompress, through ctypes), since no
Python binding is installed.
"""
from __future__ import annotations

import ctypes
import ctypes.util
import lzma
import zlib
from typing import List

import numpy as np


def order(logits_row: np.ndarray) -> np.ndarray:
    """sigma_0, sigma_1, ...: token ids by non-increasing logit, ties by id."""
    lg = np.asarray(logits_row)
    return np.lexsort((np.arange(lg.shape[0]), -lg))


def rank_of(logits_row: np.ndarray, s: int) -> int:
    return int(np.flatnonzero(order(logits_row) == s)[0])


def symbol_at(logits_row: np.ndarray, r: int) -> int:
    return int(order(logits_row)[r])


def varint_encode(values) -> bytes:
    out = bytearray()
    for v in values:
        v = int(v)
        if v < 0:
            raise ValueError("varint of a negative value")
        while True:
            b = v & 0x7F
            v >>= 7
            if v:
                out.append(b | 0x80)
            else:
                out.append(b)
                break
    return bytes(out)


def varint_decode(data: bytes, n: int, pos: int = 0):
    """n values from data[pos:]; returns (values, next position)."""
    vals: List[int] = []
    for _ in range(n):
        v, shift = 0, 0
        while True:
            if pos >= len(data):
                raise ValueError("varint stream ended early")
            b = data[pos]
            pos += 1
            v |= (b & 0x7F) << shift
            shift += 7
            if not b & 0x80:
                break
            if shift > 63:
                raise ValueError("varint longer than 64 bits")
        vals.append(v)
    return vals, pos


_ZSTD = None


def zstd_library():
    """The system libzstd (ctypes), or None when it is not installed."""
    global _ZSTD
    if _ZSTD is None:
        name = ctypes.util.find_library("zstd") or "libzstd.so.1"
        try:
            lib = ctypes.CDLL(name)
        except OSError:
            _ZSTD = False
            return None
        sz, vp, cvp = ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p
        lib.ZSTD_compressBound.restype = sz
        lib.ZSTD_compressBound.argtypes = [sz]
        lib.ZSTD_compress.restype = sz
        lib.ZSTD_compress.argtypes = [vp, sz, cvp, sz, ctypes.c_int]
        lib.ZSTD_decompress.restype = sz
        lib.ZSTD_decompress.argtypes = [vp, sz, cvp, sz]
        lib.ZSTD_getFrameContentSize.restype = ctypes.c_ulonglong
        lib.ZSTD_getFrameContentSize.argtypes = [cvp, sz]
        lib.ZSTD_isError.restype = ctypes.c_uint
        lib.ZSTD_isError.argtypes = [sz]
        _ZSTD = lib
    return _ZSTD or None


def _zstd_compress(data: bytes, level: int) -> bytes:
    lib = zstd_library()
    if lib is None:
        raise RuntimeError("libzstd is not installed")
    cap = lib.ZSTD_compressBound(len(data))
    out = ctypes.create_string_buffer(max(cap, 1))
    n = lib.ZSTD_compress(out, cap, bytes(data), len(data), level)
    if lib.ZSTD_isError(n):
        raise ValueError("zstd compression failed")
    return out.raw[:n]


def _zstd_decompress(blob: bytes) -> bytes:
    """One zstd frame that states its content size (RFC 8878, Frame_Content_Size)."""
    lib = zstd_library()
    if lib is None:
        raise RuntimeError("libzstd is not installed")
    blob = bytes(blob)
    size = lib.ZSTD_getFrameContentSize(blob, len(blob))
    if size >= (1 << 64) - 2:  # unknown (2^64 - 1) or not a frame (2^64 - 2)
        raise ValueError("not a zstd frame with a content size")
    out = ctypes.create_string_buffer(max(size, 1))
    n = lib.ZSTD_decompress(out, size, blob, len(blob))
    if lib.ZSTD_isError(n) or n != size:
        raise ValueError("corrupt zstd frame")
    return out.raw[:n]


def compress(data: bytes, kind: str, level: int) -> bytes:
    if kind == "none":
        return bytes(data)
    if kind == "zlib":
        return zlib.compress(bytes(data), level)
    if kind == "lzma":
        return lzma.compress(bytes(data), format=lzma.FORMAT_XZ, preset=level)
    if kind == "zstd":
        return _zstd_compress(data, level)
    raise ValueError(kind)


def decompress(blob: bytes, kind: str) -> bytes:
    if kind == "none":
        return bytes(blob)
    if kind == "zlib":
        return zlib.decompress(blob)
    if kind == "lzma":
        return lzma.decompress(blob, format=lzma.FORMAT_XZ)
    if kind == "zstd":
        return _zstd_decompress(blob)
    raise ValueError(kind)
