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
one block ("none", "zlib" at a level, "lzma" xz at a preset).
"""
from __future__ import annotations

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


def compress(data: bytes, kind: str, level: int) -> bytes:
    if kind == "none":
        return bytes(data)
    if kind == "zlib":
        return zlib.compress(bytes(data), level)
    if kind == "lzma":
        return lzma.compress(bytes(data), format=lzma.FORMAT_XZ, preset=level)
    raise ValueError(kind)


def decompress(blob: bytes, kind: str) -> bytes:
    if kind == "none":
        return bytes(blob)
    if kind == "zlib":
        return zlib.decompress(blob)
    if kind == "lzma":
        return lzma.decompress(blob, format=lzma.FORMAT_XZ)
    raise ValueError(kind)
