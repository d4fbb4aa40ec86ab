"""The iterative diffusion compression pipeline (Diffusion-Based Compression
Pipeline section, Figure 1).

Per window (chunk) of the input: start from the fully masked state S(0)
(initial context c = 0), then repeat until no position is masked: one forward
pass gives a distribution at every masked position; the commitment schedule
picks positions; their true symbols are coded with their predicted (quantised)
distributions in ascending position order; the symbols are revealed in the
state.  Decoding replays exactly the same decisions from the header
parameters alone.  Windows are non-overlapping and independent, so every
chunk has its own coder state and bitstream; a final partial chunk is coded at
its own length.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from . import model as M
from .cdf import cdf_row
from .coder import RangeDecoder, RangeEncoder
from .schedule import entropy_bits, select


@dataclass
class ChunkResult:
    payload: bytes
    passes: int
    selections: List[np.ndarray] = field(default_factory=list)
    entropies: List[np.ndarray] = field(default_factory=list)
    ideal_bits: float = 0.0       # sum of -log2 q over coded symbols (q = f / 2**P)
    coded_bits: float = 0.0       # fractional coder length before the flush
    unquantised_bits: float = 0.0  # sum of -log2 p with the fp64 softmax p


def _pass(shape, W, state):
    lg, pos = M.logits(shape, W, state)
    return lg, pos, entropy_bits(lg)


def encode_chunk(shape, W, tokens: np.ndarray, codec, forced: Optional[list] = None) -> ChunkResult:
    """Encode one chunk.  ``forced`` replays a given list of per-pass
    selections instead of the schedule's own (used to compare code lengths
    along another implementation's trajectory)."""
    tokens = np.asarray(tokens, dtype=np.int64)
    T = tokens.shape[0]
    state = np.full(T, shape.mask_id, dtype=np.int64)
    enc = RangeEncoder(codec.coder_bits, codec.cdf_bits)
    res = ChunkResult(b"", 0)
    P = codec.cdf_bits
    while np.any(state == shape.mask_id):
        lg, pos, H = _pass(shape, W, state)
        if forced is not None:
            sel = np.asarray(forced[res.passes], dtype=np.int64)
            if np.any(state[sel] != shape.mask_id) or len(sel) == 0:
                raise ValueError("forced selection is not a set of masked positions")
        else:
            sel = select(H, pos, codec.tau_bits, codec.m_min, codec.m_max)
        row_of = {int(p): i for i, p in enumerate(pos)}
        for p in sel:
            row = lg[row_of[int(p)]]
            cdf = cdf_row(row, P)
            s = int(tokens[p])
            f = int(cdf[s + 1] - cdf[s])
            enc.encode(int(cdf[s]), f)
            res.ideal_bits += -math.log2(f / float(1 << P))
            pr = M.softmax(row)
            res.unquantised_bits += -math.log2(pr[s])
        res.selections.append(sel)
        res.entropies.append(H)
        state[sel] = tokens[sel]
        res.passes += 1
    res.coded_bits = enc.code_length_bits()
    res.payload = enc.finish()
    return res


def decode_chunk(shape, W, payload: bytes, T: int, codec) -> np.ndarray:
    state = np.full(T, shape.mask_id, dtype=np.int64)
    dec = RangeDecoder(payload, codec.coder_bits, codec.cdf_bits)
    P = codec.cdf_bits
    while np.any(state == shape.mask_id):
        lg, pos, H = _pass(shape, W, state)
        sel = select(H, pos, codec.tau_bits, codec.m_min, codec.m_max)
        row_of = {int(p): i for i, p in enumerate(pos)}
        for p in sel:
            cdf = cdf_row(lg[row_of[int(p)]], P)
            state[p] = dec.decode(cdf)
    return state


def chunk_bounds(n: int, chunk_len: int):
    return [(s, min(n, s + chunk_len)) for s in range(0, n, chunk_len)]


def encode(shape, W, tokens: np.ndarray, codec) -> List[ChunkResult]:
    return [encode_chunk(shape, W, tokens[a:b], codec) for a, b in chunk_bounds(len(tokens), codec.chunk_len)]


def decode(shape, W, payloads: List[bytes], n: int, codec) -> np.ndarray:
    parts = [decode_chunk(shape, W, p, b - a, codec)
             for p, (a, b) in zip(payloads, chunk_bounds(n, codec.chunk_len))]
    return np.concatenate(parts) if parts else np.zeros(0, dtype=np.int64)
