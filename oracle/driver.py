"""The iterative diffusion compression pipeline (Diffusion-Based Compression
Pipeline section, Figure 1).

Per window (chunk) of the input: start from the state S(0) in which every
position is masked except the c initial-context positions (Initial Context
Strategies; c = 0 is the fully masked start), then repeat until no position is
masked: one forward pass gives a distribution at every masked position; the
commitment schedule picks positions; their true symbols are coded with their
predicted (quantised) distributions in ascending position order; the symbols
are revealed in the state.  Decoding replays exactly the same decisions from
the header parameters alone.  Windows are non-overlapping and independent, so
every chunk has its own coder state and bitstream; a final partial chunk is
coded at its own length.

Chunk payload: the initial context (c little-endian u16 positions, ascending,
then their c u32 symbols) followed by the coder's bytes -- for the symbol
ranking back end, the varint ranks of the coded symbols in coding order.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

import workloads as wl

from . import model as M
from . import ranking as R
from .cdf import cdf_row
from .coder import CorruptStream, RangeDecoder, RangeEncoder, RansDecoder, RansEncoder
from .context import attention_context
from .schedule import block_sizes, entropy_bits, select


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


def context_positions(codec, T: int, chunk_index: int, shape=None, W=None,
                      tokens=None) -> np.ndarray:
    """The chunk's initial-context positions (ascending): the first c, the c
    positions with the smallest seeded keys (seed context_seed + chunk index),
    or the c highest attention-rollout scores (needs the model and tokens)."""
    c = min(int(codec.context), T)
    if c == 0:
        return np.zeros(0, dtype=np.int64)
    if codec.context_kind == "attention":
        return attention_context(shape, W, tokens, c)
    if codec.context_kind == "contiguous":
        return np.arange(c, dtype=np.int64)
    if codec.context_kind == "random":
        perm = wl.seeded_permutation(codec.context_seed + chunk_index, T)
        return np.sort(perm[:c])
    raise ValueError(codec.context_kind)


class _RankEncoder:
    def __init__(self):
        self.ranks = []

    def finish(self) -> bytes:
        return R.varint_encode(self.ranks)


class _RankDecoder:
    def __init__(self, data: bytes):
        self.data, self.pos = data, 0

    def next_rank(self) -> int:
        (r,), self.pos = R.varint_decode(self.data, 1, self.pos)
        return r

    def done(self) -> bool:
        return self.pos == len(self.data)


def _encoder(codec):
    if codec.coder == "rank":
        return _RankEncoder()
    if codec.coder == "rans":
        return RansEncoder(codec.cdf_bits)
    return RangeEncoder(codec.coder_bits, codec.cdf_bits)


def _decoder(codec, data: bytes):
    if codec.coder == "rank":
        return _RankDecoder(data)
    if codec.coder == "rans":
        return RansDecoder(data, codec.cdf_bits)
    return RangeDecoder(data, codec.coder_bits, codec.cdf_bits)


def _selection(codec, state, mask_id, pos, H, sizes, k):
    if codec.schedule == "entropy":
        return select(H, pos, codec.tau_bits, codec.m_min, codec.m_max)
    masked = np.flatnonzero(state == mask_id)
    return masked[: sizes[k]]


def encode_chunk(shape, W, tokens: np.ndarray, codec, forced: Optional[list] = None,
                 chunk_index: int = 0) -> ChunkResult:
    """Encode one chunk.  ``forced`` replays a given list of per-pass
    selections instead of the schedule's own (used to compare code lengths
    along another implementation's trajectory)."""
    tokens = np.asarray(tokens, dtype=np.int64)
    T = tokens.shape[0]
    state = np.full(T, shape.mask_id, dtype=np.int64)
    ctx = context_positions(codec, T, chunk_index, shape, W, tokens)
    state[ctx] = tokens[ctx]
    sizes = None if codec.schedule == "entropy" else block_sizes(codec, T - len(ctx))
    enc = _encoder(codec)
    res = ChunkResult(b"", 0)
    P = codec.cdf_bits
    while np.any(state == shape.mask_id):
        lg, pos, H = _pass(shape, W, state)
        if forced is not None:
            sel = np.asarray(forced[res.passes], dtype=np.int64)
            if np.any(state[sel] != shape.mask_id) or len(sel) == 0:
                raise ValueError("forced selection is not a set of masked positions")
        else:
            sel = _selection(codec, state, shape.mask_id, pos, H, sizes, res.passes)
        row_of = {int(p): i for i, p in enumerate(pos)}
        for p in sel:
            row = lg[row_of[int(p)]]
            s = int(tokens[p])
            if codec.coder == "rank":
                enc.ranks.append(R.rank_of(row, s))
                continue
            cdf = cdf_row(row, P)
            f = int(cdf[s + 1] - cdf[s])
            enc.encode(int(cdf[s]), f)
            res.ideal_bits += -math.log2(f / float(1 << P))
            pr = M.softmax(row)
            res.unquantised_bits += -math.log2(pr[s])
        res.selections.append(sel)
        res.entropies.append(H)
        state[sel] = tokens[sel]
        res.passes += 1
    head = ctx.astype("<u2").tobytes() + tokens[ctx].astype("<u4").tobytes()
    if codec.coder in ("rans", "rank"):
        body = enc.finish()
        res.coded_bits = 8.0 * len(body)
    else:
        res.coded_bits = enc.code_length_bits()
        body = enc.finish()
    res.payload = head + body
    return res


def decode_chunk(shape, W, payload: bytes, T: int, codec) -> np.ndarray:
    c = min(int(codec.context), T)
    if len(payload) < 6 * c:
        raise CorruptStream("chunk shorter than its initial context")
    ctx = np.frombuffer(payload[: 2 * c], dtype="<u2").astype(np.int64)
    sym = np.frombuffer(payload[2 * c: 6 * c], dtype="<u4").astype(np.int64)
    if np.any(ctx >= T) or np.any(np.diff(ctx) <= 0) or np.any(sym >= shape.vocab):
        raise CorruptStream("bad initial context")
    state = np.full(T, shape.mask_id, dtype=np.int64)
    state[ctx] = sym
    sizes = None if codec.schedule == "entropy" else block_sizes(codec, T - c)
    dec = _decoder(codec, payload[6 * c:])
    P = codec.cdf_bits
    k = 0
    while np.any(state == shape.mask_id):
        lg, pos, H = _pass(shape, W, state)
        sel = _selection(codec, state, shape.mask_id, pos, H, sizes, k)
        row_of = {int(p): i for i, p in enumerate(pos)}
        for p in sel:
            row = lg[row_of[int(p)]]
            if codec.coder == "rank":
                r = dec.next_rank()
                if r >= shape.vocab:
                    raise CorruptStream("rank out of range")
                state[p] = R.symbol_at(row, r)
            else:
                state[p] = dec.decode(cdf_row(row, P))
        k += 1
    if codec.coder in ("rans", "rank") and not dec.done():
        raise CorruptStream("coded stream has trailing or missing data")
    return state


def chunk_bounds(n: int, chunk_len: int):
    return [(s, min(n, s + chunk_len)) for s in range(0, n, chunk_len)]


def encode(shape, W, tokens: np.ndarray, codec) -> List[ChunkResult]:
    return [encode_chunk(shape, W, tokens[a:b], codec, chunk_index=i)
            for i, (a, b) in enumerate(chunk_bounds(len(tokens), codec.chunk_len))]


def decode(shape, W, payloads: List[bytes], n: int, codec) -> np.ndarray:
    parts = [decode_chunk(shape, W, p, b - a, codec)
             for p, (a, b) in zip(payloads, chunk_bounds(n, codec.chunk_len))]
    return np.concatenate(parts) if parts else np.zeros(0, dtype=np.int64)


def pack_payloads(payloads: List[bytes], codec) -> bytes:
    """The container's payload section: chunk payloads concatenated, compressed
    as one block for the symbol ranking back end."""
    blob = b"".join(payloads)
    if codec.coder == "rank":
        return R.compress(blob, codec.rank_compressor, codec.rank_level)
    return blob
