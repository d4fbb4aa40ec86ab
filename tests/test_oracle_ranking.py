"""Pins of the oracle's symbol ranking back end: ranks against a counting
definition on tiny rows with ties, published varint encodings, and
compressor round trips."""
import dataclasses

import numpy as np
import pytest

import workloads as wl
from oracle import driver as OD
from oracle import ranking as R
from oracle import weights as OW


@pytest.mark.parametrize("seed", range(6))
def test_rank_matches_counting_definition(seed):
    rng = np.random.default_rng(seed)
    V = int(rng.integers(1, 40))
    lg = rng.integers(-3, 4, size=V).astype(np.float32)   # many ties
    ranks = [R.rank_of(lg, s) for s in range(V)]
    assert sorted(ranks) == list(range(V))                 # a permutation of 0..V-1
    for s in range(V):
        # symbols strictly more probable, plus equally probable ones with a lower id
        expect = int(np.sum(lg > lg[s]) + np.sum(lg[:s] == lg[s]))
        assert ranks[s] == expect
        assert R.symbol_at(lg, ranks[s]) == s


def test_rank_special_cases():
    assert [R.rank_of(np.zeros(5), s) for s in range(5)] == [0, 1, 2, 3, 4]   # uniform: by id
    lg = np.full(7, -5.0)
    lg[4] = 3.0
    assert R.rank_of(lg, 4) == 0 and R.rank_of(lg, 0) == 1 and R.rank_of(lg, 6) == 6


def test_varint_published_examples():
    # unsigned LEB128, as in the Protocol Buffers encoding guide (300 -> AC 02)
    assert R.varint_encode([0, 1, 127, 128, 300]) == bytes([0, 1, 0x7F, 0x80, 0x01, 0xAC, 0x02])
    assert R.varint_encode([(1 << 63) - 1]) == bytes([0xFF] * 8 + [0x7F])
    vals = [0, 5, 127, 128, 16383, 16384, 2 ** 31, 126463]
    assert R.varint_decode(R.varint_encode(vals), len(vals)) == (vals, len(R.varint_encode(vals)))
    with pytest.raises(ValueError):
        R.varint_decode(b"\x80", 1)


@pytest.mark.parametrize("kind,level", [("none", 0), ("zlib", 9), ("lzma", 9), ("lzma", 0)])
def test_compressor_roundtrip(kind, level):
    data = R.varint_encode(np.random.default_rng(1).geometric(0.3, size=5000))
    blob = R.compress(data, kind, level)
    assert R.decompress(blob, kind) == data
    if kind != "none":
        assert len(blob) < len(data)


needs_zstd = pytest.mark.skipif(R.zstd_library() is None, reason="libzstd is not installed")


def zstd_frame(blocks, content_size):
    """A zstd frame written out from RFC 8878: magic 0xFD2FB528, a frame header
    descriptor with only Single_Segment_flag set (so a one-byte
    Frame_Content_Size follows, no window descriptor), then blocks, each a
    3-byte little-endian header (bit 0 Last_Block, bits 1-2 Block_Type: 0 Raw,
    1 RLE; bits 3-23 Block_Size) and its content."""
    assert content_size < 256
    out = bytearray((0xFD2FB528).to_bytes(4, "little")) + bytes([0x20, content_size])
    for i, (kind, payload, size) in enumerate(blocks):
        last = 1 if i == len(blocks) - 1 else 0
        out += (last | (kind << 1) | (size << 3)).to_bytes(3, "little") + payload
    return bytes(out)


@needs_zstd
def test_zstd_pinned_to_hand_built_frames():
    """The oracle's zstd decoder against frames built from the format's
    definition: a raw block, an RLE block, and a raw block followed by an RLE
    block; a frame with a damaged magic number is refused."""
    raw = bytes(range(7, 107))
    assert R.decompress(zstd_frame([(0, raw, len(raw))], len(raw)), "zstd") == raw
    assert R.decompress(zstd_frame([(1, b"\x2a", 200)], 200), "zstd") == b"\x2a" * 200
    two = zstd_frame([(0, b"abc", 3), (1, b"z", 5)], 8)
    assert R.decompress(two, "zstd") == b"abczzzzz"
    bad = bytearray(two)
    bad[0] ^= 1
    with pytest.raises(ValueError):
        R.decompress(bytes(bad), "zstd")


@needs_zstd
@pytest.mark.parametrize("level", [1, 19])
def test_zstd_roundtrip_and_frame_header(level):
    """Round trip at two levels; the frame starts with the magic number and
    states its content size (Single_Segment_flag or a nonzero
    Frame_Content_Size_flag), which the decoder needs."""
    data = R.varint_encode(np.random.default_rng(2).geometric(0.3, size=5000))
    blob = R.compress(data, "zstd", level)
    assert blob[:4] == (0xFD2FB528).to_bytes(4, "little")
    fhd = blob[4]
    assert (fhd & 0x20) or (fhd >> 6)
    assert R.decompress(blob, "zstd") == data and len(blob) < len(data)


@pytest.mark.parametrize("kw", [
    dict(m_min=4, m_max=4),
    dict(schedule="uniform", blocks=6, context=3, context_kind="random", context_seed=2),
    dict(tau_bits=6.0, m_min=1, m_max=6, context=2),
])
def test_rank_backend_roundtrip(kw):
    w = wl.WORKLOADS["tiny"]
    codec = dataclasses.replace(w.codec, chunk_len=24, coder="rank", rank_compressor="lzma",
                                rank_level=6, **kw)
    W = OW.Weights(w.model)
    toks = wl.markov2_bytes(53, 17)
    res = OD.encode(w.model, W, toks, codec)
    blob = OD.pack_payloads([r.payload for r in res], codec)
    assert R.decompress(blob, "lzma") == b"".join(r.payload for r in res)
    back = OD.decode(w.model, W, [r.payload for r in res], 53, codec)
    assert np.array_equal(back, toks)
