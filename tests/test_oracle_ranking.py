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
