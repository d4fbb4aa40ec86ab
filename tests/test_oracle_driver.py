"""Pins of the oracle's iterative pipeline: exact round trips, coverage,
schedule replay and code-length bounds."""
import dataclasses
import math

import numpy as np
import pytest

import workloads as wl
from oracle import driver as OD
from oracle import weights as OW


def tiny(chunk_len, **codec):
    w = wl.WORKLOADS["tiny"]
    c = dataclasses.replace(w.codec, chunk_len=chunk_len, **codec)
    return w.model, OW.Weights(w.model), c


@pytest.mark.parametrize("n,chunk,k", [(8, 8, 1), (24, 8, 3), (19, 8, 4), (64, 32, 4)])
def test_roundtrip_fixed_k(n, chunk, k):
    shape, W, codec = tiny(chunk, m_min=k, m_max=k)
    toks = wl.markov2_bytes(n, 40 + n)
    res = OD.encode(shape, W, toks, codec)
    # coverage: every position is committed exactly once per chunk, u_k = k
    for (a, b), r in zip(OD.chunk_bounds(n, chunk), res):
        allsel = np.concatenate(r.selections)
        assert sorted(allsel.tolist()) == list(range(b - a))
        assert r.passes == math.ceil((b - a) / k)
        assert all(len(s) == min(k, b - a - k * i) for i, s in enumerate(r.selections))
    dec = OD.decode(shape, W, [r.payload for r in res], n, codec)
    assert np.array_equal(dec, toks)


@pytest.mark.parametrize("tau,mmin,mmax", [(7.2, 1, 5), (0.0, 2, 8), (100.0, 1, 3)])
def test_roundtrip_threshold_schedule(tau, mmin, mmax):
    shape, W, codec = tiny(32, tau_bits=tau, m_min=mmin, m_max=mmax)
    toks = wl.markov2_bytes(32, 5)
    (r,) = OD.encode(shape, W, toks, codec)
    assert sorted(np.concatenate(r.selections).tolist()) == list(range(32))
    assert all(1 <= len(s) <= mmax for s in r.selections)
    assert np.array_equal(OD.decode(shape, W, [r.payload], 32, codec), toks)


def test_code_length_within_two_bits_of_ideal():
    shape, W, codec = tiny(256)
    toks = wl.make_tokens(wl.WORKLOADS["tiny"], 256)
    (r,) = OD.encode(shape, W, toks, codec)
    assert 0.0 <= r.coded_bits - r.ideal_bits < 2.0
    # the payload is the coded length rounded up plus the W-bit flush
    assert len(r.payload) * 8 - r.coded_bits <= 32 + 8
    # quantisation to 16-bit CDFs costs at most ~V/2**16 of the mass per symbol
    assert r.ideal_bits - r.unquantised_bits < 256 * -math.log2(1 - 256 / 2 ** 16) + 1e-6


def test_forced_trajectory_replays_own_selection():
    shape, W, codec = tiny(16, m_min=3, m_max=3)
    toks = wl.markov2_bytes(16, 9)
    (r,) = OD.encode(shape, W, toks, codec)
    (f,) = [OD.encode_chunk(shape, W, toks, codec, forced=r.selections)]
    assert f.payload == r.payload and f.passes == r.passes


def test_wrong_payload_does_not_roundtrip():
    shape, W, codec = tiny(16, m_min=4, m_max=4)
    toks = wl.markov2_bytes(16, 3)
    (r,) = OD.encode(shape, W, toks, codec)
    bad = bytearray(r.payload)
    bad[0] ^= 0x40
    try:
        dec = OD.decode(shape, W, [bytes(bad)], 16, codec)
    except ValueError:
        return
    assert not np.array_equal(dec, toks)


# ------------------------------------------------- block schedules, rANS, initial context
from oracle.coder import CorruptStream  # noqa: E402
from oracle.schedule import block_sizes  # noqa: E402


@pytest.mark.parametrize("codec_kw", [
    dict(schedule="uniform", blocks=5),
    dict(schedule="uniform", blocks=24),                  # autoregressive: one per pass
    dict(schedule="progressive", u1=1, growth=1.7),
    dict(schedule="uniform", blocks=3, coder="rans"),
    dict(schedule="progressive", u1=2, growth=1.3, context=4, context_kind="random", context_seed=7),
    dict(schedule="uniform", blocks=4, context=3, context_kind="contiguous", coder="rans"),
    dict(m_min=3, m_max=3, context=5, context_kind="random", context_seed=1, coder="rans"),
])
def test_block_schedules_context_and_rans_roundtrip(codec_kw):
    shape, W, codec = tiny(24, **codec_kw)
    toks = wl.markov2_bytes(53, 11)
    res = OD.encode(shape, W, toks, codec)
    for i, ((a, b), r) in enumerate(zip(OD.chunk_bounds(53, 24), res)):
        T = b - a
        ctx = OD.context_positions(codec, T, i)
        assert len(ctx) == min(codec.context, T) and len(set(ctx.tolist())) == len(ctx)
        if codec.context_kind == "contiguous":
            assert ctx.tolist() == list(range(len(ctx)))
        rest = sorted(set(range(T)) - set(ctx.tolist()))
        allsel = np.concatenate(r.selections) if r.selections else np.zeros(0, dtype=np.int64)
        assert sorted(allsel.tolist()) == rest          # coverage of the masked positions
        if codec.schedule != "entropy":
            # left to right: the passes commit consecutive runs of the masked positions
            assert allsel.tolist() == rest
            assert [len(s) for s in r.selections] == block_sizes(codec, len(rest))
    dec = OD.decode(shape, W, [r.payload for r in res], 53, codec)
    assert np.array_equal(dec, toks)


def test_autoregressive_special_case():
    shape, W, codec = tiny(12, schedule="uniform", blocks=12)
    toks = wl.markov2_bytes(12, 3)
    (r,) = OD.encode(shape, W, toks, codec)
    assert [s.tolist() for s in r.selections] == [[i] for i in range(12)]


def test_full_context_chunk_stores_symbols_only():
    shape, W, codec = tiny(10, context=16, coder="rans")
    toks = wl.markov2_bytes(10, 4)
    (r,) = OD.encode(shape, W, toks, codec)
    assert r.passes == 0 and len(r.payload) == 6 * 10 + 8
    assert np.array_equal(OD.decode(shape, W, [r.payload], 10, codec), toks)


def test_rans_corrupt_tail_is_detected():
    shape, W, codec = tiny(16, m_min=4, m_max=4, coder="rans")
    toks = wl.markov2_bytes(16, 8)
    (r,) = OD.encode(shape, W, toks, codec)
    bad = r.payload[:-4]
    with pytest.raises(CorruptStream):
        OD.decode(shape, W, [bad], 16, codec)
