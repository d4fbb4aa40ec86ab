"""Pins of the oracle CDF quantisation and range coder."""
import math

import numpy as np
import pytest

from oracle import cdf as OC
from oracle import coder as ORC


@pytest.mark.parametrize("V,P", [(256, 16), (32768, 24), (126464, 24), (5, 8)])
def test_cdf_invariants(V, P):
    rng = np.random.default_rng(V)
    lg = rng.standard_normal(V) * 6.0
    g = OC.quantise_g(lg)
    cdf = OC.integer_cdf(g, P)
    f = np.diff(cdf)
    assert cdf[0] == 0 and cdf[-1] == 1 << P
    assert f.min() >= 1
    assert g.max() == 1 << 24 and g[np.argmax(lg)] == 1 << 24
    # f is nondecreasing in g away from the argmax, which holds the largest f
    a = int(np.argmax(g))
    rest = np.delete(np.arange(V), a)
    order = rest[np.argsort(g[rest], kind="stable")]
    assert np.all(np.diff(f[order]) >= 0) and f[a] >= f.max()
    R = (1 << P) - int((1 + (g * ((1 << P) - V)) // int(g.sum())).sum())
    assert 0 <= R < V


@pytest.mark.parametrize("V,P", [(256, 16), (1000, 16), (126464, 24)])
def test_cdf_all_equal_closed_form(V, P):
    cdf = OC.cdf_row(np.zeros(V), P)
    f = np.diff(cdf)
    base = 1 + ((1 << P) - V) // V
    R = ((1 << P) - V) % V
    assert f[0] == base + R and np.all(f[1:] == base)


@pytest.mark.parametrize("V,P", [(256, 16), (126464, 24)])
def test_cdf_single_dominant_closed_form(V, P):
    lg = np.full(V, -1000.0)
    lg[V // 3] = 0.0
    f = np.diff(OC.cdf_row(lg, P))
    assert f[V // 3] == (1 << P) - (V - 1)
    assert np.all(np.delete(f, V // 3) == 1)


def test_cdf_remainder_goes_to_lowest_maximal_index():
    g = np.array([5, 1 << 24, 7, 1 << 24, 0])
    f = np.diff(OC.integer_cdf(g, 8))
    base = 1 + (g * (256 - 5)) // int(g.sum())
    R = 256 - int(base.sum())
    assert R > 0
    assert f[1] == base[1] + R and f[3] == base[3]


def test_range_coder_hand_example():
    # W=32, P=16.  range0 = 2**32-1, r = 0xFFFF.
    # sym1 (start=0x8000, f=0x4000): low = 0xFFFF*0x8000 = 0x7FFF8000,
    #   range = 0xFFFF*0x4000 = 0x3FFFC000 (>= 2**24: no output).
    # sym2 (start=1, f=1): r = 0x3FFF; low = 0x7FFFBFFF; range = 0x3FFF
    #   -> emit 0x7F (range 0x3FFF00, low 0xFFBFFF00), emit 0xFF (range 0x3FFF0000,
    #   low 0xBFFF0000).  flush -> BF FF 00 00.
    enc = ORC.RangeEncoder(32, 16)
    enc.encode(0x8000, 0x4000)
    enc.encode(1, 1)
    assert enc.finish() == bytes([0x7F, 0xFF, 0xBF, 0xFF, 0x00, 0x00])
    dec = ORC.RangeDecoder(bytes([0x7F, 0xFF, 0xBF, 0xFF, 0x00, 0x00]), 32, 16)
    c1 = [0, 0x8000, 0xC000, 0x10000]
    c2 = [0, 1, 2, 0x10000]
    assert dec.decode(c1) == 1 and dec.decode(c2) == 1


def random_cdf(rng, V, P):
    w = rng.dirichlet(np.full(V, 0.3))
    lg = np.log(np.maximum(w, 1e-300))
    return OC.cdf_row(lg, P)


@pytest.mark.parametrize("W,P,V", [(32, 16, 256), (64, 24, 1000), (32, 16, 3)])
def test_range_coder_roundtrip_and_exact_length_identity(W, P, V):
    rng = np.random.default_rng(W + V)
    n = 600
    cdfs = [random_cdf(rng, V, P) for _ in range(n)]
    syms = [int(rng.choice(V, p=np.diff(c) / 2.0 ** P)) for c in cdfs]
    enc = ORC.RangeEncoder(W, P)
    excess = 0.0
    carries = 0
    for c, s in zip(cdfs, syms):
        before = bytes(enc.out)
        r = enc.range >> P
        excess += math.log2(enc.range / (r * 2.0 ** P))
        enc.encode(int(c[s]), int(c[s + 1] - c[s]))
        carries += bytes(enc.out[: len(before)]) != before
    # exact identity: coded length = sum -log2 q + sum log2(range_i / (r_i 2**P))
    q_bits = sum(-math.log2((int(c[s + 1] - c[s])) / 2.0 ** P) for c, s in zip(cdfs, syms))
    assert enc.code_length_bits() == pytest.approx(q_bits + excess, abs=1e-7)
    assert excess <= n * math.log2(1 + 2.0 ** -(W - 8 - P)) + 1e-9
    payload = enc.finish()
    dec = ORC.RangeDecoder(payload, W, P)
    assert [dec.decode(c) for c in cdfs] == syms
    if W == 32 and V == 256:
        assert carries > 0          # the carry path was exercised


def test_range_decoder_rejects_out_of_range_target():
    dec = ORC.RangeDecoder(b"\xff" * 8, 32, 16)
    with pytest.raises(ORC.CorruptStream):
        dec.decode([0, 1, 1 << 16])


# ---------------------------------------------------------------- rANS
from oracle.coder import RANS_L, CorruptStream, RansDecoder, RansEncoder  # noqa: E402


def _random_cdf(rng, V, P):
    w = rng.random(V) ** 3 + 1e-9
    f = 1 + (w / w.sum() * ((1 << P) - V)).astype(np.int64)
    f[int(np.argmax(f))] += (1 << P) - int(f.sum())
    return np.concatenate([[0], np.cumsum(f)]).astype(np.int64), f


@pytest.mark.parametrize("P", [2, 16, 24, 31])
def test_rans_roundtrip(P):
    rng = np.random.default_rng(P)
    for trial in range(10):
        V = int(rng.integers(2, min(300, 1 << P) + 1))
        cdf, f = _random_cdf(rng, V, P)
        syms = rng.integers(0, V, size=int(rng.integers(0, 2000)))
        enc = RansEncoder(P)
        for s in syms:
            enc.encode(int(cdf[s]), int(f[s]))
        data = enc.finish()
        dec = RansDecoder(data, P)
        assert [dec.decode(cdf) for _ in syms] == list(syms)
        assert dec.done()


@pytest.mark.parametrize("P", [8, 16, 24])
def test_rans_length_bound(P):
    """Coded length minus the information I = sum log2(2^P / f) lies in
    (32 - n d, 64 + n d]: the initial state L = 2^31 and the 64-bit flush
    cost 95 - log2(x_final) bits with x_final in [2^31, 2^63), and each step
    maps x to x 2^P / f within a factor (1 +- 2^(P-31)), d = -log2(1 - 2^(P-31))."""
    rng = np.random.default_rng(100 + P)
    d = -math.log2(1.0 - 2.0 ** (P - 31))
    for trial in range(20):
        V = int(rng.integers(2, min(500, 1 << P) + 1))
        cdf, f = _random_cdf(rng, V, P)
        syms = rng.integers(0, V, size=int(rng.integers(1, 4000)))
        enc = RansEncoder(P)
        info = 0.0
        for s in syms:
            enc.encode(int(cdf[s]), int(f[s]))
            info += math.log2((1 << P) / f[s])
        excess = 8 * len(enc.finish()) - info
        n = len(syms)
        assert 32 - n * d - 1e-9 < excess <= 64 + n * d + 1e-9, (trial, excess)


def test_rans_empty_and_corrupt_streams():
    data = RansEncoder(16).finish()
    assert data == RANS_L.to_bytes(8, "little")      # no symbol: the initial state only
    assert RansDecoder(data, 16).done()
    with pytest.raises(CorruptStream):
        RansDecoder(b"\x00" * 8, 16)                  # state below L
    with pytest.raises(CorruptStream):
        RansDecoder(data + b"\x01", 16)               # not a whole number of words
