"""A carry-propagating range coder over integer CDFs (Python integers).

The paper codes committed symbols with a statistical coder (rANS).  The
workloads name a range coder ("16-bit CDF precision with a 32-bit range
coder"), so this is a W-bit range coder with P-bit CDFs:

encode(start, f):  r = range >> P;  low += r * start;  range = r * f;
                   a carry out of bit W is added into the bytes already
                   emitted; while range < 2**(W-8) emit the top byte of low
                   and shift low and range left by 8 bits.
finish():          emit the W/8 bytes of low, most significant first.
decode(cdf):       track D = code - low; t = D // r (t >= 2**P is a corrupt
                   stream); the symbol s has cdf[s] <= t < cdf[s+1];
                   D -= r * cdf[s]; range = r * f_s; renormalise by shifting
                   in bytes (zeros past the end).
"""
from __future__ import annotations

import bisect
import math


class CorruptStream(ValueError):
    pass


class RangeEncoder:
    def __init__(self, W: int, P: int):
        if W % 8 or P > W - 16:
            raise ValueError("unsupported coder width / CDF precision")
        self.W, self.P = W, P
        self.low = 0
        self.range = (1 << W) - 1
        self.out = bytearray()
        self.ranges = []            # range before each symbol (for code-length checks)

    def encode(self, start: int, freq: int) -> None:
        if freq <= 0 or start < 0 or start + freq > (1 << self.P):
            raise ValueError("bad symbol interval")
        self.ranges.append(self.range)
        r = self.range >> self.P
        self.low += r * start
        self.range = r * freq
        if self.low >> self.W:
            self.low -= 1 << self.W
            i = len(self.out) - 1
            while self.out[i] == 0xFF:
                self.out[i] = 0
                i -= 1
            self.out[i] += 1
        while self.range < (1 << (self.W - 8)):
            self.out.append((self.low >> (self.W - 8)) & 0xFF)
            self.low = (self.low << 8) & ((1 << self.W) - 1)
            self.range <<= 8

    def code_length_bits(self) -> float:
        """Bits consumed so far: 8 per emitted byte plus log2(range_0 / range)."""
        return 8.0 * len(self.out) + math.log2(((1 << self.W) - 1) / self.range)

    def finish(self) -> bytes:
        for i in range(self.W // 8):
            self.out.append((self.low >> (self.W - 8 - 8 * i)) & 0xFF)
        return bytes(self.out)


class RangeDecoder:
    def __init__(self, data: bytes, W: int, P: int):
        self.data, self.W, self.P = data, W, P
        self.pos = 0
        self.range = (1 << W) - 1
        self.D = 0
        for _ in range(W // 8):
            self.D = (self.D << 8) | self._byte()

    def _byte(self) -> int:
        b = self.data[self.pos] if self.pos < len(self.data) else 0
        self.pos += 1
        return b

    def decode(self, cdf) -> int:
        r = self.range >> self.P
        t = self.D // r
        if t >= (1 << self.P):
            raise CorruptStream("range decoder target out of range")
        s = bisect.bisect_right(cdf, t) - 1
        lo, hi = int(cdf[s]), int(cdf[s + 1])
        self.D -= r * lo
        self.range = r * (hi - lo)
        while self.range < (1 << (self.W - 8)):
            self.D = (self.D << 8) | self._byte()
            self.range <<= 8
        return s


# ---------------------------------------------------------------------------
# rANS (range Asymmetric Numeral Systems, Duda 2013), the statistical coder
# the paper adopts.  State x in [L, L * 2^32) with L = 2^31, 32-bit words, so
# any P <= 31 works.  Coding a symbol with interval [start, start + f) of a
# 2^P total maps x to floor(x / f) * 2^P + (x mod f) + start, after first
# writing the low word of x while x >= (L >> P) * 2^32 * f.  rANS is last in,
# first out: the encoder keeps the chunk's intervals and codes them in
# reverse, so the decoder reads them in coding order.  Stream: the final
# state as 8 little-endian bytes, then the 32-bit words in the order the
# decoder consumes them (little-endian).  Decoding ends in state L; any other
# end state is a corrupt stream.
RANS_L = 1 << 31


class RansEncoder:
    def __init__(self, P: int):
        if not 1 <= P <= 31:
            raise ValueError("rANS needs 1 <= P <= 31")
        self.P = P
        self.intervals = []

    def encode(self, start: int, freq: int) -> None:
        if freq <= 0 or start < 0 or start + freq > (1 << self.P):
            raise ValueError("bad symbol interval")
        self.intervals.append((start, freq))

    def finish(self) -> bytes:
        x, words = RANS_L, []
        for start, f in reversed(self.intervals):
            x_max = ((RANS_L >> self.P) << 32) * f
            while x >= x_max:
                words.append(x & 0xFFFFFFFF)
                x >>= 32
            x = (x // f << self.P) + (x % f) + start
        out = bytearray(x.to_bytes(8, "little"))
        for w in reversed(words):
            out += w.to_bytes(4, "little")
        return bytes(out)


class RansDecoder:
    def __init__(self, data: bytes, P: int):
        if len(data) < 8 or (len(data) - 8) % 4:
            raise CorruptStream("rANS stream length")
        self.data, self.P = data, P
        self.x = int.from_bytes(data[:8], "little")
        self.pos = 8
        if not RANS_L <= self.x < (RANS_L << 32):
            raise CorruptStream("rANS state out of range")

    def decode(self, cdf) -> int:
        mask = (1 << self.P) - 1
        slot = self.x & mask
        s = bisect.bisect_right(cdf, slot) - 1
        lo, hi = int(cdf[s]), int(cdf[s + 1])
        self.x = (hi - lo) * (self.x >> self.P) + slot - lo
        while self.x < RANS_L:
            if self.pos + 4 > len(self.data):
                raise CorruptStream("rANS stream ended early")
            self.x = (self.x << 32) | int.from_bytes(self.data[self.pos:self.pos + 4], "little")
            self.pos += 4
        return s

    def done(self) -> bool:
        """True when the stream is fully consumed and the state is back at L."""
        return self.pos == len(self.data) and self.x == RANS_L
