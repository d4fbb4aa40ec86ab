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
