// Host rANS coder (range Asymmetric Numeral Systems, Duda 2013) over P-bit
// integer CDFs: the statistical coder the paper adopts (Preliminaries).
//
// State x in [L, L 2^32), L = 2^31, written in 32-bit words, so P <= 31.
// Coding the interval [start, start + f) of a 2^P total maps
// x -> floor(x / f) 2^P + (x mod f) + start, after moving the low word of x
// out while x >= (L >> P) 2^32 f.  rANS is last in, first out: the encoder
// keeps a chunk's intervals and codes them in reverse, so the decoder meets
// them in coding order.  Stream: the final state (8 bytes, little endian),
// then the words in the order the decoder reads them (4 bytes each, little
// endian).  Decoding ends in state L; any other end is a corrupt stream.
#pragma once

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <vector>

namespace dlmc {

constexpr uint64_t RANS_L = 1ull << 31;

class RansEncoder {
 public:
  void reset(int P) {
    P_ = P;
    iv_.clear();
  }
  // start + freq <= 2^P, freq >= 1 (checked by the caller)
  void encode(uint32_t start, uint32_t freq) { iv_.push_back({start, freq}); }
  std::vector<uint8_t> finish() {
    uint64_t x = RANS_L;
    std::vector<uint32_t> words;
    for (size_t i = iv_.size(); i-- > 0;) {
      const uint64_t f = iv_[i].freq;
      const uint64_t x_max = ((RANS_L >> P_) << 32) * f;
      while (x >= x_max) {
        words.push_back((uint32_t)x);
        x >>= 32;
      }
      x = ((x / f) << P_) + (x % f) + iv_[i].start;
    }
    std::vector<uint8_t> out(8 + 4 * words.size());
    for (int b = 0; b < 8; ++b) out[b] = (uint8_t)(x >> (8 * b));
    size_t o = 8;
    for (size_t i = words.size(); i-- > 0; o += 4)
      for (int b = 0; b < 4; ++b) out[o + b] = (uint8_t)(words[i] >> (8 * b));
    iv_.clear();
    return out;
  }

 private:
  struct Interval {
    uint32_t start, freq;
  };
  int P_ = 16;
  std::vector<Interval> iv_;
};

class RansDecoder {
 public:
  // false for a stream that cannot be an rANS stream (length, initial state)
  bool reset(const uint8_t* data, size_t len, int P) {
    data_ = data;
    len_ = len;
    P_ = P;
    pos_ = 8;
    x_ = 0;
    if (len < 8 || (len - 8) % 4) return false;
    for (int b = 7; b >= 0; --b) x_ = (x_ << 8) | data[b];
    return x_ >= RANS_L && (x_ >> 31) < (1ull << 32);
  }
  // returns the symbol, or -1 for a corrupt stream
  int decode(const uint32_t* cdf, int V) {
    const uint64_t mask = (1ull << P_) - 1;
    const uint32_t slot = (uint32_t)(x_ & mask);
    const int s = (int)(std::upper_bound(cdf, cdf + V + 1, slot) - cdf) - 1;
    if (s < 0 || s >= V || cdf[s + 1] <= cdf[s]) return -1;
    x_ = (uint64_t)(cdf[s + 1] - cdf[s]) * (x_ >> P_) + slot - cdf[s];
    while (x_ < RANS_L) {
      if (pos_ + 4 > len_) return -1;
      uint32_t w;
      std::memcpy(&w, data_ + pos_, 4);
      pos_ += 4;
      x_ = (x_ << 32) | w;
    }
    return s;
  }
  bool done() const { return pos_ == len_ && x_ == RANS_L; }
  uint64_t state() const { return x_; }
  size_t position() const { return pos_; }

 private:
  const uint8_t* data_ = nullptr;
  size_t len_ = 0, pos_ = 8;
  int P_ = 16;
  uint64_t x_ = 0;
};

}  // namespace dlmc
