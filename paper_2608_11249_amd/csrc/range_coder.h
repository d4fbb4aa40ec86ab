// Host range coder over P-bit integer CDFs, W in {32, 64}.
//
// The committed symbols are entropy coded with their predicted distributions
// (the statistical-coding pipeline of the paper).  Encoder state: low (W bits
// plus a carry into the bytes already written), range.  Per symbol with
// interval [start, start + f) of a 2^P total: r = range >> P, low += r start,
// range = r f; a carry out of bit W increments the written bytes; while
// range < 2^(W-8) the top byte of low is written and low, range shift left by
// 8.  finish() writes the W/8 bytes of low.  The decoder tracks D = code - low
// and finds the symbol with cdf[s] <= D / r < cdf[s+1].
#pragma once

#include <algorithm>
#include <cstdint>
#include <vector>

namespace dlmc {

class RangeEncoder {
 public:
  RangeEncoder() = default;
  RangeEncoder(int W, int P) { reset(W, P); }
  void reset(int W, int P) {
    W_ = W;
    P_ = P;
    low_ = 0;
    range_ = W == 64 ? ~0ull : ((1ull << W) - 1);
    out_.clear();
  }
  // start + freq <= 2^P, freq >= 1 (checked by the caller)
  void encode(uint32_t start, uint32_t freq) {
    const uint64_t r = range_ >> P_;
    const uint64_t add = r * start;
    bool carry;
    if (W_ == 64) {
      const uint64_t nl = low_ + add;
      carry = nl < low_;
      low_ = nl;
    } else {
      low_ += add;
      carry = (low_ >> 32) != 0;
      low_ &= 0xFFFFFFFFull;
    }
    if (carry) {
      size_t i = out_.size();
      while (i > 0 && out_[i - 1] == 0xFF) out_[--i] = 0;
      if (i > 0) ++out_[i - 1];
    }
    range_ = r * freq;
    const uint64_t lim = 1ull << (W_ - 8);
    while (range_ < lim) {
      out_.push_back((uint8_t)(low_ >> (W_ - 8)));
      low_ = W_ == 64 ? (low_ << 8) : ((low_ << 8) & 0xFFFFFFFFull);
      range_ <<= 8;
    }
  }
  std::vector<uint8_t> finish() {
    for (int i = 0; i < W_ / 8; ++i) out_.push_back((uint8_t)(low_ >> (W_ - 8 - 8 * i)));
    return std::move(out_);
  }

 private:
  int W_ = 32, P_ = 16;
  uint64_t low_ = 0, range_ = 0;
  std::vector<uint8_t> out_;
};

class RangeDecoder {
 public:
  RangeDecoder() = default;
  RangeDecoder(const uint8_t* data, size_t len, int W, int P) { reset(data, len, W, P); }
  void reset(const uint8_t* data, size_t len, int W, int P) {
    data_ = data;
    len_ = len;
    pos_ = 0;
    W_ = W;
    P_ = P;
    range_ = W == 64 ? ~0ull : ((1ull << W) - 1);
    D_ = 0;
    for (int i = 0; i < W / 8; ++i) D_ = (D_ << 8) | next();
  }
  // returns the symbol, or -1 for a corrupt stream
  int decode(const uint32_t* cdf, int V) {
    const uint64_t r = range_ >> P_;
    const uint64_t t = D_ / r;
    if (t >= (1ull << P_)) return -1;
    const int s = (int)(std::upper_bound(cdf, cdf + V + 1, (uint32_t)t) - cdf) - 1;
    if (s < 0 || s >= V || cdf[s + 1] <= cdf[s]) return -1;
    D_ -= r * cdf[s];
    range_ = r * (uint64_t)(cdf[s + 1] - cdf[s]);
    const uint64_t lim = 1ull << (W_ - 8);
    while (range_ < lim) {
      D_ = (D_ << 8) | next();
      range_ <<= 8;
    }
    return s;
  }
  size_t consumed() const { return pos_; }
  uint64_t code_minus_low() const { return D_; }
  uint64_t range() const { return range_; }

 private:
  uint8_t next() { return pos_ < len_ ? data_[pos_++] : (++pos_, 0); }
  const uint8_t* data_ = nullptr;
  size_t len_ = 0, pos_ = 0;
  int W_ = 32, P_ = 16;
  uint64_t range_ = 0, D_ = 0;
};

}  // namespace dlmc
