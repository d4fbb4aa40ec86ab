// Softmax statistics of logit rows for the entropy of the commitment
// schedule (Symbol Commitment Schedules, item 3: H = -sum p log p over the
// predicted distribution), in one fixed partition shared by the LM head's
// epilogue and the standalone statistics kernel, so both give the same bits.
//
// A row of V logits is cut into groups of 128 columns.  The statistics of a
// group are taken by one thread in column order: the group's max m first,
// then Z and A added column by column.  A row's groups are merged by one
// wave: lane l folds groups l, l + 64, ... in order, then the wave merges
// with butterflies over lane distances 1 .. 32.
//
// Statistics of a set of logits relative to its max m: Z = sum e^(l - m),
// A = sum e^(l - m) (l - m); then H (nats) = ln Z - A / Z.  Columns past V
// and -inf logits carry nothing.
#pragma once

#include "common.h"

namespace dlmc {

struct RowStat {
  float m, Z, A;
};

constexpr int STAT_GROUP = 128;  // columns per group

__host__ __device__ constexpr int stat_groups(int V) { return (V + STAT_GROUP - 1) / STAT_GROUP; }

// e^t for t <= 0 on the hardware 2^x (a few ulps of fp32)
__device__ __forceinline__ float stat_exp(float t) {
  return __builtin_amdgcn_exp2f(t * 1.4426950408889634f);
}

__device__ __forceinline__ RowStat stat_merge(RowStat x, RowStat y) {
  if (y.Z == 0.0f) return x;
  if (x.Z == 0.0f) return y;
  const float m = fmaxf(x.m, y.m);
  const float cx = stat_exp(x.m - m), cy = stat_exp(y.m - m);
  RowStat r;
  r.m = m;
  r.Z = cx * x.Z + cy * y.Z;
  r.A = cx * (x.A + (x.m - m) * x.Z) + cy * (y.A + (y.m - m) * y.Z);
  return r;
}

// The statistics of the n <= 128 logits p[0 .. n) of one group (in LDS or
// global memory), in column order.  vec: p is 16-byte aligned, and a full
// group is read as float4s (the same values in the same order).
__device__ __forceinline__ RowStat group_stat(const float* p, int n, bool vec) {
  float m = -INFINITY;
  if (vec && n == STAT_GROUP) {
#pragma unroll 8
    for (int c = 0; c < STAT_GROUP; c += 4) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(p + c);
      m = fmaxf(m, fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w)));
    }
  } else {
    for (int c = 0; c < n; ++c) m = fmaxf(m, p[c]);
  }
  RowStat s{m, 0.0f, 0.0f};
  if (m == -INFINITY) return s;
  auto add = [&](float v) {
    if (v == -INFINITY) return;
    const float t = v - m;
    const float e = stat_exp(t);
    s.Z += e;
    s.A += e * t;
  };
  if (vec && n == STAT_GROUP) {
#pragma unroll 4
    for (int c = 0; c < STAT_GROUP; c += 4) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(p + c);
      add(v.x);
      add(v.y);
      add(v.z);
      add(v.w);
    }
  } else {
    for (int c = 0; c < n; ++c) add(p[c]);
  }
  return s;
}

// merge over lanes at xor distances 1 .. W/2
template <int W>
__device__ __forceinline__ RowStat stat_butterfly(RowStat s) {
#pragma unroll
  for (int o = 1; o < W; o <<= 1) {
    RowStat t{__shfl_xor(s.m, o), __shfl_xor(s.Z, o), __shfl_xor(s.A, o)};
    s = stat_merge(s, t);
  }
  return s;
}

// entropy in bits of a merged row statistic
__device__ __forceinline__ float stat_entropy_bits(RowStat r) {
  return (logf(r.Z) - r.A / r.Z) * 1.4426950408889634f;
}

}  // namespace dlmc
