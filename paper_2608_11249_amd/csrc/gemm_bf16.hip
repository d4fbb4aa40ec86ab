// bf16 MFMA GEMM for gfx950 with fused epilogues: C = A * B^T, fp32 accumulate.
//
// Every dense contraction of the forward pass (QKV, O, FFN in/out, LM head)
// runs here.  Block tile BM x BN x 64 built from v_mfma_f32_32x32x16_bf16
// tiles.  Operand tiles move global -> LDS with direct loads
// (global_load_lds_dwordx4) into a double-buffered LDS tile.  LDS rows are 64
// bf16 (128 B) with the eight 16-byte chunks XOR-swizzled (swz below) so
// fragment loads are free of bank conflicts.  Two kernels:
//  - gemm_bf16_kernel: four waves in a 2 x 2 grid, one barrier per k-tile,
//    the fragment reads of k step s + 1 scheduled between the MFMAs of step s
//    (128 x 128 tiles, two blocks per CU; small and ragged shapes);
//  - gemm_bf16_w4_kernel: four waves, one per SIMD, on a 256 x 256 or
//    256 x 128 tile, A double- and B triple-buffered in LDS (every GEMM of
//    the 8B-shaped pass); gemm_bf16_w4_split_kernel runs both tile shapes
//    in one launch, on two column ranges.
//
// Numerics: each output element is a sequential sum over k-tiles, each k-tile
// four MFMA steps in order, independent of the kernel, the tile shape and of
// which other rows are in the launch, so results are identical for any batch
// composition.
#include "kernels.h"
#include "rowstats.h"

#include <type_traits>
#include <utility>

namespace dlmc {
namespace {

constexpr int BK = 64;

// LDS swizzle of the 16-byte chunks of a 128-byte tile row.  gfx950 serves a
// ds_read_b128 16 lanes at a time from 64 four-byte banks (256 B): rows r and
// r + 2 start on the same bank, so chunk c of row r is stored at position
// c ^ ((r >> 1) & 7) -- the 16 rows a 16-lane group reads then cover the 16
// distinct 16-byte bank slots (8 for even rows, 8 for odd rows).
__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }

// Tile of this block among the tiles with live rows (the first Mv of M).
// Hardware block ids go round robin over the 8 XCDs; the remap gives each XCD
// a contiguous range of the live tiles (launches use a multiple of 8 blocks,
// at least one per tile), and the logical order walks groups of 8 m-tiles (m
// fastest inside a group), so the blocks resident on one XCD at a time cover
// about 8 x 8 tiles and share their operand panels through that XCD's L2.
// Spreading the live tiles, not all M rows' tiles, keeps every XCD busy when
// few rows are live.  Returns false for a block without a tile.
__device__ __forceinline__ bool tile_coords(int bid, int n_tm, int n_tn, int bm, int Mv, int& tm, int& tn) {
  const int tm_live = min(n_tm, (Mv + bm - 1) / bm);
  const int n_live = tm_live * n_tn;
  const int nb = (n_live + 7) & ~7;
  int l = bid;
  if (l >= nb) return false;
  l = (l & 7) * (nb >> 3) + (l >> 3);
  if (l >= n_live) return false;
  constexpr int G = 8;
  const int per_group = G * n_tn;
  const int g = l / per_group, first = g * G;
  const int gsize = min(tm_live - first, G);
  const int r = l - g * per_group;
  tm = first + r % gsize;
  tn = r / gsize;
  return true;
}

// GELU, 0.5 v (1 + erf(v / sqrt 2)), with erfc(x) for x = |v| / sqrt 2 from the
// rational approximation of Abramowitz and Stegun, formula 7.1.26 (absolute
// error at most 1.5e-7), on the hardware 2^x and reciprocal; the result is
// rounded to bf16 right after.
__device__ __forceinline__ float gelu_erf(float v) {
  const float x = fabsf(v) * 0.70710678118654752440f;
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, x, 1.0f));
  const float poly =
      t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 1.061405429f, -1.453152027f), 1.421413741f), -0.284496736f),
               0.254829592f);
  const float erfc_x = poly * __builtin_amdgcn_exp2f(-x * x * 1.4426950408889634f);
  // v >= 0: 0.5 v (2 - erfc); v < 0: 0.5 v erfc
  return v >= 0.0f ? v * (1.0f - 0.5f * erfc_x) : 0.5f * v * erfc_x;
}
// SiLU from the hardware 2^x and reciprocal (v_exp_f32, v_rcp_f32): a few
// ulps of fp32, and the product with the up projection is rounded to bf16
// right after.  Large negative v: 2^x overflows to +inf and the result is -0.
__device__ __forceinline__ float silu(float v) {
  const float e = __builtin_amdgcn_exp2f(-v * 1.4426950408889634f);
  return v * __builtin_amdgcn_rcpf(1.0f + e);
}

// Rotary embedding of the pair (lo, hi) = (q_i, q_{i + d_head/2}) at angle
// (c, s) = (cos, sin): one fused multiply-add each, written out so that every
// kernel rounds it the same way.
__device__ __forceinline__ float rot_lo(float lo, float hi, float c, float s) {
  return fmaf(lo, c, -(hi * s));
}
__device__ __forceinline__ float rot_hi(float lo, float hi, float c, float s) {
  return fmaf(hi, c, lo * s);
}

// Softmax statistics of every 128-column group of the rows of a staged fp32
// tile (rowstats.h): sf holds tile rows [0, R) at pitch PF, the tile's
// first row and column are m0 and n0; one thread per (row, group), the
// group folded in column order from LDS.
template <int R, int BN, int PF, int NT>
__device__ __forceinline__ void tile_group_stats(const float* sf, int m0, int n0, int tid, int Mv,
                                                 int N, const EpiArgs& ea) {
  constexpr int GPR = BN / STAT_GROUP;
  static_assert(BN % STAT_GROUP == 0, "whole groups per tile");
  for (int p = tid; p < R * GPR; p += NT) {
    const int row = p / GPR, gi = p % GPR;
    const int grow = m0 + row, gcol = n0 + gi * STAT_GROUP;
    if (grow >= Mv || gcol >= N) continue;
    const RowStat st = group_stat(sf + row * PF + gi * STAT_GROUP, min(STAT_GROUP, N - gcol), true);
    ((RowStat*)ea.stats)[(size_t)grow * ea.stat_ld + gcol / STAT_GROUP] = st;
  }
}

// acc[i][j][r] holds C[row][col] with row = i*32 + (r/4)*8 + lg*4 + r%4 and
// col = j*32 + lr inside the wave tile of wave (wm, wn).
template <int BM, int BN, int EPI, int WM, int WN>
__device__ __forceinline__ void epilogue_w(f32x16 (&acc)[WM / 32][WN / 32], int m0, int n0, int wm,
                                           int wn, int lane, int Mv, int N, const EpiArgs& ea) {
  constexpr int TM = WM / 32, TN = WN / 32;
  static_assert(EPI != EPI_STORE_F32, "fp32 stores go through a staged epilogue (row statistics)");
  const int lr = lane & 31, lg = lane >> 5;
  const int wrow0 = m0 + wm * WM, wcol0 = n0 + wn * WN;
  if constexpr (EPI == EPI_QKV_ROPE) {
    const int d = ea.d, dh = ea.dh, T = ea.T, Tp = ea.Tp, H = ea.H, half = dh / 2;
#pragma unroll
    for (int j = 0; j < TN; j += 2) {
      const int col0 = wcol0 + j * 32;  // multiple of 64: a (lo, hi) pair of 32-col blocks
      const int which = col0 / d, within = col0 % d;
      const int h = within / dh, jb = (within % dh) / 32;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wrow0 + i * 32 + (r >> 2) * 8 + lg * 4 + (r & 3);
          if (row >= Mv) continue;
          const int b = row / T, t = row - b * T;
          const size_t bh = (size_t)b * H + h;
          const float lo = acc[i][j][r], hi = acc[i][j + 1][r];
          if (which < 2) {
            const int dlo = (jb >> 1) * 32 + lr;
            const float c = ea.rope_cos[t * half + dlo], s = ea.rope_sin[t * half + dlo];
            bf16_t* dst = (bf16_t*)(which == 0 ? ea.q : ea.k) + (bh * Tp + t) * dh;
            dst[dlo] = f32_to_bf16(rot_lo(lo, hi, c, s));
            dst[dlo + half] = f32_to_bf16(rot_hi(lo, hi, c, s));
          } else {
            bf16_t* dst = (bf16_t*)ea.vt + bh * dh * Tp + t;
            const int dim = jb * 32 + lr;
            dst[(size_t)dim * Tp] = f32_to_bf16(lo);
            dst[(size_t)(dim + 32) * Tp] = f32_to_bf16(hi);
          }
        }
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
    for (int j = 0; j < TN; j += 2) {
      const int f = (wcol0 + j * 32) / 2 + lr;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wrow0 + i * 32 + (r >> 2) * 8 + lg * 4 + (r & 3);
          if (row >= Mv) continue;
          const float g = acc[i][j][r], u = acc[i][j + 1][r];
          ((bf16_t*)ea.out)[(size_t)row * ea.ldo + f] = f32_to_bf16(silu(g) * u);
        }
    }
  } else {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = wcol0 + j * 32 + lr;
        if (col >= N) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wrow0 + i * 32 + (r >> 2) * 8 + lg * 4 + (r & 3);
          if (row >= Mv) continue;
          const size_t o = (size_t)row * ea.ldo + col;
          if constexpr (EPI == EPI_STORE_F32) {
            ((float*)ea.out)[o] = acc[i][j][r];
          } else if constexpr (EPI == EPI_RESIDUAL) {
            ((float*)ea.out)[o] += acc[i][j][r];
          } else {
            ((bf16_t*)ea.out)[o] = f32_to_bf16(gelu_erf(acc[i][j][r]));
          }
        }
      }
  }
}

template <int BM, int BN, int EPI>
__device__ __forceinline__ void epilogue(f32x16 (&acc)[BM / 64][BN / 64], int m0, int n0, int wm,
                                         int wn, int lane, int Mv, int N, const EpiArgs& ea) {
  epilogue_w<BM, BN, EPI, BM / 2, BN / 2>(acc, m0, n0, wm, wn, lane, Mv, N, ea);
}

// ---------------------------------------------------------------------------
// LDS-staged epilogue.  After the main loop the LDS tile is free: phase 1 has
// every wave apply its epilogue arithmetic in registers (the same operations,
// in the same order, as epilogue_w) and park the results in an LDS tile;
// phase 2 has all threads move 16-byte chunks from LDS to global memory, so
// stores are coalesced -- including V, which the QKV epilogue writes
// transposed ([dh, Tp] per head).  Rows of an LDS tile carry 8 elements of
// padding, which puts the two row groups a wave writes at once on different
// banks.
// MAIN: LDS bytes of the main loop; BPC: blocks per CU the registers allow
// (0: as many as the main loop's LDS allows).
template <int BM, int BN, int EPI, int MAIN = 2 * (BM + BN) * BK * 2, int BPC = 0>
struct StagedEpi {
  static constexpr int PF = BN + 8;       // fp32 tile pitch (STORE, RESIDUAL)
  static constexpr int PB = BN + 8;       // bf16 tile pitch (GELU, Q/K)
  static constexpr int PS = BN / 2 + 8;   // bf16 tile pitch (SwiGLU output)
  static constexpr int PV = BM + 8;       // bf16 dim-major pitch (V)
  static constexpr int bytes =
      (EPI == EPI_STORE_F32 || EPI == EPI_RESIDUAL) ? BM * PF * 4
      : EPI == EPI_GELU                              ? BM * PB * 2
      : EPI == EPI_SWIGLU                            ? BM * PS * 2
      : (BM * PB > BN * PV ? BM * PB : BN * PV) * 2;
  static constexpr int main_bytes = MAIN;
  // staged only where it keeps the blocks-per-CU count of the main loop
  static constexpr int lds_cu = 160 * 1024;
  static constexpr int bpc = BPC > 0 && BPC < lds_cu / main_bytes ? BPC : lds_cu / main_bytes;
  static constexpr bool enabled = bytes <= lds_cu && lds_cu / (bytes > main_bytes ? bytes : main_bytes) >= bpc;
  static constexpr int smem_elems = (enabled && bytes > main_bytes ? bytes : main_bytes) / 2;
};

template <int BM, int BN, int EPI, int WM, int WN, int NT>
__device__ __forceinline__ void epilogue_staged(f32x16 (&acc)[WM / 32][WN / 32], bf16_t* smem,
                                                int m0, int n0, int wm, int wn, int tid, int Mv,
                                                int N, const EpiArgs& ea) {
  using SE = StagedEpi<BM, BN, EPI>;  // pitches only: they do not depend on MAIN / BPC
  constexpr int TM = WM / 32, TN = WN / 32;
  const int lane = tid & 63, lr = lane & 31, lg = lane >> 5;
  const int wr0 = wm * WM, wc0 = wn * WN;  // wave tile origin inside the block tile
  float* sf = reinterpret_cast<float*>(smem);
  // RESIDUAL: the residual rows this thread updates in phase 2 are loaded
  // first, so their latency hides under phase 1
  constexpr int CPR4 = BN / 4, IT4 = BM * CPR4 / NT;  // float4 chunks per row / per thread
  static_assert(BM * CPR4 % NT == 0, "fp32 chunks must split evenly over the threads");
  const bool vec4 = (ea.ldo & 3) == 0;
  float4 xres[EPI == EPI_RESIDUAL ? IT4 : 1];
  if constexpr (EPI == EPI_RESIDUAL) {
#pragma unroll
    for (int it = 0; it < IT4; ++it) {
      const int qi = tid + it * NT, row = qi / CPR4, c = (qi % CPR4) * 4;
      const int grow = m0 + row, gcol = n0 + c;
      if (grow < Mv && gcol + 4 <= N && vec4)
        xres[it] = *reinterpret_cast<const float4*>((const float*)ea.out + (size_t)grow * ea.ldo + gcol);
    }
  }
  // the main loop's last barrier ends every read of the operand tiles
  if constexpr (EPI == EPI_STORE_F32 || EPI == EPI_RESIDUAL || EPI == EPI_GELU) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wr0 + i * 32 + (r >> 2) * 8 + lg * 4 + (r & 3), col = wc0 + j * 32 + lr;
          if constexpr (EPI == EPI_GELU)
            smem[row * SE::PB + col] = f32_to_bf16(gelu_erf(acc[i][j][r]));
          else
            sf[row * SE::PF + col] = acc[i][j][r];
        }
  } else if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
    for (int j = 0; j < TN; j += 2)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wr0 + i * 32 + (r >> 2) * 8 + lg * 4 + (r & 3);
          const int f = (wc0 + j * 32) / 2 + lr;
          smem[row * SE::PS + f] = f32_to_bf16(silu(acc[i][j][r]) * acc[i][j + 1][r]);
        }
  } else {  // EPI_QKV_ROPE: the block tile lies inside one of Q, K, V (d % BN == 0)
    const int d = ea.d, dh = ea.dh, T = ea.T, half = dh / 2;
    const int which = n0 / d;
    if (which < 2) {
      constexpr int NP = TN / 2;  // (lo, hi) pairs of 32-column blocks per wave tile row
      int hb[NP], dlo[NP];        // local column of the head's first dim; dim of lo
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        const int lc0 = wc0 + 2 * p * 32;
        const int in_head = (n0 + lc0) % d % dh;
        hb[p] = lc0 - in_head;
        dlo[p] = ((in_head / 32) >> 1) * 32 + lr;
      }
      // the cos / sin gathers of a 32-row block are all issued before the
      // first is used: issued one at a time, each would wait out an L2 round
      // trip, and those waits made this epilogue cost more than half as much
      // as the tile's main loop
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        float cv[NP][16], sv[NP][16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wr0 + i * 32 + (r >> 2) * 8 + lg * 4 + (r & 3);
          const int t = min(m0 + row, Mv - 1) % T;
#pragma unroll
          for (int p = 0; p < NP; ++p) {
            cv[p][r] = ea.rope_cos[t * half + dlo[p]];
            sv[p][r] = ea.rope_sin[t * half + dlo[p]];
          }
        }
#pragma unroll
        for (int p = 0; p < NP; ++p)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = wr0 + i * 32 + (r >> 2) * 8 + lg * 4 + (r & 3);
            const float lo = acc[i][2 * p][r], hi = acc[i][2 * p + 1][r];
            const float c = cv[p][r], s = sv[p][r];
            smem[row * SE::PB + hb[p] + dlo[p]] = f32_to_bf16(rot_lo(lo, hi, c, s));
            smem[row * SE::PB + hb[p] + dlo[p] + half] = f32_to_bf16(rot_hi(lo, hi, c, s));
          }
      }
    } else {
      // V, dim-major: 4 consecutive rows of one column are one 8-byte write
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int row = wr0 + i * 32 + q * 8 + lg * 4, col = wc0 + j * 32 + lr;
            u32x2 v;
            v[0] = (uint32_t)f32_to_bf16(acc[i][j][4 * q]) | ((uint32_t)f32_to_bf16(acc[i][j][4 * q + 1]) << 16);
            v[1] = (uint32_t)f32_to_bf16(acc[i][j][4 * q + 2]) | ((uint32_t)f32_to_bf16(acc[i][j][4 * q + 3]) << 16);
            *reinterpret_cast<u32x2*>(smem + col * SE::PV + row) = v;
          }
    }
  }
  __syncthreads();
  // phase 2: 16-byte chunks, a fixed number per thread (EPI_STORE_F32 with
  // no output: the row statistics only)
  if constexpr (EPI == EPI_STORE_F32 || EPI == EPI_RESIDUAL) {
#pragma unroll
    for (int it = 0; it < IT4; ++it) {
      if (EPI == EPI_STORE_F32 && !ea.out) break;
      const int qi = tid + it * NT, row = qi / CPR4, c = (qi % CPR4) * 4;
      const int grow = m0 + row, gcol = n0 + c;
      if (grow >= Mv) continue;
      float* dst = (float*)ea.out + (size_t)grow * ea.ldo + gcol;
      const float* src = sf + row * SE::PF + c;
      if (gcol + 4 <= N && vec4) {
        float4 v = *reinterpret_cast<const float4*>(src);
        if constexpr (EPI == EPI_RESIDUAL) {
          const float4 o = xres[it];
          v.x = o.x + v.x; v.y = o.y + v.y; v.z = o.z + v.z; v.w = o.w + v.w;
        }
        *reinterpret_cast<float4*>(dst) = v;
      } else {
        for (int e = 0; e < 4 && gcol + e < N; ++e) {
          if constexpr (EPI == EPI_RESIDUAL) dst[e] += src[e];
          else dst[e] = src[e];
        }
      }
    }
    // the tile is still in LDS: the entropy's group statistics of its rows
    if constexpr (EPI == EPI_STORE_F32)
      if (ea.stats) tile_group_stats<BM, BN, SE::PF, NT>(sf, m0, n0, tid, Mv, N, ea);
  } else if constexpr (EPI == EPI_GELU || EPI == EPI_SWIGLU) {
    constexpr int W = EPI == EPI_GELU ? BN : BN / 2;
    constexpr int P = EPI == EPI_GELU ? SE::PB : SE::PS;
    constexpr int CPR = W / 8;
    const int gc0 = EPI == EPI_GELU ? n0 : n0 / 2;
    const int Nout = EPI == EPI_GELU ? N : N / 2;
    static_assert(BM * CPR % NT == 0, "bf16 chunks must split evenly over the threads");
#pragma unroll
    for (int it = 0; it < BM * CPR / NT; ++it) {
      const int qi = tid + it * NT, row = qi / CPR, c = (qi % CPR) * 8;
      const int grow = m0 + row, gcol = gc0 + c;
      if (grow >= Mv) continue;
      bf16_t* dst = (bf16_t*)ea.out + (size_t)grow * ea.ldo + gcol;
      const bf16_t* src = smem + row * P + c;
      if (gcol + 8 <= Nout && (ea.ldo & 7) == 0) {
        *reinterpret_cast<u32x4*>(dst) = *reinterpret_cast<const u32x4*>(src);
      } else {
        for (int e = 0; e < 8 && gcol + e < Nout; ++e) dst[e] = src[e];
      }
    }
  } else {
    const int d = ea.d, dh = ea.dh, T = ea.T, Tp = ea.Tp, H = ea.H;
    const int which = n0 / d, nb = n0 - which * d;  // first column inside Q, K or V
    if (which < 2) {
      constexpr int CPR = BN / 8;
      bf16_t* base = (bf16_t*)(which == 0 ? ea.q : ea.k);
      static_assert(BM * CPR % NT == 0, "bf16 chunks must split evenly over the threads");
#pragma unroll
      for (int it = 0; it < BM * CPR / NT; ++it) {
        const int qi = tid + it * NT, row = qi / CPR, c = (qi % CPR) * 8;
        const int grow = m0 + row;
        if (grow >= Mv) continue;
        const int b = grow / T, t = grow - b * T;
        const int h = (nb + c) / dh, dim = (nb + c) % dh;
        bf16_t* dst = base + (((size_t)b * H + h) * Tp + t) * dh + dim;
        *reinterpret_cast<u32x4*>(dst) = *reinterpret_cast<const u32x4*>(smem + row * SE::PB + c);
      }
    } else {
      constexpr int CPC = BM / 8;  // chunks of 8 rows per column
      bf16_t* base = (bf16_t*)ea.vt;
      static_assert(BN * CPC % NT == 0, "bf16 chunks must split evenly over the threads");
#pragma unroll
      for (int it = 0; it < BN * CPC / NT; ++it) {
        const int qi = tid + it * NT, col = qi / CPC, r0 = (qi % CPC) * 8;
        const int grow = m0 + r0;
        if (grow >= Mv) continue;
        const int h = (nb + col) / dh, dim = (nb + col) % dh;
        const int b = grow / T, t = grow - b * T;
        const bf16_t* src = smem + col * SE::PV + r0;
        if (t % 8 == 0 && t + 8 <= T && grow + 8 <= Mv) {
          bf16_t* dst = base + (((size_t)b * H + h) * dh + dim) * Tp + t;
          *reinterpret_cast<u32x4*>(dst) = *reinterpret_cast<const u32x4*>(src);
        } else {
          for (int e = 0; e < 8 && grow + e < Mv; ++e) {
            const int ge = grow + e, be = ge / T, te = ge - be * T;
            base[(((size_t)be * H + h) * dh + dim) * Tp + te] = src[e];
          }
        }
      }
    }
  }
}

// fp32 store or residual update of a tile whose staging buffer would not fit
// in LDS (256 x 256): the same two phases as epilogue_staged, once per
// 128-row half -- the waves holding the half park it in LDS, then all threads
// store it (or add it to the residual rows) as float4s.
template <int EPI, int BM, int BN, int WM, int WN, int NT>
__device__ __forceinline__ void epilogue_store_halves(f32x16 (&acc)[WM / 32][WN / 32], bf16_t* smem,
                                                      int m0, int n0, int wm, int wn, int tid,
                                                      int Mv, int N, const EpiArgs& ea) {
  static_assert(BM == 2 * WM, "two wave rows");
  static_assert(EPI == EPI_STORE_F32 || EPI == EPI_RESIDUAL, "fp32 epilogues");
  constexpr int TM = WM / 32, TN = WN / 32, PF = BN + 8;
  constexpr int CPR4 = BN / 4, IT4 = WM * CPR4 / NT;
  static_assert(WM * CPR4 % NT == 0, "fp32 chunks must split evenly over the threads");
  const int lane = tid & 63, lr = lane & 31, lg = lane >> 5;
  float* sf = reinterpret_cast<float*>(smem);
  const bool vec4 = (ea.ldo & 3) == 0;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (wm == h) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            sf[(i * 32 + (r >> 2) * 8 + lg * 4 + (r & 3)) * PF + wn * WN + j * 32 + lr] = acc[i][j][r];
    }
    __syncthreads();
#pragma unroll
    for (int it = 0; it < IT4; ++it) {
      if (EPI == EPI_STORE_F32 && !ea.out) break;  // row statistics only
      const int qi = tid + it * NT, row = qi / CPR4, c = (qi % CPR4) * 4;
      const int grow = m0 + h * WM + row, gcol = n0 + c;
      if (grow >= Mv) continue;
      float* dst = (float*)ea.out + (size_t)grow * ea.ldo + gcol;
      const float* src = sf + row * PF + c;
      if (gcol + 4 <= N && vec4) {
        float4 v = *reinterpret_cast<const float4*>(src);
        if constexpr (EPI == EPI_RESIDUAL) {
          const float4 o = *reinterpret_cast<const float4*>(dst);
          v.x = o.x + v.x; v.y = o.y + v.y; v.z = o.z + v.z; v.w = o.w + v.w;
        }
        *reinterpret_cast<float4*>(dst) = v;
      } else {
        for (int e = 0; e < 4 && gcol + e < N; ++e) {
          if constexpr (EPI == EPI_RESIDUAL) dst[e] += src[e];
          else dst[e] = src[e];
        }
      }
    }
    // the half is still in LDS: the entropy's group statistics of its rows
    if constexpr (EPI == EPI_STORE_F32)
      if (ea.stats) tile_group_stats<WM, BN, PF, NT>(sf, m0 + h * WM, n0, tid, Mv, N, ea);
    __syncthreads();
  }
}

// 16-byte direct global -> LDS load (global_load_lds_dwordx4).  `lds` must be
// wave-uniform: lane l writes lds + 16 l bytes.  The builtin exists only for
// the device target, so the host pass sees an empty body.
__device__ __forceinline__ void lds_dma16(const bf16_t* g, bf16_t* lds) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0);
#endif
}

// MFMA fragment loads of one 16-deep k step: rows w0 + 32 i + lr, 16-byte
// chunk kc of each 128-byte LDS row (XOR-swizzled by row & 7).
template <int NT>
__device__ __forceinline__ void load_frags(bf16x8 (&f)[NT], const bf16_t* base, int w0, int lr,
                                           int kc) {
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    const int row = w0 + i * 32 + lr;
    f[i] = *reinterpret_cast<const bf16x8*>(base + row * BK + ((kc ^ swz(row)) << 3));
  }
}

template <int TM, int TN>
__device__ __forceinline__ void mfma_block(f32x16 (&acc)[TM][TN], const bf16x8 (&a)[TM],
                                           const bf16x8 (&b)[TN]) {
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
}

// Each wave load instruction fills one contiguous 1 KB LDS window (8 tile
// rows); the XOR swizzle is applied on the global side, lane l of the window
// fetching chunk (l & 7) ^ swz(row) of its row.  No VGPR staging, no
// ds_write.  MFMA fragments are double buffered in registers across the four
// k steps.
template <int BM, int BN, int EPI>
__global__ void __launch_bounds__(256)
gemm_bf16_kernel(const bf16_t* __restrict__ A, const bf16_t* __restrict__ Bw, int M, int N,
                 int K, const int* __restrict__ M_dev, EpiArgs ea, int n_tm, int n_tn) {
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int A_IN = BM / 32;  // 1 KB load instructions per wave per k-tile
  constexpr int B_IN = BN / 32;
  __shared__ __attribute__((aligned(16))) bf16_t smem[StagedEpi<BM, BN, EPI>::smem_elems];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 31, lg = lane >> 5;
  const int Mv = M_dev ? min(*M_dev, M) : M;
  int tm, tn;
  if (!tile_coords(blockIdx.x, n_tm, n_tn, BM, Mv, tm, tn)) return;
  const int m0 = tm * BM, n0 = tn * BN;

  bf16_t* As = smem;
  bf16_t* Bs = smem + 2 * BM * BK;
  int a_off[A_IN], b_off[B_IN];
#pragma unroll
  for (int j = 0; j < A_IN; ++j) {
    const int sl = (wave * A_IN + j) * 64 + lane, row = sl >> 3;
    a_off[j] = min(m0 + row, Mv - 1) * K + (((sl & 7) ^ swz(row)) << 3);
  }
#pragma unroll
  for (int j = 0; j < B_IN; ++j) {
    const int sl = (wave * B_IN + j) * 64 + lane, row = sl >> 3;
    b_off[j] = min(n0 + row, N - 1) * K + (((sl & 7) ^ swz(row)) << 3);
  }
  const int a_win = wave * A_IN * 512, b_win = wave * B_IN * 512;  // this wave's LDS windows

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = K / BK;
#pragma unroll
  for (int j = 0; j < A_IN; ++j)
    lds_dma16(A + a_off[j], As + a_win + j * 512);
#pragma unroll
  for (int j = 0; j < B_IN; ++j)
    lds_dma16(Bw + b_off[j], Bs + b_win + j * 512);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      const int k1 = (kt + 1) * BK;
      bf16_t* an = As + (cur ^ 1) * BM * BK + a_win;
      bf16_t* bn = Bs + (cur ^ 1) * BN * BK + b_win;
#pragma unroll
      for (int j = 0; j < A_IN; ++j)
        lds_dma16(A + a_off[j] + k1, an + j * 512);
#pragma unroll
      for (int j = 0; j < B_IN; ++j)
        lds_dma16(Bw + b_off[j] + k1, bn + j * 512);
    }
    const bf16_t* as = As + cur * BM * BK;
    const bf16_t* bs = Bs + cur * BN * BK;
    bf16x8 a0[TM], b0[TN], a1[TM], b1[TN];
    load_frags<TM>(a0, as, wm * WM, lr, lg);
    load_frags<TN>(b0, bs, wn * WN, lr, lg);
    load_frags<TM>(a1, as, wm * WM, lr, 2 + lg);
    load_frags<TN>(b1, bs, wn * WN, lr, 2 + lg);
    mfma_block<TM, TN>(acc, a0, b0);
    load_frags<TM>(a0, as, wm * WM, lr, 4 + lg);
    load_frags<TN>(b0, bs, wn * WN, lr, 4 + lg);
    mfma_block<TM, TN>(acc, a1, b1);
    load_frags<TM>(a1, as, wm * WM, lr, 6 + lg);
    load_frags<TN>(b1, bs, wn * WN, lr, 6 + lg);
    mfma_block<TM, TN>(acc, a0, b0);
    mfma_block<TM, TN>(acc, a1, b1);
    {
      // software pipeline: the DS reads of k step s+1 and the direct loads of
      // the next k-tile are spread between the MFMAs of k step s
      constexpr int NF = TM + TN, NM = TM * TN, NV = A_IN + B_IN;
      __builtin_amdgcn_sched_group_barrier(0x100, NF, 0);
#pragma unroll
      for (int i = 0; i < NF; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        if (i < NV) __builtin_amdgcn_sched_group_barrier(0x020, NV / NF > 0 ? NV / NF : 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, NM / NF, 0);
      }
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int i = 0; i < NF; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, NM / NF, 0);
        }
      __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }
  if constexpr (StagedEpi<BM, BN, EPI>::enabled)
    epilogue_staged<BM, BN, EPI, BM / 2, BN / 2, 256>(acc, smem, m0, n0, wm, wn, tid, Mv, N, ea);
  else if constexpr ((EPI == EPI_STORE_F32 || EPI == EPI_RESIDUAL) &&
                     BM / 2 * (BN + 8) * 4 <= StagedEpi<BM, BN, EPI>::smem_elems * 2)
    // an fp32 tile too large for the main loop's LDS, staged in two row halves
    epilogue_store_halves<EPI, BM, BN, BM / 2, BN / 2, 256>(acc, smem, m0, n0, wm, wn, tid, Mv, N, ea);
  else
    epilogue<BM, BN, EPI>(acc, m0, n0, wm, wn, lane, Mv, N, ea);
}

// ---------------------------------------------------------------------------
// 4-wave 256 x BN kernel (BN = 256 or 128): one wave per SIMD, each wave a
// 128 x BN/2 sub-tile (up to 16 accumulator tiles, 256 AGPRs), so a k step
// reads 8 fragments for 16 MFMAs at BN = 256.  The 256-row tile moves fewer
// operand bytes through LDS per flop than 128 x 128 tiles (the direct loads
// into LDS, not the MFMAs, are what limits those), and one block per CU
// covers the narrower GEMMs in whole waves of tiles.
//
// LDS stages: A (activation) tile k sits in stage k % NSA, B (weight) tile k
// in stage k % NSB (NSA = 2, NSB = 3 at BN = 256; 3 and 4 at BN = 128; 160 KB
// either way).  One barrier per k-tile, between k steps 2 and 3: before it
// each wave has waited for its own direct loads of tile k + 1 and for its
// fragment reads of tile k; after it, tile k's stages are free.  The loads
// into those stages -- A tile k + NSA, B tile k + NSB, together "window k",
// the operand with fewer stages first -- are spread over the next four k
// steps (step 3 of k-tile k, steps 0-2 of k-tile k + 1), so a tile is issued
// NS - 1 k-tiles, less a step or two, before it is read.  Loads arrive from
// L2 or HBM at a latency of about a k-tile, and more stages hide more of it.
//
// Each k step runs as four chunks in a fixed order, split by scheduling
// barriers: the direct loads due (NL / 16 of a window's NL loads), the next
// step's fragment reads (the first two chunks), BN / 64 MFMAs.  Spread evenly,
// the direct loads do not back up the load path and hold up the MFMAs behind
// them, as they do when issued in bursts.
//
// The last max(NSA, NSB) k-tiles are peeled: loads past the last k-tile are
// dropped at compile time, so the main loop has no branches.
//
// Numerics: each accumulator takes the k steps of each k-tile in order, as in
// gemm_bf16_kernel, so the results are identical to the other kernel's.
__device__ __forceinline__ void block_barrier() {
  // s_barrier without the memory fence of __syncthreads(), which would also
  // wait for the direct loads still in flight
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// s_waitcnt immediate: vmcnt(n) with lgkmcnt(0)
constexpr int waitcnt_vm(int n) { return 0x0070 | (n & 15) | ((n >> 4) << 14); }

template <int B0, typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, B0 + I>{}), ...);
}
// f(integral_constant<B0>) ... f(integral_constant<B1 - 1>)
template <int B0, int B1, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl<B0>(f, std::make_integer_sequence<int, (B1 > B0 ? B1 - B0 : 0)>{});
}

// Loads of a window: I < N1 are those of the operand with fewer stages.
// Stage count of load I, and the number of prologue loads (windows -NSM ..
// -2, tiles >= 0) issued after the last load of tile 0.
template <int NSA, int NSB, int N1>
constexpr int w4_ns_of(int i) {
  return ((i < N1) == (NSA <= NSB)) ? NSA : NSB;
}
template <int NSA, int NSB, int N1, int NL>
constexpr int w4_prologue_after_tile0() {
  constexpr int NSM = NSA > NSB ? NSA : NSB;
  int after = 0;
  for (int w = -NSM; w <= -2; ++w)
    for (int i = 0; i < NL; ++i) {
      const int tile = w + w4_ns_of<NSA, NSB, N1>(i);
      if (tile >= 0) after = tile == 0 ? 0 : after + 1;
    }
  return after;
}

// LDS elements (bf16) of one 4-wave block: the operand stages, or the staged
// epilogue's tile where that is larger
template <int EPI, int BN, int NSA, int NSB>
constexpr int w4_smem_elems() {
  return StagedEpi<256, BN, EPI, (NSA * 256 + NSB * BN) * BK * 2, 1>::smem_elems;
}

// One block of the 4-wave kernel: tile number `bid` of a launch over n_tm x
// n_tn tiles whose columns start at tile tn_off, with `smem` the block's LDS.
template <int EPI, int BN, int NSA, int NSB>
__device__ __forceinline__ void w4_tile(const bf16_t* __restrict__ A, const bf16_t* __restrict__ Bw,
                                        int M, int N, int K, const int* __restrict__ M_dev,
                                        const EpiArgs& ea, int n_tm, int n_tn, int tn_off, int bid,
                                        bf16_t* smem) {
  static_assert(BN == 256 || BN == 128, "256 x 256 or 256 x 128 tiles");
  constexpr int BM = 256, WM = 128, WN = BN / 2, TM = WM / 32, TN = WN / 32;
  constexpr int A_IN = BM / 32, B_IN = BN / 32;  // 1 KB direct loads per wave per k-tile
  using SE = StagedEpi<BM, BN, EPI, (NSA * BM + NSB * BN) * BK * 2, 1>;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, kept scalar
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 31, lg = lane >> 5;
  const int Mv = M_dev ? min(*M_dev, M) : M;
  int tm, tn;
  if (!tile_coords(bid, n_tm, n_tn, BM, Mv, tm, tn)) return;
  const int m0 = tm * BM, n0 = (tn + tn_off) * BN;  // the launch covers column tiles tn_off ..
  const int nk = K / BK;

  bf16_t* As = smem;
  bf16_t* Bs = smem + NSA * BM * BK;
  // direct loads: window j of wave w fills A tile rows 64 w + 8 j .. + 7 (1 KB)
  // or B tile rows (BN / 4) w + 8 j .. + 7; lane l fills row 8 j + l / 8 of the
  // wave's range, 16-byte slot l % 8, with chunk (l % 8) ^ swz(row) of that
  // row.  The swizzle depends only on j % 2.  A rows past the live rows (Mv)
  // are clamped; N % BN == 0 keeps B tiles whole.
  const int lrow = 64 * wave + (lane >> 3);
  const int brow = (BN / 4) * wave + (lane >> 3);
  int boff[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) boff[e] = brow * K + (((lane & 7) ^ swz(brow + 8 * e)) << 3);
  const size_t stride8 = (size_t)8 * K;
  const bf16_t* b_src = Bw + (size_t)n0 * K;
  const int a_win = wave * A_IN * 512, b_win = wave * B_IN * 512;
  auto dma_a = [&](int kt, int j) {
    const int chunk = ((lane & 7) ^ swz(lrow + 8 * (j & 1))) << 3;
    lds_dma16(A + (min(m0 + lrow + 8 * j, Mv - 1) * K + kt * BK + chunk),
              As + (kt % NSA) * BM * BK + a_win + j * 512);
  };
  auto dma_b = [&](int kt, int j) {
    lds_dma16(b_src + kt * BK + j * stride8 + boff[j & 1], Bs + (kt % NSB) * BN * BK + b_win + j * 512);
  };
  auto frag = [&](bf16x8& f, const bf16_t* base, int row, int kc) {
    f = *reinterpret_cast<const bf16x8*>(base + row * BK + ((kc ^ swz(row)) << 3));
  };
  // load I of window w: A tile w + NSA, B tile w + NSB, fewer stages first
  constexpr bool A_FIRST = NSA <= NSB;
  constexpr int NL = A_IN + B_IN, N1 = A_FIRST ? A_IN : B_IN;
  constexpr int NSM = NSA > NSB ? NSA : NSB, NSMIN = NSA < NSB ? NSA : NSB;
  auto load = [&](int w, auto i_) {
    constexpr int I = decltype(i_)::value;
    constexpr bool IS_A = (I < N1) == A_FIRST;
    constexpr int J = I < N1 ? I : I - N1;
    if constexpr (IS_A)
      dma_a(w + NSA, J);
    else
      dma_b(w + NSB, J);
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // Wait counts.  At the end of k-tile t the windows up to t - 1 have been
  // issued; YOUNGER of their loads follow the last load of tile t + 1.
  constexpr int YOUNGER = (NSA == NSB ? 0 : (A_FIRST ? B_IN : A_IN)) + (NSMIN - 2) * NL;
  // prologue: windows -NSM .. -2, tiles >= 0; PROL loads follow the last
  // load of tile 0
  constexpr int PROL = w4_prologue_after_tile0<NSA, NSB, N1, NL>();
  static_assert(YOUNGER < 64 && PROL < 64, "vmcnt field");
  static_for<-NSM, -1>([&](auto w_) {
    constexpr int W = decltype(w_)::value;
    static_for<0, NL>([&](auto i_) {
      constexpr int TILE = W + w4_ns_of<NSA, NSB, N1>(decltype(i_)::value);
      if constexpr (TILE >= 0)
        if (TILE < nk) load(W, i_);
    });
  });
  if (nk >= NSM - 1)
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(PROL));
  else
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  block_barrier();
  // the first quarter of window -1 (what step 3 of k-tile -1 would issue)
  static_for<0, NL / 4>([&](auto i_) {
    if (w4_ns_of<NSA, NSB, N1>(decltype(i_)::value) - 1 < nk) load(-1, i_);
  });
  bf16x8 fa[2][TM], fb[2][TN];
  load_frags<TM>(fa[0], As, wm * WM, lr, lg);
  load_frags<TN>(fb[0], Bs, wn * WN, lr, lg);

  // One k-tile.  Steps 0-2 issue the last three quarters of window kt - 1,
  // step 3 (after the barrier) the first quarter of window kt.  R < 0: a
  // main-loop k-tile, every load exists; R >= 0: k-tile nk - NSM + R, loads
  // of tiles >= nk dropped.
  auto trip = [&](int kt, auto r_) {
    constexpr int R = decltype(r_)::value;
    // k step S: MFMAs on fragment set S % 2 while the other set is read from
    // (an, bn) at 16-byte chunk kc
    auto step = [&](auto s_, const bf16_t* an, const bf16_t* bn, int kc) {
      constexpr int S = decltype(s_)::value, c = S & 1;
      constexpr int W_OFF = S == 3 ? 0 : -1;  // window kt + W_OFF
      auto chunk = [&](auto q_) {
        constexpr int Q = decltype(q_)::value;
        constexpr int SLOT = ((S + 1) & 3) * 4 + Q;  // slots 0-3: step 3; 4-15: steps 0-2
        static_for<SLOT * NL / 16, (SLOT + 1) * NL / 16>([&](auto i_) {
          // tile - nk of this load in k-tile nk - NSM + R
          constexpr int PAST = W_OFF + w4_ns_of<NSA, NSB, N1>(decltype(i_)::value) - NSM + R;
          if constexpr (R < 0 || PAST < 0) load(kt + W_OFF, i_);
        });
        // the next step's first MFMAs need A fragment 0 and every B fragment
        if constexpr (Q == 0) {
#pragma unroll
          for (int e = 0; e < TN; ++e) frag(fb[c ^ 1][e], bn, wn * WN + e * 32 + lr, kc);
          frag(fa[c ^ 1][0], an, wm * WM + lr, kc);
        } else if constexpr (Q == 1) {
#pragma unroll
          for (int e = 1; e < TM; ++e) frag(fa[c ^ 1][e], an, wm * WM + e * 32 + lr, kc);
        }
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[Q][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[c][Q], fb[c][j], acc[Q][j], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      };
      static_assert(TM == 4, "four chunks per k step");
      static_for<0, 4>(chunk);
    };
    const bf16_t* as = As + (kt % NSA) * BM * BK;
    const bf16_t* bs = Bs + (kt % NSB) * BN * BK;
    step(std::integral_constant<int, 0>{}, as, bs, 2 + lg);
    step(std::integral_constant<int, 1>{}, as, bs, 4 + lg);
    step(std::integral_constant<int, 2>{}, as, bs, 6 + lg);
    // tile kt + 1 has landed and this wave's reads of tile kt are done; once
    // loads have been dropped, fewer than YOUNGER follow it: wait for all
    if constexpr (R <= 0)
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(YOUNGER));
    else
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    block_barrier();
    step(std::integral_constant<int, 3>{}, As + ((kt + 1) % NSA) * BM * BK,
         Bs + ((kt + 1) % NSB) * BN * BK, lg);
  };
  for (int kt = 0; kt < nk - NSM; ++kt) trip(kt, std::integral_constant<int, -1>{});
  static_for<0, NSM>([&](auto r_) {
    constexpr int R = decltype(r_)::value;
    if (nk - NSM + R >= 0) trip(nk - NSM + R, r_);  // its fragment reads past the last k-tile are unused
  });
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  block_barrier();
  if constexpr (SE::enabled)
    epilogue_staged<BM, BN, EPI, WM, WN, 256>(acc, smem, m0, n0, wm, wn, tid, Mv, N, ea);
  else if constexpr ((EPI == EPI_STORE_F32 || EPI == EPI_RESIDUAL) && WM * (BN + 8) * 4 <= 160 * 1024)
    epilogue_store_halves<EPI, BM, BN, WM, WN, 256>(acc, smem, m0, n0, wm, wn, tid, Mv, N, ea);
  else
    epilogue_w<BM, BN, EPI, WM, WN>(acc, m0, n0, wm, wn, lane, Mv, N, ea);
}

template <int EPI, int BN, int NSA, int NSB>
__global__ void __launch_bounds__(256)
gemm_bf16_w4_kernel(const bf16_t* __restrict__ A, const bf16_t* __restrict__ Bw, int M, int N,
                    int K, const int* __restrict__ M_dev, EpiArgs ea, int n_tm, int n_tn,
                    int tn_off) {
  __shared__ __attribute__((aligned(16))) bf16_t smem[w4_smem_elems<EPI, BN, NSA, NSB>()];
  w4_tile<EPI, BN, NSA, NSB>(A, Bw, M, N, K, M_dev, ea, n_tm, n_tn, tn_off, blockIdx.x, smem);
}

// A column split in one launch: blocks [0, nb1) take the 256 x 256 tiles of
// columns [0, 256 n_tn1), the others the 256 x 128 tiles of the remaining
// 128 n_tn2 columns.  Blocks start in id order, so the 256 x 128 tiles begin
// on each CU as soon as its 256 x 256 tile ends; nb1 is a multiple of 8,
// which keeps each part's XCD mapping.
template <int EPI>
__global__ void __launch_bounds__(256)
gemm_bf16_w4_split_kernel(const bf16_t* __restrict__ A, const bf16_t* __restrict__ Bw, int M,
                          int N, int K, const int* __restrict__ M_dev, EpiArgs ea, int n_tm,
                          int n_tn1, int n_tn2, int nb1) {
  constexpr int E1 = w4_smem_elems<EPI, 256, 2, 3>(), E2 = w4_smem_elems<EPI, 128, 3, 4>();
  __shared__ __attribute__((aligned(16))) bf16_t smem[E1 > E2 ? E1 : E2];
  if ((int)blockIdx.x < nb1)
    w4_tile<EPI, 256, 2, 3>(A, Bw, M, N, K, M_dev, ea, n_tm, n_tn1, 0, blockIdx.x, smem);
  else
    w4_tile<EPI, 128, 3, 4>(A, Bw, M, N, K, M_dev, ea, n_tm, n_tn2, 2 * n_tn1,
                            (int)blockIdx.x - nb1, smem);
}

// columns [c0, c1) of C, both multiples of BN
template <int EPI, int BN>
void launch_w4(hipStream_t st, const bf16_t* A, const bf16_t* B, int M, int N, int K,
               const int* M_dev, const EpiArgs& ea, int c0, int c1) {
  // stage counts: 160 KB of LDS either way
  constexpr int NSA = BN == 256 ? 2 : 3, NSB = BN == 256 ? 3 : 4;
  const int n_tm = ceil_div(M, 256), n_tn = (c1 - c0) / BN;
  if (n_tn <= 0) return;
  gemm_bf16_w4_kernel<EPI, BN, NSA, NSB><<<dim3(round_up(n_tm * n_tn, 8)), dim3(256), 0, st>>>(
      A, B, M, N, K, M_dev, ea, n_tm, n_tn, c0 / BN);
  DLMC_HIP(hipGetLastError());
}

// 256 x 256 tiles on columns [0, c1), 256 x 128 tiles on [c1, N), one launch
template <int EPI>
void launch_w4_split(hipStream_t st, const bf16_t* A, const bf16_t* B, int M, int N, int K,
                     const int* M_dev, const EpiArgs& ea, int c1) {
  const int n_tm = ceil_div(M, 256), n_tn1 = c1 / 256, n_tn2 = (N - c1) / 128;
  const int nb1 = round_up(n_tm * n_tn1, 8), nb2 = round_up(n_tm * n_tn2, 8);
  gemm_bf16_w4_split_kernel<EPI><<<dim3(nb1 + nb2), dim3(256), 0, st>>>(
      A, B, M, N, K, M_dev, ea, n_tm, n_tn1, n_tn2, nb1);
  DLMC_HIP(hipGetLastError());
}

void launch_split(hipStream_t st, const bf16_t* A, const bf16_t* B, int M, int N, int K,
                  const int* M_dev, EpiKind epi, const EpiArgs& ea, int c1) {
  switch (epi) {
    case EPI_STORE_F32: launch_w4_split<EPI_STORE_F32>(st, A, B, M, N, K, M_dev, ea, c1); break;
    case EPI_RESIDUAL: launch_w4_split<EPI_RESIDUAL>(st, A, B, M, N, K, M_dev, ea, c1); break;
    case EPI_GELU: launch_w4_split<EPI_GELU>(st, A, B, M, N, K, M_dev, ea, c1); break;
    case EPI_QKV_ROPE: launch_w4_split<EPI_QKV_ROPE>(st, A, B, M, N, K, M_dev, ea, c1); break;
    case EPI_SWIGLU: launch_w4_split<EPI_SWIGLU>(st, A, B, M, N, K, M_dev, ea, c1); break;
  }
}

template <int BM, int BN, int EPI>
void launch_epi(hipStream_t st, const bf16_t* A, const bf16_t* B, int M, int N, int K,
                const int* M_dev, const EpiArgs& ea) {
  const int n_tm = ceil_div(M, BM), n_tn = ceil_div(N, BN);
  gemm_bf16_kernel<BM, BN, EPI><<<dim3(round_up(n_tm * n_tn, 8)), dim3(256), 0, st>>>(A, B, M, N, K, M_dev, ea, n_tm, n_tn);
  DLMC_HIP(hipGetLastError());
}

template <int BN>
void launch_256(hipStream_t st, const bf16_t* A, const bf16_t* B, int M, int N, int K,
                const int* M_dev, EpiKind epi, const EpiArgs& ea, int c0, int c1) {
  switch (epi) {
    case EPI_STORE_F32: launch_w4<EPI_STORE_F32, BN>(st, A, B, M, N, K, M_dev, ea, c0, c1); break;
    case EPI_RESIDUAL: launch_w4<EPI_RESIDUAL, BN>(st, A, B, M, N, K, M_dev, ea, c0, c1); break;
    case EPI_GELU: launch_w4<EPI_GELU, BN>(st, A, B, M, N, K, M_dev, ea, c0, c1); break;
    case EPI_QKV_ROPE: launch_w4<EPI_QKV_ROPE, BN>(st, A, B, M, N, K, M_dev, ea, c0, c1); break;
    case EPI_SWIGLU: launch_w4<EPI_SWIGLU, BN>(st, A, B, M, N, K, M_dev, ea, c0, c1); break;
  }
}

template <int BM, int BN>
void launch(hipStream_t st, const bf16_t* A, const bf16_t* B, int M, int N, int K,
            const int* M_dev, EpiKind epi, const EpiArgs& ea) {
  switch (epi) {
    case EPI_STORE_F32: launch_epi<BM, BN, EPI_STORE_F32>(st, A, B, M, N, K, M_dev, ea); break;
    case EPI_RESIDUAL: launch_epi<BM, BN, EPI_RESIDUAL>(st, A, B, M, N, K, M_dev, ea); break;
    case EPI_GELU: launch_epi<BM, BN, EPI_GELU>(st, A, B, M, N, K, M_dev, ea); break;
    case EPI_QKV_ROPE:
    case EPI_SWIGLU:
      if constexpr (BN == 256) {
        throw Error(DLMC_E_INVAL, "paired epilogues use BN = 128");
      } else if (epi == EPI_QKV_ROPE) {
        launch_epi<BM, BN, EPI_QKV_ROPE>(st, A, B, M, N, K, M_dev, ea);
      } else {
        launch_epi<BM, BN, EPI_SWIGLU>(st, A, B, M, N, K, M_dev, ea);
      }
      break;
  }
}

}  // namespace

GemmTiles gemm_bf16_tiles(int M, int N, int K, EpiKind epi, int d, int rows_hint) {
  // Tile choice (never changes the result).  Estimated time of an option:
  // waves of tiles x (c0 + k-tiles x c1), where c1 is a tile's main-loop time
  // per 64-wide k-tile with every CU busy, and c0 its fixed cost (prologue
  // and epilogue, which a one-block-per-CU kernel cannot overlap with other
  // work), both in microseconds, fitted to timings on MI355X at M = 2048,
  // K = 4096 and 12288 (8B-shaped layers) and M = 65536, K = 768 and 3072
  // (small layers).  Only the tiles of live rows count.  128 x 128 and
  // 192 x 128 tiles run two blocks per CU (512 slots), so one block's
  // epilogue overlaps the other's main loop; the 4-wave kernel one (256
  // slots).  The
  // 4-wave kernel may also split the columns: 256 x 256 tiles on the first
  // c1, 256 x 128 tiles on the rest (one launch), so that each part fills
  // whole waves of tiles (QKV at M = 2048: Q and K on 256 tiles, V on 256
  // more, instead of three waves of 256 x 128 tiles).
  const int live = std::max(1, rows_hint >= 0 ? std::min(rows_hint, M) : M);
  const int ei = (int)epi;
  //                    fp32 store  residual  QKV   GELU  SwiGLU
  static const double c0_128[5] = {9.3, 9.6, 5.9, 5.0, 5.0};
  static const double c0_w128[5] = {10.6, 13.0, 8.5, 11.7, 11.7};
  static const double c0_w256[5] = {21.5, 50.7, 18.3, 25.9, 7.0};
  static const double c0_192[5] = {17.9, 20.5, 9.0, 9.7, 5.0};
  const double nk = (double)K / BK;
  // c0s: the fixed cost of a wave of tiles that follows another, where it
  // differs from the first wave's
  auto t_of = [&](int bm, int bn, long slots, double c0, double c1, long cols, double c0s = -1.0) -> double {
    if (cols <= 0) return 0.0;
    const long tiles = (long)ceil_div(live, bm) * ceil_div((int)cols, bn);
    const double waves = (double)((tiles + slots - 1) / slots);
    return waves * nk * c1 + c0 + (waves - 1.0) * (c0s >= 0.0 ? c0s : c0);
  };
  // The residual update of 256 x 128 tiles: in a launch of one wave every
  // tile's fp32 read and write of the residual rows happen at once (c0); in
  // later waves they overlap other tiles' main loops, the more so the longer
  // the main loop (about 12.9, 5.8 and 3.3 us per wave at K = 768, 4096 and
  // 12288, M = 65536).
  const double c0s_w128 =
      epi == EPI_RESIDUAL ? c0_w128[ei] * std::min(1.0, std::sqrt(768.0 / (double)K)) : -1.0;
  const double t128 = t_of(128, 128, 512, c0_128[ei], 1.26, N);
  // 192 x 128: QKV tiles must lie inside Q, K or V (d % 128 == 0 holds)
  const double t192 = t_of(192, 128, 512, c0_192[ei], 1.253, N);
  double t4 = 1e300;
  int split = -1;  // columns on 256 x 256 tiles
  // a QKV tile must lie inside one of Q, K, V: 256-wide tiles need d % 256 == 0
  const bool wide_ok = epi != EPI_QKV_ROPE || d % 256 == 0;
  if (N % 128 == 0) {
    auto t_split = [&](int c1) {
      return t_of(256, 256, 256, c0_w256[ei], 1.53, c1) + t_of(256, 128, 256, c0_w128[ei], 0.98, N - c1, c0s_w128);
    };
    // one tile shape (all 256 x 128, or all 256 x 256), then a split if it
    // is more than 3% faster (the estimate rounds each part up to whole
    // waves on its own, a margin for the split's tiles that share a wave)
    split = 0;
    t4 = t_split(0);
    if (wide_ok && N % 256 == 0 && t_split(N) < t4 * (1.0 - 1e-9)) {
      split = N;
      t4 = t_split(N);
    }
    for (int c1 = 256; wide_ok && c1 < N; c1 += 256) {
      const double t = t_split(c1);
      if (t < t4 * 0.97) {
        t4 = t;
        split = c1;
      }
    }
  }
  if (t192 < t128 && (split < 0 || t192 < t4)) return {GEMM_TILES_192x128, 0};
  if (split >= 0 && t4 <= t128) return {GEMM_TILES_4WAVE, split};
  return {GEMM_TILES_128x128, 0};
}

void gemm_bf16(hipStream_t st, const bf16_t* A, const bf16_t* B, int M, int N, int K,
               const int* M_dev, EpiKind epi, const EpiArgs& ea, int rows_hint) {
  DLMC_CHECK(K % BK == 0 && K > 0, DLMC_E_INVAL, "bf16 GEMM needs K % 64 == 0");
  DLMC_CHECK((int64_t)M * K < (1ll << 31) && (int64_t)N * K < (1ll << 31), DLMC_E_INVAL,
             "GEMM operand too large for 32-bit offsets");
  if (M <= 0 || N <= 0) return;
  DLMC_CHECK(!ea.stats || epi == EPI_STORE_F32, DLMC_E_INVAL, "row statistics need the fp32 store");
  const bool paired = (epi == EPI_QKV_ROPE || epi == EPI_SWIGLU);
  DLMC_CHECK(!paired || N % 128 == 0, DLMC_E_INVAL, "paired epilogue needs N % 128 == 0");
  DLMC_CHECK(epi != EPI_QKV_ROPE || (ea.d % 128 == 0 && (ea.dh == 64 || ea.dh == 128)),
             DLMC_E_INVAL, "QKV epilogue needs d % 128 == 0 and head dim 64 or 128");
  const GemmTiles tc = gemm_bf16_tiles(M, N, K, epi, ea.d, rows_hint);
  if (tc.kind == GEMM_TILES_192x128) {
    launch<192, 128>(st, A, B, M, N, K, M_dev, epi, ea);
  } else if (tc.kind == GEMM_TILES_4WAVE) {
    if (tc.split > 0 && tc.split < N) {
      launch_split(st, A, B, M, N, K, M_dev, epi, ea, tc.split);
    } else {
      launch_256<256>(st, A, B, M, N, K, M_dev, epi, ea, 0, tc.split);
      launch_256<128>(st, A, B, M, N, K, M_dev, epi, ea, tc.split, N);
    }
  } else {
    launch<128, 128>(st, A, B, M, N, K, M_dev, epi, ea);
  }
}

}  // namespace dlmc
