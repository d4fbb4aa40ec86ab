// Symbol ranking on the GPU (Definition of Symbol Ranking): the rank of a
// symbol is its index in the list of all symbols ordered by non-increasing
// probability, equal probabilities by token id.  Probability order is logit
// order, so both kernels compare 32-bit keys of the fp32 logits that sort
// ascending in rank order (larger logits first; -0 counts as +0).
//
// Encode: rank = #{v : (key_v, v) < (key_s, s)} -- one read of the row.
// Decode: the symbol of rank r by radix selection over the keys (four 8-bit
// digit passes with LDS histograms), then the r'-th id among the symbols that
// carry the selected key, found by a block-wide prefix count in id order.
// Both kernels also reveal the symbol in the state.
#include "kernels.h"

namespace dlmc {
namespace {

constexpr int RT = 1024;  // threads per row

__device__ __forceinline__ uint32_t rank_key(float l) {
  uint32_t u = __float_as_uint(l);
  if (u == 0x80000000u) u = 0u;
  const uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);  // ascending in l
  return ~asc;
}

// exclusive prefix sum over the RT threads of a block; returns the block total in *total
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t x, uint32_t* lds, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t incl = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == 63) lds[wave] = incl;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t run = 0;
    for (int w = 0; w < RT / 64; ++w) {
      const uint32_t t = lds[w];
      lds[w] = run;
      run += t;
    }
    lds[RT / 64] = run;
  }
  __syncthreads();
  const uint32_t ex = lds[wave] + incl - x;
  *total = lds[RT / 64];
  __syncthreads();
  return ex;
}

__global__ void __launch_bounds__(RT)
rank_kernel(const float* __restrict__ logits, const int32_t* __restrict__ sel_row,
            const int32_t* __restrict__ sel_pos, const int32_t* __restrict__ n_sel,
            const int32_t* __restrict__ tokens, const int64_t* __restrict__ slot_base,
            int32_t* __restrict__ state, int T, int m_max, int V, uint32_t* __restrict__ out) {
  __shared__ uint32_t lds[RT / 64 + 1];
  const int b = blockIdx.y, j = blockIdx.x;
  if (j >= n_sel[b]) return;
  const int slot = b * m_max + j, pos = sel_pos[slot];
  const int s = tokens[slot_base[b] + pos];
  const float* row = logits + (size_t)sel_row[slot] * V;
  const uint32_t ks = rank_key(row[s]);
  uint32_t cnt = 0;
  for (int v = threadIdx.x; v < V; v += RT) {
    const uint32_t kv = rank_key(row[v]);
    cnt += (kv < ks) || (kv == ks && v < s);
  }
  uint32_t total;
  (void)block_exclusive_scan(cnt, lds, &total);
  if (threadIdx.x == 0) {
    out[2 * slot] = total;
    out[2 * slot + 1] = (uint32_t)s;
    state[(size_t)b * T + pos] = s;
  }
}

__global__ void __launch_bounds__(RT)
select_rank_kernel(const float* __restrict__ logits, const int32_t* __restrict__ sel_row,
                   const int32_t* __restrict__ sel_pos, const int32_t* __restrict__ n_sel,
                   int32_t* __restrict__ dec, int32_t* __restrict__ state, int T, int m_max, int V) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t lds[RT / 64 + 1];
  __shared__ uint32_t sh_prefix, sh_rest;
  const int b = blockIdx.y, j = blockIdx.x;
  if (j >= n_sel[b]) return;
  const int slot = b * m_max + j, pos = sel_pos[slot];
  const float* row = logits + (size_t)sel_row[slot] * V;
  uint32_t prefix = 0, mask = 0, rest = (uint32_t)dec[slot];  // rank, 0 <= rank < V
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int d = threadIdx.x; d < 256; d += RT) hist[d] = 0;
    __syncthreads();
    for (int v = threadIdx.x; v < V; v += RT) {
      const uint32_t k = rank_key(row[v]);
      if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t cum = 0, d = 0;
      for (; d < 255; ++d) {
        if (cum + hist[d] > rest) break;
        cum += hist[d];
      }
      sh_prefix = prefix | (d << shift);
      sh_rest = rest - cum;
    }
    __syncthreads();
    prefix = sh_prefix;
    rest = sh_rest;
    mask |= 255u << shift;
    __syncthreads();
  }
  // the rest-th id (in id order) among the symbols whose key is `prefix`
  const int per = (V + RT - 1) / RT, lo = threadIdx.x * per, hi = min(lo + per, V);
  uint32_t c = 0;
  for (int v = lo; v < hi; ++v) c += rank_key(row[v]) == prefix;
  uint32_t total;
  uint32_t base = block_exclusive_scan(c, lds, &total);
  if (rest >= base && rest < base + c) {
    for (int v = lo; v < hi; ++v) {
      if (rank_key(row[v]) != prefix) continue;
      if (base == rest) {
        dec[slot] = v;
        state[(size_t)b * T + pos] = v;
        break;
      }
      ++base;
    }
  }
}

}  // namespace

void rank_symbols(hipStream_t st, const float* logits, const int32_t* sel_row,
                  const int32_t* sel_pos, const int32_t* n_sel, const int32_t* tokens,
                  const int64_t* slot_base, int32_t* state, int B, int T, int m_max, int V,
                  uint32_t* out) {
  if (B <= 0 || m_max <= 0) return;
  DLMC_CHECK(m_max <= 65535 && B <= 65535, DLMC_E_INVAL, "too many rank rows per launch");
  rank_kernel<<<dim3(m_max, B), RT, 0, st>>>(logits, sel_row, sel_pos, n_sel, tokens, slot_base,
                                             state, T, m_max, V, out);
  DLMC_HIP(hipGetLastError());
}

void select_by_rank(hipStream_t st, const float* logits, const int32_t* sel_row,
                    const int32_t* sel_pos, const int32_t* n_sel, int32_t* dec, int32_t* state,
                    int B, int T, int m_max, int V) {
  if (B <= 0 || m_max <= 0) return;
  DLMC_CHECK(m_max <= 65535 && B <= 65535, DLMC_E_INVAL, "too many rank rows per launch");
  select_rank_kernel<<<dim3(m_max, B), RT, 0, st>>>(logits, sel_row, sel_pos, n_sel, dec, state, T,
                                                    m_max, V);
  DLMC_HIP(hipGetLastError());
}

}  // namespace dlmc
