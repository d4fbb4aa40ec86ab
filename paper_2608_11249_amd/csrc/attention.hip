// Non-causal (bidirectional) attention of the masked diffusion LM.
//
// Every position attends to every position of its chunk, [MASK] tokens
// included as keys (the bidirectional-conditioning remark after Definition 3):
// O = softmax(Q K^T / sqrt(dh)) V over all T keys, one chunk per batch entry.
//
// bf16 path (gfx950 MFMA): flash-style single pass over 64-key tiles staged
// in LDS, fp32 online-softmax statistics.  Each wave owns 32 queries and
// computes S^T = K Q^T with v_mfma_f32_32x32x16_bf16, so one lane holds 32
// scores of ONE query: the row max / row sum need one cross-lane exchange
// (lane ^ 32) instead of a 32-lane reduction.  The probabilities then feed
// O^T += V^T P^T directly from the S^T accumulator registers; the MFMA k-slot
// order of P^T is a permutation of the keys, and the V^T fragment is read
// from LDS with the same permutation.  Key tiles are visited in a fixed order,
// so results do not depend on the launch shape or on other chunks.
#include "kernels.h"

namespace dlmc {
namespace {

constexpr int KT = 64;   // keys per tile
constexpr int QB = 128;  // queries per block (4 waves x 32)

// LDS swizzles for gfx950's 64 four-byte banks (256 B per cycle).
// K tile: rows of DH bf16; the 16 keys a 16-lane ds_read_b128 group reads in
// one k step must hit 16 distinct 16-byte slots: with 256-byte rows (DH = 128)
// XOR the chunk with key & 15, with 128-byte rows (DH = 64) rows r and r + 2
// share banks, so XOR with (key >> 1) & 7.
template <int DH>
__device__ __forceinline__ int kswz(int key) {
  return DH == 128 ? (key & 15) : ((key >> 1) & 7);
}
// V^T tile: rows d of 64 keys (128 B) in 8-byte units; the 32 rows a 32-lane
// ds_read_b64 group reads must hit 32 distinct 8-byte slots: rows d and d + 2
// share banks, so unit u of row d is stored at u ^ ((d >> 1) & 15).
__device__ __forceinline__ int vswz(int d) { return (d >> 1) & 15; }

// 2^x for x <= 0 (or -inf) with the hardware exponential
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int DH>
__global__ void __launch_bounds__(256)
attn_bf16_kernel(const bf16_t* __restrict__ Q, const bf16_t* __restrict__ Kg,
                 const bf16_t* __restrict__ Vt, bf16_t* __restrict__ O, int H, int T, int Tp,
                 float scale_log2) {
  constexpr int DC = DH / 8;                 // 16-byte chunks per key row
  constexpr int K_CH = KT * DC / 256;        // K-tile chunks per thread
  constexpr int V_CH = DH * (KT / 8) / 256;  // V^T-tile chunks per thread
  __shared__ __attribute__((aligned(16))) bf16_t Ks[2][KT * DH];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[2][DH * KT];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lg = lane >> 5;
  const int h = blockIdx.y, b = blockIdx.z;
  const size_t bh = (size_t)b * H + h;
  const bf16_t* Qp = Q + bh * Tp * DH;
  const bf16_t* Kp = Kg + bh * Tp * DH;
  const bf16_t* Vp = Vt + bh * DH * Tp;
  const int q0 = blockIdx.x * QB + wave * 32;

  // B operand of S^T = K Q^T: lane holds Q[q0 + lr][16 s + 8 lg .. + 7]
  bf16x8 qf[DH / 16];
#pragma unroll
  for (int s = 0; s < DH / 16; ++s)
    qf[s] = *reinterpret_cast<const bf16x8*>(Qp + (size_t)(q0 + lr) * DH + s * 16 + lg * 8);

  // tile loaders (Tp is a multiple of QB, so every row read is inside the buffer;
  // rows at or beyond T hold finite values and get zero probability)
  u32x4 rk[K_CH], rv[V_CH];
  auto gload = [&](int k0) {
#pragma unroll
    for (int j = 0; j < K_CH; ++j) {
      const int c = tid + 256 * j, key = c / DC, dc = c % DC;
      rk[j] = *reinterpret_cast<const u32x4*>(Kp + (size_t)(k0 + key) * DH + dc * 8);
    }
#pragma unroll
    for (int j = 0; j < V_CH; ++j) {
      const int c = tid + 256 * j, d = c >> 3, kc = c & 7;
      rv[j] = *reinterpret_cast<const u32x4*>(Vp + (size_t)d * Tp + k0 + kc * 8);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int j = 0; j < K_CH; ++j) {
      const int c = tid + 256 * j, key = c / DC, dc = c % DC;
      *reinterpret_cast<u32x4*>(&Ks[buf][key * DH + ((dc ^ kswz<DH>(key)) << 3)]) = rk[j];
    }
#pragma unroll
    for (int j = 0; j < V_CH; ++j) {
      // V^T row d holds 16 8-byte units (4 keys each); unit u is stored at
      // u ^ vswz(d).  A 16-byte chunk = units (2kc, 2kc+1) lands on the unit
      // pair kc ^ (x >> 1), halves swapped when x is odd.
      const int c = tid + 256 * j, d = c >> 3, kc = c & 7, x = vswz(d);
      u32x4 v = rv[j];
      if (x & 1) v = u32x4{v.z, v.w, v.x, v.y};
      *reinterpret_cast<u32x4*>(&Vs[buf][d * KT + ((kc ^ (x >> 1)) << 3)]) = v;
    }
  };

  f32x16 o[DH / 32];
#pragma unroll
  for (int t = 0; t < DH / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;

  const int n_kt = (T + KT - 1) / KT;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < n_kt; ++kt) {
    const int cur = kt & 1, k0 = kt * KT;
    if (kt + 1 < n_kt) gload(k0 + KT);

    // S^T tiles: keys 0-31 (s0) and 32-63 (s1) of this tile x 32 queries
    f32x16 s0, s1;
#pragma unroll
    for (int r = 0; r < 16; ++r) s0[r] = s1[r] = 0.0f;
#pragma unroll
    for (int s = 0; s < DH / 16; ++s) {
      const int dc = s * 2 + lg;
      const int key0 = lr, key1 = 32 + lr;
      const bf16x8 k0f = *reinterpret_cast<const bf16x8*>(&Ks[cur][key0 * DH + ((dc ^ kswz<DH>(key0)) << 3)]);
      const bf16x8 k1f = *reinterpret_cast<const bf16x8*>(&Ks[cur][key1 * DH + ((dc ^ kswz<DH>(key1)) << 3)]);
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0f, qf[s], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1f, qf[s], s1, 0, 0, 0);
    }

    // online softmax (base 2) for query q0 + lr; this lane holds keys
    // (r/4)*8 + lg*4 + r%4 (+32 for s1) of the tile
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = k0 + (r >> 2) * 8 + lg * 4 + (r & 3);
      s0[r] = key < T ? s0[r] * scale_log2 : -INFINITY;
      s1[r] = key + 32 < T ? s1[r] * scale_log2 : -INFINITY;
      mx = fmaxf(mx, fmaxf(s0[r], s1[r]));
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = fast_exp2(m_run - m_new);
    float psum = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s0[r] = fast_exp2(s0[r] - m_new);
      s1[r] = fast_exp2(s1[r] - m_new);
      psum += s0[r] + s1[r];
    }
    psum += __shfl_xor(psum, 32);
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < DH / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][r] *= alpha;

    // P^T fragments: k-step j covers keys 16j..16j+15 of the tile; this lane's
    // k-slots 8lg+0..3 are keys 16j+4lg+0..3, slots 8lg+4..7 keys 16j+8+4lg+0..3,
    // i.e. accumulator registers 8(j%2) .. 8(j%2)+7 of tile j/2.
    bf16x8 pf[4];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pf[0][e] = (__bf16)s0[e];
      pf[1][e] = (__bf16)s0[8 + e];
      pf[2][e] = (__bf16)s1[e];
      pf[3][e] = (__bf16)s1[8 + e];
    }
#pragma unroll
    for (int t = 0; t < DH / 32; ++t) {
      const int d = t * 32 + lr, x = vswz(d);
      const bf16_t* vrow = &Vs[cur][d * KT];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int u1 = 4 * j + lg, u2 = 4 * j + 2 + lg;
        const u32x2 a = *reinterpret_cast<const u32x2*>(vrow + ((u1 ^ x) << 2));
        const u32x2 c = *reinterpret_cast<const u32x2*>(vrow + ((u2 ^ x) << 2));
        const bf16x8 vf = __builtin_bit_cast(bf16x8, u32x4{a.x, a.y, c.x, c.y});
        o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[j], o[t], 0, 0, 0);
      }
    }
    if (kt + 1 < n_kt) sstore(cur ^ 1);
    __syncthreads();
  }

  const int q = q0 + lr;
  if (q < T) {
    const float inv = 1.0f / l_run;
    bf16_t* orow = O + ((size_t)b * T + q) * (size_t)(H * DH) + h * DH;
#pragma unroll
    for (int t = 0; t < DH / 32; ++t)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int d = t * 32 + a * 8 + lg * 4;
        const uint32_t w0 = (uint32_t)f32_to_bf16(o[t][4 * a] * inv) |
                            ((uint32_t)f32_to_bf16(o[t][4 * a + 1] * inv) << 16);
        const uint32_t w1 = (uint32_t)f32_to_bf16(o[t][4 * a + 2] * inv) |
                            ((uint32_t)f32_to_bf16(o[t][4 * a + 3] * inv) << 16);
        *reinterpret_cast<u32x2*>(orow + d) = u32x2{w0, w1};
      }
  }
}

// fp32 path: one thread per query, 64-key tiles staged in LDS, exact-order
// online softmax with expf.  Used by the fp32 model only (small shapes).
template <int DH>
__global__ void __launch_bounds__(64)
attn_f32_kernel(const float* __restrict__ Q, const float* __restrict__ Kg,
                const float* __restrict__ Vt, float* __restrict__ O, int H, int T, int Tp,
                float scale) {
  __shared__ float Ks[64][DH + 1];
  __shared__ float Vs[64][DH + 1];
  const int tid = threadIdx.x, h = blockIdx.y, b = blockIdx.z;
  const size_t bh = (size_t)b * H + h;
  const int q = blockIdx.x * 64 + tid;
  float qv[DH], o[DH];
#pragma unroll
  for (int d = 0; d < DH; ++d) {
    qv[d] = Q[(bh * Tp + min(q, T - 1)) * DH + d];
    o[d] = 0.0f;
  }
  float m = -INFINITY, l = 0.0f;
  for (int k0 = 0; k0 < T; k0 += 64) {
    const int nk = min(64, T - k0);
    for (int i = tid; i < 64 * DH; i += 64) {
      const int kk = i / DH, d = i % DH;
      const int key = min(k0 + kk, T - 1);
      Ks[kk][d] = Kg[(bh * Tp + key) * DH + d];
      Vs[kk][d] = Vt[(bh * DH + d) * Tp + key];
    }
    __syncthreads();
    for (int kk = 0; kk < nk; ++kk) {
      float s = 0.0f;
#pragma unroll
      for (int d = 0; d < DH; ++d) s += qv[d] * Ks[kk][d];
      s *= scale;
      if (s > m) {
        const float corr = expf(m - s);
        l *= corr;
#pragma unroll
        for (int d = 0; d < DH; ++d) o[d] *= corr;
        m = s;
      }
      const float p = expf(s - m);
      l += p;
#pragma unroll
      for (int d = 0; d < DH; ++d) o[d] += p * Vs[kk][d];
    }
    __syncthreads();
  }
  if (q < T) {
    float* orow = O + ((size_t)b * T + q) * (size_t)(H * DH) + h * DH;
#pragma unroll
    for (int d = 0; d < DH; ++d) orow[d] = o[d] / l;
  }
}

}  // namespace

void attention_bf16(hipStream_t st, const bf16_t* q, const bf16_t* k, const bf16_t* vt,
                    bf16_t* out, int B, int H, int T, int Tp, int dh) {
  if (B <= 0 || T <= 0) return;
  DLMC_CHECK(Tp % QB == 0 && Tp >= T, DLMC_E_INVAL, "attention: padded length must be a multiple of 128");
  dim3 grid(ceil_div(T, QB), H, B), block(256);
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)dh);
  if (dh == 128) {
    attn_bf16_kernel<128><<<grid, block, 0, st>>>(q, k, vt, out, H, T, Tp, scale_log2);
  } else if (dh == 64) {
    attn_bf16_kernel<64><<<grid, block, 0, st>>>(q, k, vt, out, H, T, Tp, scale_log2);
  } else {
    throw Error(DLMC_E_INVAL, "bf16 attention supports head dims 64 and 128");
  }
  DLMC_HIP(hipGetLastError());
}

void attention_f32(hipStream_t st, const float* q, const float* k, const float* vt, float* out,
                   int B, int H, int T, int Tp, int dh) {
  if (B <= 0 || T <= 0) return;
  dim3 grid(ceil_div(T, 64), H, B), block(64);
  const float scale = 1.0f / sqrtf((float)dh);
  switch (dh) {
    case 16: attn_f32_kernel<16><<<grid, block, 0, st>>>(q, k, vt, out, H, T, Tp, scale); break;
    case 32: attn_f32_kernel<32><<<grid, block, 0, st>>>(q, k, vt, out, H, T, Tp, scale); break;
    case 64: attn_f32_kernel<64><<<grid, block, 0, st>>>(q, k, vt, out, H, T, Tp, scale); break;
    case 128: attn_f32_kernel<128><<<grid, block, 0, st>>>(q, k, vt, out, H, T, Tp, scale); break;
    default: throw Error(DLMC_E_INVAL, "fp32 attention supports head dims 16, 32, 64, 128");
  }
  DLMC_HIP(hipGetLastError());
}

}  // namespace dlmc
