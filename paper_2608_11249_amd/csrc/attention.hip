// Non-causal (bidirectional) attention of the masked diffusion LM.
//
// Every position attends to every position of its chunk, [MASK] tokens
// included as keys (the bidirectional-conditioning remark after Definition 3):
// O = softmax(Q K^T / sqrt(dh)) V over all T keys, one chunk per batch entry.
//
// bf16 path (gfx950 MFMA): flash-style single pass over 64-key tiles with
// fp32 online-softmax statistics.  Each wave owns 32 queries and computes
// S^T = K Q^T with v_mfma_f32_32x32x16_bf16, so one lane holds 32 scores of
// ONE query and the row max / row sum need one cross-lane exchange
// (lane ^ 32).  The probabilities feed O^T += V^T P^T straight from the S^T
// accumulator registers.  To make the k-slots of P^T consecutive keys, the K
// tile is stored in LDS with its rows permuted inside every group of 16
// (row i holds key sigma(i), bits 2 and 3 of i swapped); the V^T fragment of
// a lane is then 8 consecutive keys, one ds_read_b128.  Tiles move global ->
// LDS with direct loads (global_load_lds_dwordx4) into a double buffer, so no
// registers stage them and two waves fit per SIMD.  Key tiles are visited in
// a fixed order, so results do not depend on the launch shape or on other
// chunks.  A block holds QB = 128 or 256 queries (4 or 8 waves, two waves per
// SIMD either way); with 256 every K / V tile moved into LDS serves twice as
// many queries, which halves the tile traffic per CU.
//
// Tiles go through a ring of NB LDS buffers, issued NB - 1 tiles ahead.  The
// end of a tile waits (s_waitcnt vmcnt) only for the loads of the next tile
// -- those of the tiles after it stay in flight -- and then meets the other
// waves at a bare s_barrier: __syncthreads() would also wait for every direct
// load still in flight, which would take away the lookahead.
#include <type_traits>

#include "kernels.h"

namespace dlmc {
namespace {

constexpr int KT = 64;  // keys per tile

// LDS row i of a K tile holds key sigma(i) of the tile (an involution)
__device__ __forceinline__ int sigma(int i) { return (i & ~12) | ((i & 4) << 1) | ((i & 8) >> 1); }

// LDS swizzles for gfx950's 64 four-byte banks (256 B per cycle): the 16
// rows a 16-lane ds_read_b128 group reads must hit 16 distinct 16-byte slots.
// K rows of DH bf16: with 256-byte rows (DH = 128) XOR the chunk with i & 15;
// with 128-byte rows (DH = 64) rows i and i + 2 share banks, so XOR with
// (i >> 1) & 7.  V^T rows are 64 keys (128 bytes): XOR with (d >> 1) & 7.
template <int DH>
__device__ __forceinline__ int kswz(int i) {
  return DH == 128 ? (i & 15) : ((i >> 1) & 7);
}
__device__ __forceinline__ int vswz(int d) { return (d >> 1) & 7; }

// 2^x for x <= 0 (or -inf) with the hardware exponential
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// 16-byte direct global -> LDS load; `lds` is wave-uniform, lane l writes
// lds + 16 l bytes.  The builtin exists only for the device target.
__device__ __forceinline__ void lds_dma16(const bf16_t* g, bf16_t* lds) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0);
#endif
}

// s_barrier without the memory fence of __syncthreads(), which would also wait
// for the direct loads still in flight
__device__ __forceinline__ void block_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// s_waitcnt immediate: vmcnt(n) with lgkmcnt(0)
constexpr int waitcnt_vm(int n) { return 0x0070 | (n & 15) | ((n >> 4) << 14); }

template <int DH, int QB, int NB>
__global__ void __launch_bounds__(2 * QB, 256 / QB)
attn_bf16_kernel(const bf16_t* __restrict__ Q, const bf16_t* __restrict__ Kg,
                 const bf16_t* __restrict__ Vt, bf16_t* __restrict__ O, int H, int T, int Tp,
                 float scale_log2) {
  constexpr int NWV = QB / 32;       // waves per block (32 queries each)
  constexpr int NS = DH / 16;        // k steps of S^T
  constexpr int RB = DH * 2;         // bytes per K row
  constexpr int KRW = 1024 / RB;     // K rows per 1 KB load window
  constexpr int KW = KT / KRW / NWV; // K windows per wave
  constexpr int VW = DH / 8 / NWV;   // V^T windows (8 rows of 128 B) per wave
  static_assert(KW >= 1 && VW >= 1 && KW * KRW * NWV == KT && VW * 8 * NWV == DH, "tile split");
  constexpr int NV = DH / 32 * 4;    // PV MFMAs per tile
  constexpr int NL = KW + VW;        // direct loads per wave per tile
  constexpr int LA = NB - 1;         // tiles loaded ahead
  static_assert(LA >= 1 && (LA - 1) * NL < 64 && NB <= 3, "ring size / vmcnt field");
  __shared__ __attribute__((aligned(16))) bf16_t Ks[NB][KT * DH];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[NB][DH * KT];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lg = lane >> 5;
  // 1-D grid of (query block, head, batch).  Hardware block ids go round
  // robin over the 8 XCDs; the remap gives each XCD a contiguous range of
  // logical blocks, so the query blocks of a head run on one XCD and share
  // that head's K / V tiles through its L2.
  const int nqb = (T + QB - 1) / QB;
  const int nb = gridDim.x;
  int bid = blockIdx.x;
  if ((nb & 7) == 0) bid = (bid & 7) * (nb >> 3) + (bid >> 3);
  const int qblk = bid % nqb, h = (bid / nqb) % H, b = bid / (nqb * H);
  const size_t bh = (size_t)b * H + h;
  const bf16_t* Qp = Q + bh * Tp * DH;
  const bf16_t* Kp = Kg + bh * Tp * DH;
  const bf16_t* Vp = Vt + bh * DH * Tp;
  const int q0 = qblk * QB + wave * 32;

  // B operand of S^T = K Q^T: lane holds Q[q0 + lr][16 s + 8 lg .. + 7]
  bf16x8 qf[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    qf[s] = *reinterpret_cast<const bf16x8*>(Qp + (size_t)(q0 + lr) * DH + s * 16 + lg * 8);

  // Per-lane sources of the direct loads (element offsets inside a tile).  Lane
  // l of a window fills LDS row i, 16-byte slot p, with chunk p ^ swizzle of
  // key sigma(i).  Tp is a multiple of 128, so every row read is inside the
  // buffer; rows at or beyond T hold finite values and get zero probability.
  int k_src[KW], v_src[VW];
#pragma unroll
  for (int w = 0; w < KW; ++w) {
    const int i = (wave * KW + w) * KRW + lane / (RB / 16), p = lane % (RB / 16);
    k_src[w] = sigma(i) * DH + ((p ^ kswz<DH>(i)) << 3);
  }
#pragma unroll
  for (int w = 0; w < VW; ++w) {
    const int d = (wave * VW + w) * 8 + (lane >> 3), p = lane & 7;
    v_src[w] = d * Tp + ((p ^ vswz(d)) << 3);
  }
  auto load_tile = [&](int kt, int buf) {
#pragma unroll
    for (int w = 0; w < KW; ++w)
      lds_dma16(Kp + (size_t)kt * KT * DH + k_src[w], &Ks[buf][(wave * KW + w) * 512]);
#pragma unroll
    for (int w = 0; w < VW; ++w)
      lds_dma16(Vp + kt * KT + v_src[w], &Vs[buf][(wave * VW + w) * 512]);
  };

  // LDS byte offsets of this lane's fragment reads inside one K / V^T tile
  // (loop invariant; the buffer half is a constant added per unrolled trip)
  int koff[NS][2], voff[NV];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const int dc = 2 * s + lg;
    koff[s][0] = (lr * DH + ((dc ^ kswz<DH>(lr)) << 3)) * 2;
    koff[s][1] = ((32 + lr) * DH + ((dc ^ kswz<DH>(32 + lr)) << 3)) * 2;
  }
#pragma unroll
  for (int idx = 0; idx < NV; ++idx) {
    const int t = idx >> 2, j = idx & 3, d = t * 32 + lr, c = 2 * j + lg;
    voff[idx] = (d * KT + ((c ^ vswz(d)) << 3)) * 2;
  }

  f32x16 o[DH / 32];
#pragma unroll
  for (int t = 0; t < DH / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;
  // Running max in log2 units.  It is raised only when a tile's max exceeds
  // it by more than RESCALE_LOG2: until then every probability 2^(s - m_run)
  // stays below 2^RESCALE_LOG2 (exact in fp32, no loss in bf16), and O and l
  // share the stale max, so O / l is unchanged -- the rescale of O is skipped
  // on most tiles.
  constexpr float RESCALE_LOG2 = 8.0f;
  float m_run = -INFINITY, l_run = 0.0f;

  const int n_kt = (T + KT - 1) / KT;
  const char* ks_base = reinterpret_cast<const char*>(&Ks[0][0]);
  const char* vs_base = reinterpret_cast<const char*>(&Vs[0][0]);
  // S^T of the tile in buffer `cur` for LDS rows 0-31 (s0) and 32-63 (s1).
  // Fragment reads run KA k steps ahead of the MFMAs; the scheduling fences
  // keep the compiler from sinking them next to their use, which would expose
  // the LDS latency at every step.  The last steps also start the reads of
  // the first VA V^T fragments of the same tile, for the PV product.
  constexpr int KA = NS < 4 ? NS : 4;
  constexpr int VA = 4;
  auto scores = [&](int cur, f32x16& s0, f32x16& s1, bf16x8(&vf)[VA]) {
#pragma unroll
    for (int r = 0; r < 16; ++r) s0[r] = s1[r] = 0.0f;
    const char* kb = ks_base + cur * KT * DH * 2;
    const char* vb = vs_base + cur * DH * KT * 2;
    bf16x8 kf[KA][2];
    auto kload = [&](int s, bf16x8(&f)[2]) {
      f[0] = *reinterpret_cast<const bf16x8*>(kb + koff[s][0]);
      f[1] = *reinterpret_cast<const bf16x8*>(kb + koff[s][1]);
    };
#pragma unroll
    for (int s = 0; s < KA; ++s) kload(s, kf[s]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s % KA][0], qf[s], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s % KA][1], qf[s], s1, 0, 0, 0);
      if (s + KA < NS) kload(s + KA, kf[s % KA]);
      if (s + KA >= NS && s + KA - NS < VA)
        vf[s + KA - NS] = *reinterpret_cast<const bf16x8*>(vb + voff[s + KA - NS]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // online softmax (base 2) of the tile starting at key k0 for query q0 + lr,
  // leaving the P^T fragments in pf.  Register r of s0 holds key
  // 16 (r >> 3) + 8 lg + (r & 7) of the tile (s1: + 32).
  auto softmax = [&](int k0, f32x16& s0, f32x16& s1, bf16x8(&pf)[4]) {
    if (k0 + KT > T) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + 16 * (r >> 3) + 8 * lg + (r & 7);
        if (key >= T) s0[r] = -INFINITY;
        if (key + 32 >= T) s1[r] = -INFINITY;
      }
    }
    float m4[4];
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      float m = fmaxf(s0[4 * a], s1[4 * a]);
#pragma unroll
      for (int e = 1; e < 4; ++e) m = fmaxf(m, fmaxf(s0[4 * a + e], s1[4 * a + e]));
      m4[a] = m;
    }
    float mx = fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3]));
    mx = fmaxf(mx, __shfl_xor(mx, 32)) * scale_log2;
    if (__builtin_amdgcn_ballot_w64(mx > m_run + RESCALE_LOG2)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = fast_exp2(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int t = 0; t < DH / 32; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[t][r] *= alpha;
      m_run = m_new;
    }
    float ps[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s0[r] = fast_exp2(fmaf(s0[r], scale_log2, -m_run));
      s1[r] = fast_exp2(fmaf(s1[r], scale_log2, -m_run));
      ps[r & 3] += s0[r] + s1[r];
    }
    float psum = (ps[0] + ps[1]) + (ps[2] + ps[3]);
    psum += __shfl_xor(psum, 32);
    l_run += psum;
    // P^T fragment of k step j: keys 16 j + 8 lg .. + 7 = registers
    // 8 (j % 2) .. + 7 of tile j / 2
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pf[0][e] = (__bf16)s0[e];
      pf[1][e] = (__bf16)s0[8 + e];
      pf[2][e] = (__bf16)s1[e];
      pf[3][e] = (__bf16)s1[8 + e];
    }
  };

  // O^T += V^T P^T with the V^T tile in buffer `cur`; the V^T fragment of
  // row d, k step j is chunk 2 j + lg.  Reads run VA MFMAs ahead; the first
  // VA are already in vf (started by the scores of the same tile).
  auto pv = [&](int cur, const bf16x8(&pf)[4], bf16x8(&vf)[VA]) {
    const char* vb = vs_base + cur * DH * KT * 2;
    auto vload = [&](int idx, bf16x8& f) { f = *reinterpret_cast<const bf16x8*>(vb + voff[idx]); };
#pragma unroll
    for (int idx = 0; idx < NV; ++idx) {
      o[idx >> 2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[idx % VA], pf[idx & 3], o[idx >> 2], 0, 0, 0);
      if (idx + VA < NV) vload(idx + VA, vf[idx % VA]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Interval kt: start the loads of tile kt + LA into the buffer of tile
  // kt - 1, which every wave finished before the barrier that ended the
  // previous interval; compute; wait until tile kt + 1 has landed (this wave's
  // loads; the LA - 1 tiles after it may still be in flight) and meet the
  // other waves, after which every wave's loads of tile kt + 1 have landed.
  auto interval_end = [&](int kt) {
    if (kt + LA < n_kt)
      __builtin_amdgcn_s_waitcnt(waitcnt_vm((LA - 1) * NL));
    else
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    block_barrier();
  };
  auto tile = [&](int kt, auto cur_c) {
    constexpr int cur = decltype(cur_c)::value;  // kt % NB
    if (kt + LA < n_kt) load_tile(kt + LA, (cur + LA) % NB);
    f32x16 s0, s1;
    bf16x8 vf[VA], pf[4];
    scores(cur, s0, s1, vf);
    softmax(kt * KT, s0, s1, pf);
    pv(cur, pf, vf);
    interval_end(kt);
  };

  // prologue: tiles 0 .. LA - 1; tile 0 landed before the first interval
#pragma unroll
  for (int t = 0; t < LA; ++t)
    if (t < n_kt) load_tile(t, t);
  if (LA <= n_kt)
    __builtin_amdgcn_s_waitcnt(waitcnt_vm((LA - 1) * NL));
  else
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  block_barrier();
  // NB tiles per trip, so each trip's buffer offsets are constants
  for (int kt = 0; kt < n_kt; kt += NB) {
    tile(kt, std::integral_constant<int, 0>{});
    if (kt + 1 < n_kt) tile(kt + 1, std::integral_constant<int, 1>{});
    if constexpr (NB >= 3)
      if (kt + 2 < n_kt) tile(kt + 2, std::integral_constant<int, 2 % NB>{});
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
  DLMC_CHECK(Tp % 128 == 0 && Tp >= T, DLMC_E_INVAL, "attention: padded length must be a multiple of 128");
  DLMC_CHECK(dh == 128 || dh == 64, DLMC_E_INVAL, "bf16 attention supports head dims 64 and 128");
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)dh);
  // 256-query blocks (half the K / V traffic per CU) when the padded rows
  // cover them and there is at least one block per CU; else 128
  const bool wide = Tp % 256 == 0 && (long)(Tp / 256) * H * B >= 256;
  auto run = [&](auto dh_c, auto qb_c) {
    constexpr int DH = decltype(dh_c)::value, QB = decltype(qb_c)::value;
    // three tile buffers (96 KB) for one 256-query block per CU; two (64 KB)
    // keep two 128-query blocks per CU
    constexpr int NB = QB == 256 ? 3 : 2;
    dim3 grid(ceil_div(T, QB) * H * B), block(2 * QB);
    attn_bf16_kernel<DH, QB, NB><<<grid, block, 0, st>>>(q, k, vt, out, H, T, Tp, scale_log2);
  };
  using I64 = std::integral_constant<int, 64>;
  using I128 = std::integral_constant<int, 128>;
  using I256 = std::integral_constant<int, 256>;
  if (dh == 128) {
    if (wide) run(I128{}, I256{}); else run(I128{}, I128{});
  } else {
    if (wide) run(I64{}, I256{}); else run(I64{}, I128{});
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
