// bf16 MFMA GEMM for gfx950 with fused epilogues: C = A * B^T, fp32 accumulate.
//
// Every dense contraction of the forward pass (QKV, O, FFN in/out, LM head)
// runs here.  Block tile BM x BN x 64 with four 64-wide waves in a 2 x 2
// grid; each wave owns a (BM/2) x (BN/2) sub-tile built from
// v_mfma_f32_32x32x16_bf16 tiles.  Global -> register -> LDS staging is double
// buffered (one barrier per k-tile).  LDS rows are 64 bf16 (128 B); the eight
// 16-byte chunks of row r are stored XOR-swizzled by (r & 7) so the
// ds_read_b128 fragment loads of 8 consecutive rows hit 8 distinct bank groups.
//
// Numerics: each output element is a sequential sum over k-tiles, each k-tile
// four MFMA steps in order, independent of the tile shape and of which other
// rows are in the launch, so results are identical for any batch composition.
#include "kernels.h"

namespace dlmc {
namespace {

constexpr int BK = 64;

__device__ __forceinline__ float gelu_erf(float v) {
  return 0.5f * v * (1.0f + erff(v * 0.70710678118654752440f));
}
__device__ __forceinline__ float silu(float v) { return v / (1.0f + expf(-v)); }

template <int BM, int BN, int EPI>
__global__ void __launch_bounds__(256)
gemm_bf16_kernel(const bf16_t* __restrict__ A, const bf16_t* __restrict__ Bw, int M, int N,
                 int K, const int* __restrict__ M_dev, EpiArgs ea, int n_tm) {
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int A_CH = BM * BK / 8 / 256;  // 16-byte chunks per thread per k-tile
  constexpr int B_CH = BN * BK / 8 / 256;
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * (BM + BN) * BK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int Mv = M_dev ? min(*M_dev, M) : M;

  // XCD-aware remap: consecutive hardware block ids land on different XCDs
  // (round robin over 8); give each XCD a contiguous range of logical tiles
  // so tiles that share an operand panel share an L2.
  int bid = blockIdx.x;
  const int nb = gridDim.x;
  if ((nb & 7) == 0) bid = (bid & 7) * (nb >> 3) + (bid >> 3);
  const int tm = bid % n_tm, tn = bid / n_tm;
  const int m0 = tm * BM, n0 = tn * BN;
  if (m0 >= Mv) return;

  bf16_t* As = smem;
  bf16_t* Bs = smem + 2 * BM * BK;

  // This thread's 16-byte chunks: rows row0 + 32 j (j < A_CH / B_CH) of the
  // tile, 8-element column chunk kc; the swizzle depends on row & 7 only, so
  // every chunk of the thread shares it.
  const int row0 = tid >> 3, kc0 = tid & 7;
  const int sw = (kc0 ^ (row0 & 7)) << 3;
  int a_off[A_CH], b_off[B_CH];  // element offsets (< 2^31, checked on the host)
#pragma unroll
  for (int j = 0; j < A_CH; ++j) a_off[j] = min(m0 + row0 + 32 * j, Mv - 1) * K + kc0 * 8;
#pragma unroll
  for (int j = 0; j < B_CH; ++j) b_off[j] = min(n0 + row0 + 32 * j, N - 1) * K + kc0 * 8;
  const int lds0 = row0 * BK + sw;

  const int lr = lane & 31, lg = lane >> 5;
  u32x4 ra[A_CH], rb[B_CH];
  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = K / BK;
#pragma unroll
  for (int j = 0; j < A_CH; ++j) ra[j] = *reinterpret_cast<const u32x4*>(A + a_off[j]);
#pragma unroll
  for (int j = 0; j < B_CH; ++j) rb[j] = *reinterpret_cast<const u32x4*>(Bw + b_off[j]);
#pragma unroll
  for (int j = 0; j < A_CH; ++j) *reinterpret_cast<u32x4*>(As + lds0 + 32 * j * BK) = ra[j];
#pragma unroll
  for (int j = 0; j < B_CH; ++j) *reinterpret_cast<u32x4*>(Bs + lds0 + 32 * j * BK) = rb[j];
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      const int k1 = (kt + 1) * BK;
#pragma unroll
      for (int j = 0; j < A_CH; ++j) ra[j] = *reinterpret_cast<const u32x4*>(A + a_off[j] + k1);
#pragma unroll
      for (int j = 0; j < B_CH; ++j) rb[j] = *reinterpret_cast<const u32x4*>(Bw + b_off[j] + k1);
    }
    const bf16_t* as = As + cur * BM * BK;
    const bf16_t* bs = Bs + cur * BN * BK;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int kc = ks * 2 + lg;
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = wm * WM + i * 32 + lr;
        af[i] = *reinterpret_cast<const bf16x8*>(as + row * BK + ((kc ^ (row & 7)) << 3));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int row = wn * WN + j * 32 + lr;
        bfr[j] = *reinterpret_cast<const bf16x8*>(bs + row * BK + ((kc ^ (row & 7)) << 3));
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      bf16_t* an = As + (cur ^ 1) * BM * BK;
      bf16_t* bn = Bs + (cur ^ 1) * BN * BK;
#pragma unroll
      for (int j = 0; j < A_CH; ++j) *reinterpret_cast<u32x4*>(an + lds0 + 32 * j * BK) = ra[j];
#pragma unroll
      for (int j = 0; j < B_CH; ++j) *reinterpret_cast<u32x4*>(bn + lds0 + 32 * j * BK) = rb[j];
    }
    __syncthreads();
  }

  // ---------------------------------------------------------------- epilogue
  // acc[i][j][r] holds C[row][col] with row = i*32 + (r/4)*8 + lg*4 + r%4 and
  // col = j*32 + lr inside the wave tile.
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
            dst[dlo] = f32_to_bf16(lo * c - hi * s);
            dst[dlo + half] = f32_to_bf16(hi * c + lo * s);
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

template <int BM, int BN>
void launch(hipStream_t st, const bf16_t* A, const bf16_t* B, int M, int N, int K,
            const int* M_dev, EpiKind epi, const EpiArgs& ea) {
  const int n_tm = ceil_div(M, BM), n_tn = ceil_div(N, BN);
  dim3 grid(n_tm * n_tn), block(256);
  switch (epi) {
    case EPI_STORE_F32:
      gemm_bf16_kernel<BM, BN, EPI_STORE_F32><<<grid, block, 0, st>>>(A, B, M, N, K, M_dev, ea, n_tm);
      break;
    case EPI_RESIDUAL:
      gemm_bf16_kernel<BM, BN, EPI_RESIDUAL><<<grid, block, 0, st>>>(A, B, M, N, K, M_dev, ea, n_tm);
      break;
    case EPI_GELU:
      gemm_bf16_kernel<BM, BN, EPI_GELU><<<grid, block, 0, st>>>(A, B, M, N, K, M_dev, ea, n_tm);
      break;
    case EPI_QKV_ROPE:
    case EPI_SWIGLU:
      if constexpr (BN == 256) {
        throw Error(DLMC_E_INVAL, "paired epilogues use BN = 128");
      } else if (epi == EPI_QKV_ROPE) {
        gemm_bf16_kernel<BM, BN, EPI_QKV_ROPE><<<grid, block, 0, st>>>(A, B, M, N, K, M_dev, ea, n_tm);
      } else {
        gemm_bf16_kernel<BM, BN, EPI_SWIGLU><<<grid, block, 0, st>>>(A, B, M, N, K, M_dev, ea, n_tm);
      }
      break;
  }
  DLMC_HIP(hipGetLastError());
}

}  // namespace

void gemm_bf16(hipStream_t st, const bf16_t* A, const bf16_t* B, int M, int N, int K,
               const int* M_dev, EpiKind epi, const EpiArgs& ea) {
  DLMC_CHECK(K % BK == 0 && K > 0, DLMC_E_INVAL, "bf16 GEMM needs K % 64 == 0");
  DLMC_CHECK((int64_t)M * K < (1ll << 31) && (int64_t)N * K < (1ll << 31), DLMC_E_INVAL,
             "GEMM operand too large for 32-bit offsets");
  if (M <= 0 || N <= 0) return;
  const bool paired = (epi == EPI_QKV_ROPE || epi == EPI_SWIGLU);
  // Tile choice: large tiles when there are enough of them to fill 256 CUs.
  const long tiles256 = (long)ceil_div(M, 256) * ceil_div(N, 256);
  // (the paired epilogues keep 2 x 256 accumulators live and spill at 256 x 256)
  if (!paired && N % 256 == 0 && M >= 256 && tiles256 >= 512) {
    launch<256, 256>(st, A, B, M, N, K, M_dev, epi, ea);
  } else if ((!paired || N % 128 == 0) && M >= 128 && (long)ceil_div(M, 256) * ceil_div(N, 128) >= 256) {
    launch<256, 128>(st, A, B, M, N, K, M_dev, epi, ea);
  } else {
    DLMC_CHECK(!paired || N % 128 == 0, DLMC_E_INVAL, "paired epilogue needs N % 128 == 0");
    launch<128, 128>(st, A, B, M, N, K, M_dev, epi, ea);
  }
}

}  // namespace dlmc
