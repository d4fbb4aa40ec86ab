// Weight init, embedding, normalisation and the fp32 model's GEMM / helpers.
#include "kernels.h"

namespace dlmc {
namespace {

constexpr uint64_t GOLDEN = 0x9E3779B97F4A7C15ull;

// splitmix64 (Steele, Lea, Flood, OOPSLA 2014): one output for state x
__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + GOLDEN;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ int map_row(int r, int map, int dh) {
  if (map == MAP_QK_PAIRS) {
    const int h = r / dh, w = r % dh, half = dh / 2;
    const int p = w < half ? w : w - half;
    const int jb = 2 * (p / 32) + (w < half ? 0 : 1);
    return h * dh + jb * 32 + (p % 32);
  }
  if (map == MAP_GLU_PAIRS) return (r / 32) * 64 + (r % 32);
  return r;
}

// w_i = ((u_i >> 40) - 2^23) * 2^(-23-e), u_i = splitmix64(key + i), i the
// canonical row-major index; written at the mapped row of the device buffer.
__global__ void init_weights_kernel(void* __restrict__ dst, int dtype, uint64_t key, int rows,
                                    int cols, float scale, int map, int row_offset, int dh) {
  const size_t n = (size_t)rows * cols;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x) {
    const int r = (int)(i / cols), c = (int)(i % cols);
    const uint64_t u = splitmix64(key + i);
    const float w = (float)((int)(u >> 40) - (1 << 23)) * scale;  // exact
    const size_t o = (size_t)(map_row(r, map, dh) + row_offset) * cols + c;
    if (dtype == DLMC_DTYPE_BF16)
      ((bf16_t*)dst)[o] = f32_to_bf16(w);
    else
      ((float*)dst)[o] = w;
  }
}

__global__ void embed_kernel(const int32_t* __restrict__ state, const void* __restrict__ table,
                             int dtype, float* __restrict__ x, int d, int max_id) {
  const int row = blockIdx.x;
  const size_t src = (size_t)min(max(state[row], 0), max_id) * d;  // ids outside [0, V] clamp
  float* dst = x + (size_t)row * d;
  if (dtype == DLMC_DTYPE_BF16) {
    const bf16_t* t = (const bf16_t*)table + src;
    for (int c = threadIdx.x; c < d; c += blockDim.x) dst[c] = bf16_to_f32(t[c]);
  } else {
    const float* t = (const float*)table + src;
    for (int c = threadIdx.x; c < d; c += blockDim.x) dst[c] = t[c];
  }
}

// fixed-order sum over a 256-thread block (butterfly inside each wave, then
// the four wave totals in order)
__device__ __forceinline__ float block_sum256(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[wave] = v;
  __syncthreads();
  return ((red[0] + red[1]) + red[2]) + red[3];
}

template <int PER>
__global__ void __launch_bounds__(256)
norm_kernel(const float* __restrict__ x, void* __restrict__ out, int out_dtype, int d,
            int norm_kind, float eps, const int32_t* __restrict__ gather,
            const int32_t* __restrict__ n_dev) {
  __shared__ float red[4];
  const int i = blockIdx.x;
  if (n_dev && i >= *n_dev) return;
  const int src = gather ? gather[i] : i;
  const float* xr = x + (size_t)src * d;
  float v[PER];
  float s = 0.0f;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int c = threadIdx.x + 256 * e;
    v[e] = c < d ? xr[c] : 0.0f;
  }
  float scale, shift = 0.0f;
  if (norm_kind == DLMC_NORM_LAYER) {
#pragma unroll
    for (int e = 0; e < PER; ++e) s += v[e];
    const float mean = block_sum256(s, red) / (float)d;
    float q = 0.0f;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int c = threadIdx.x + 256 * e;
      const float t = c < d ? v[e] - mean : 0.0f;
      q += t * t;
    }
    const float var = block_sum256(q, red) / (float)d;
    scale = 1.0f / sqrtf(var + eps);
    shift = mean;
  } else {
#pragma unroll
    for (int e = 0; e < PER; ++e) s += v[e] * v[e];
    const float ms = block_sum256(s, red) / (float)d;
    scale = 1.0f / sqrtf(ms + eps);
  }
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int c = threadIdx.x + 256 * e;
    if (c >= d) continue;
    const float y = (v[e] - shift) * scale;
    if (out_dtype == DLMC_DTYPE_BF16)
      ((bf16_t*)out)[(size_t)i * d + c] = f32_to_bf16(y);
    else
      ((float*)out)[(size_t)i * d + c] = y;
  }
}

// Same normalisation with 16-byte loads: thread t holds columns 4 (t + 256 e)
// .. + 3 (d % 1024 == 0), and writes them as one 8-byte (bf16) or 16-byte
// store.
template <int PER4>
__global__ void __launch_bounds__(256)
norm4_kernel(const float* __restrict__ x, void* __restrict__ out, int out_dtype, int d,
             int norm_kind, float eps, const int32_t* __restrict__ gather,
             const int32_t* __restrict__ n_dev) {
  __shared__ float red[4];
  const int i = blockIdx.x;
  if (n_dev && i >= *n_dev) return;
  const int src = gather ? gather[i] : i;
  const float4* xr = reinterpret_cast<const float4*>(x + (size_t)src * d);
  float4 v[PER4];
#pragma unroll
  for (int e = 0; e < PER4; ++e) v[e] = xr[threadIdx.x + 256 * e];
  float scale, shift = 0.0f;
  if (norm_kind == DLMC_NORM_LAYER) {
    float s = 0.0f;
#pragma unroll
    for (int e = 0; e < PER4; ++e) s += (v[e].x + v[e].y) + (v[e].z + v[e].w);
    const float mean = block_sum256(s, red) / (float)d;
    float q = 0.0f;
#pragma unroll
    for (int e = 0; e < PER4; ++e) {
      const float a = v[e].x - mean, b = v[e].y - mean, c = v[e].z - mean, w = v[e].w - mean;
      q += (a * a + b * b) + (c * c + w * w);
    }
    const float var = block_sum256(q, red) / (float)d;
    scale = 1.0f / sqrtf(var + eps);
    shift = mean;
  } else {
    float s = 0.0f;
#pragma unroll
    for (int e = 0; e < PER4; ++e)
      s += (v[e].x * v[e].x + v[e].y * v[e].y) + (v[e].z * v[e].z + v[e].w * v[e].w);
    const float ms = block_sum256(s, red) / (float)d;
    scale = 1.0f / sqrtf(ms + eps);
  }
#pragma unroll
  for (int e = 0; e < PER4; ++e) {
    const int c4 = threadIdx.x + 256 * e;
    const float y0 = (v[e].x - shift) * scale, y1 = (v[e].y - shift) * scale;
    const float y2 = (v[e].z - shift) * scale, y3 = (v[e].w - shift) * scale;
    if (out_dtype == DLMC_DTYPE_BF16) {
      u32x2 w;
      w[0] = (uint32_t)f32_to_bf16(y0) | ((uint32_t)f32_to_bf16(y1) << 16);
      w[1] = (uint32_t)f32_to_bf16(y2) | ((uint32_t)f32_to_bf16(y3) << 16);
      reinterpret_cast<u32x2*>((bf16_t*)out + (size_t)i * d)[c4] = w;
    } else {
      reinterpret_cast<float4*>((float*)out + (size_t)i * d)[c4] = make_float4(y0, y1, y2, y3);
    }
  }
}

__global__ void fill_kernel(int32_t* p, int32_t v, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// ---------------------------------------------------------------- fp32 model
// 64 x 64 tile, 16-deep k steps through LDS, 4 x 4 outputs per thread;
// every output is a sequential fmaf chain over k.
template <int EPI>
__global__ void __launch_bounds__(256)
gemm_f32_kernel(const float* __restrict__ A, const float* __restrict__ Bw, int M, int N, int K,
                const int* __restrict__ M_dev, EpiArgs ea) {
  __shared__ float As[16][64 + 4];
  __shared__ float Bs[16][64 + 4];
  const int Mv = M_dev ? min(*M_dev, M) : M;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  if (m0 >= Mv) return;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int lrow = tid >> 2, lk = (tid & 3) * 4;
  const float* ap = A + (size_t)min(m0 + lrow, Mv - 1) * K + lk;
  const float* bp = Bw + (size_t)min(n0 + lrow, N - 1) * K + lk;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(ap + k0);
    const f32x4 b = *reinterpret_cast<const f32x4*>(bp + k0);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      As[lk + e][lrow] = a[e];
      Bs[lk + e][lrow] = b[e];
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        av[e] = As[kk][ty * 4 + e];
        bv[e] = Bs[kk][tx * 4 + e];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= Mv) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx * 4 + j;
      if (col >= N) continue;
      float* o = (float*)ea.out + (size_t)row * ea.ldo + col;
      if constexpr (EPI == EPI_RESIDUAL)
        *o += acc[i][j];
      else
        *o = acc[i][j];
    }
  }
}

// [M, 3d] fp32 QKV (canonical columns) -> rotary Q, K and transposed V
__global__ void qkv_rope_f32_kernel(const float* __restrict__ qkv, int M, EpiArgs ea) {
  const int d = ea.d, dh = ea.dh, half = dh / 2, H = ea.H;
  const size_t n = (size_t)M * H * half;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x) {
    const int p = (int)(i % half);
    const int h = (int)((i / half) % H);
    const int row = (int)(i / ((size_t)half * H));
    const int b = row / ea.T, t = row % ea.T;
    const size_t bh = (size_t)b * H + h;
    const float* src = qkv + (size_t)row * 3 * d + h * dh;
    const float c = ea.rope_cos[t * half + p], s = ea.rope_sin[t * half + p];
    for (int w = 0; w < 2; ++w) {
      const float lo = src[w * d + p], hi = src[w * d + p + half];
      float* dst = (float*)(w == 0 ? ea.q : ea.k) + (bh * ea.Tp + t) * dh;
      dst[p] = lo * c - hi * s;
      dst[p + half] = hi * c + lo * s;
    }
    float* vt = (float*)ea.vt + bh * dh * ea.Tp + t;
    vt[(size_t)p * ea.Tp] = src[2 * d + p];
    vt[(size_t)(p + half) * ea.Tp] = src[2 * d + p + half];
  }
}

__global__ void ffn_act_f32_kernel(const float* __restrict__ in, float* __restrict__ out, int M,
                                   int F, int kind) {
  const size_t n = (size_t)M * F;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x) {
    const int row = (int)(i / F), f = (int)(i % F);
    if (kind == DLMC_FFN_GELU) {
      const float v = in[i];
      out[i] = 0.5f * v * (1.0f + erff(v * 0.70710678118654752440f));
    } else {
      const float g = in[(size_t)row * 2 * F + f], u = in[(size_t)row * 2 * F + F + f];
      out[i] = g / (1.0f + expf(-g)) * u;
    }
  }
}

inline int grid_for(size_t n, int block) {
  return (int)std::min<size_t>((n + block - 1) / block, 65536);
}

uint64_t splitmix64_host(uint64_t x) {
  uint64_t z = x + GOLDEN;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

}  // namespace

void init_weights(hipStream_t st, void* dst, int dtype, uint64_t seed, int tensor_id, int rows,
                  int cols, int exp, RowMap map, int row_offset, int dh) {
  const uint64_t key = splitmix64_host(seed ^ ((uint64_t)tensor_id * GOLDEN));
  const float scale = ldexpf(1.0f, -23 - exp);
  const size_t n = (size_t)rows * cols;
  init_weights_kernel<<<grid_for(n, 256), 256, 0, st>>>(dst, dtype, key, rows, cols, scale,
                                                         (int)map, row_offset, dh);
  DLMC_HIP(hipGetLastError());
}

// One row per wave (d == 256 PER4): lane l holds columns 4 (l + 64 e) .. + 3
// as 16-byte loads; the row sums are fixed-order butterflies over the wave
// (every lane ends with the same bits), so no block barrier is needed.
template <int PER4>
__global__ void __launch_bounds__(256)
norm_wave_kernel(const float* __restrict__ x, void* __restrict__ out, int out_dtype, int n_rows,
                 int norm_kind, float eps, const int32_t* __restrict__ gather,
                 const int32_t* __restrict__ n_dev) {
  constexpr int d = 256 * PER4;
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= n_rows || (n_dev && i >= *n_dev)) return;
  const int src = gather ? gather[i] : i;
  const float4* xr = reinterpret_cast<const float4*>(x + (size_t)src * d);
  float4 v[PER4];
#pragma unroll
  for (int e = 0; e < PER4; ++e) v[e] = xr[lane + 64 * e];
  auto wave_sum = [](float t) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) t += __shfl_xor(t, o);
    return t;
  };
  float scale, shift = 0.0f;
  if (norm_kind == DLMC_NORM_LAYER) {
    float s = 0.0f;
#pragma unroll
    for (int e = 0; e < PER4; ++e) s += (v[e].x + v[e].y) + (v[e].z + v[e].w);
    const float mean = wave_sum(s) / (float)d;
    float q = 0.0f;
#pragma unroll
    for (int e = 0; e < PER4; ++e) {
      const float a = v[e].x - mean, b = v[e].y - mean, c = v[e].z - mean, w = v[e].w - mean;
      q += (a * a + b * b) + (c * c + w * w);
    }
    const float var = wave_sum(q) / (float)d;
    scale = 1.0f / sqrtf(var + eps);
    shift = mean;
  } else {
    float s = 0.0f;
#pragma unroll
    for (int e = 0; e < PER4; ++e)
      s += (v[e].x * v[e].x + v[e].y * v[e].y) + (v[e].z * v[e].z + v[e].w * v[e].w);
    const float ms = wave_sum(s) / (float)d;
    scale = 1.0f / sqrtf(ms + eps);
  }
#pragma unroll
  for (int e = 0; e < PER4; ++e) {
    const int c4 = lane + 64 * e;
    const float y0 = (v[e].x - shift) * scale, y1 = (v[e].y - shift) * scale;
    const float y2 = (v[e].z - shift) * scale, y3 = (v[e].w - shift) * scale;
    if (out_dtype == DLMC_DTYPE_BF16) {
      u32x2 w;
      w[0] = (uint32_t)f32_to_bf16(y0) | ((uint32_t)f32_to_bf16(y1) << 16);
      w[1] = (uint32_t)f32_to_bf16(y2) | ((uint32_t)f32_to_bf16(y3) << 16);
      reinterpret_cast<u32x2*>((bf16_t*)out + (size_t)i * d)[c4] = w;
    } else {
      reinterpret_cast<float4*>((float*)out + (size_t)i * d)[c4] = make_float4(y0, y1, y2, y3);
    }
  }
}

// one block per selection slot: 16-byte chunks of the source row, or zeros
// for a slot past its chunk's committed count
__global__ void __launch_bounds__(256)
gather_slot_rows_kernel(const bf16_t* __restrict__ src, const float* __restrict__ mx,
                        const int32_t* __restrict__ sel_row, const int32_t* __restrict__ n_sel,
                        int m_max, int d, bf16_t* __restrict__ dst, float* __restrict__ dst_mx) {
  const int slot = blockIdx.x, b = slot / m_max, j = slot % m_max;
  const bool live = j < n_sel[b];
  if (threadIdx.x == 0) dst_mx[slot] = live ? mx[sel_row[slot]] : 0.0f;
  const u32x4* s = reinterpret_cast<const u32x4*>(src + (live ? (size_t)sel_row[slot] * d : 0));
  u32x4* o = reinterpret_cast<u32x4*>(dst + (size_t)slot * d);
  for (int c = threadIdx.x; c < d / 8; c += blockDim.x) o[c] = live ? s[c] : u32x4{0u, 0u, 0u, 0u};
}

void embed(hipStream_t st, const int32_t* state, const void* table, int dtype, float* x,
           int n_rows, int d, int max_id) {
  if (n_rows <= 0) return;
  embed_kernel<<<n_rows, 256, 0, st>>>(state, table, dtype, x, d, max_id);
  DLMC_HIP(hipGetLastError());
}

void norm_rows(hipStream_t st, const float* x, void* out, int out_dtype, int n_rows, int d,
               int norm_kind, float eps, const int32_t* gather_rows, const int32_t* n_dev) {
  if (n_rows <= 0) return;
  const int per = ceil_div(d, 256);
  dim3 grid(n_rows), block(256);
  if (d % 256 == 0 && d <= 2048) {
    const dim3 wgrid(ceil_div(n_rows, 4));
#define DLMC_NORMW(P)                                                                   \
  norm_wave_kernel<P><<<wgrid, block, 0, st>>>(x, out, out_dtype, n_rows, norm_kind, eps, \
                                               gather_rows, n_dev)
    switch (d / 256) {
      case 1: DLMC_NORMW(1); break;
      case 2: DLMC_NORMW(2); break;
      case 3: DLMC_NORMW(3); break;
      case 4: DLMC_NORMW(4); break;
      case 5: DLMC_NORMW(5); break;
      case 6: DLMC_NORMW(6); break;
      case 7: DLMC_NORMW(7); break;
      default: DLMC_NORMW(8); break;
    }
#undef DLMC_NORMW
    DLMC_HIP(hipGetLastError());
    return;
  }
  if (d % 1024 == 0 && d <= 8192) {
#define DLMC_NORM4(P)                                                                           \
  norm4_kernel<P><<<grid, block, 0, st>>>(x, out, out_dtype, d, norm_kind, eps, gather_rows, \
                                          n_dev)
    switch (d / 1024) {
      case 1: DLMC_NORM4(1); break;
      case 2: DLMC_NORM4(2); break;
      case 3: DLMC_NORM4(3); break;
      case 4: DLMC_NORM4(4); break;
      case 5: DLMC_NORM4(5); break;
      case 6: DLMC_NORM4(6); break;
      case 7: DLMC_NORM4(7); break;
      default: DLMC_NORM4(8); break;
    }
#undef DLMC_NORM4
    DLMC_HIP(hipGetLastError());
    return;
  }
#define DLMC_NORM(P)                                                                           \
  norm_kernel<P><<<grid, block, 0, st>>>(x, out, out_dtype, d, norm_kind, eps, gather_rows, \
                                         n_dev)
  if (per <= 1) DLMC_NORM(1);
  else if (per <= 2) DLMC_NORM(2);
  else if (per <= 4) DLMC_NORM(4);
  else if (per <= 8) DLMC_NORM(8);
  else if (per <= 16) DLMC_NORM(16);
  else if (per <= 32) DLMC_NORM(32);
  else throw Error(DLMC_E_INVAL, "d_model above 8192 is not supported");
#undef DLMC_NORM
  DLMC_HIP(hipGetLastError());
}

void gather_slot_rows(hipStream_t st, const bf16_t* src, const float* mx, const int32_t* sel_row,
                      const int32_t* n_sel, int B, int m_max, int d, bf16_t* dst, float* dst_mx) {
  DLMC_CHECK(d % 8 == 0, DLMC_E_INVAL, "row gather needs d % 8 == 0");
  if (B <= 0 || m_max <= 0) return;
  gather_slot_rows_kernel<<<B * m_max, 256, 0, st>>>(src, mx, sel_row, n_sel, m_max, d, dst, dst_mx);
  DLMC_HIP(hipGetLastError());
}

void fill_i32(hipStream_t st, int32_t* p, int32_t v, size_t n) {
  if (n == 0) return;
  fill_kernel<<<grid_for(n, 256), 256, 0, st>>>(p, v, n);
  DLMC_HIP(hipGetLastError());
}

void gemm_f32(hipStream_t st, const float* A, const float* B, int M, int N, int K,
              const int* M_dev, EpiKind epi, const EpiArgs& ea) {
  DLMC_CHECK(K % 16 == 0 && K > 0, DLMC_E_INVAL, "fp32 GEMM needs K % 16 == 0");
  if (M <= 0 || N <= 0) return;
  dim3 grid(ceil_div(N, 64), ceil_div(M, 64)), block(256);
  if (epi == EPI_RESIDUAL)
    gemm_f32_kernel<EPI_RESIDUAL><<<grid, block, 0, st>>>(A, B, M, N, K, M_dev, ea);
  else if (epi == EPI_STORE_F32)
    gemm_f32_kernel<EPI_STORE_F32><<<grid, block, 0, st>>>(A, B, M, N, K, M_dev, ea);
  else
    throw Error(DLMC_E_INVAL, "fp32 GEMM epilogue must be store or residual");
  DLMC_HIP(hipGetLastError());
}

void qkv_rope_f32(hipStream_t st, const float* qkv, int M, const EpiArgs& ea) {
  const size_t n = (size_t)M * ea.H * (ea.dh / 2);
  if (n == 0) return;
  qkv_rope_f32_kernel<<<grid_for(n, 256), 256, 0, st>>>(qkv, M, ea);
  DLMC_HIP(hipGetLastError());
}

void ffn_act_f32(hipStream_t st, const float* in, float* out, int M, int F, int kind) {
  const size_t n = (size_t)M * F;
  if (n == 0) return;
  ffn_act_f32_kernel<<<grid_for(n, 256), 256, 0, st>>>(in, out, M, F, kind);
  DLMC_HIP(hipGetLastError());
}

}  // namespace dlmc
