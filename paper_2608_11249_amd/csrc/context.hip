// Attention-based initial context (Initial Context Strategies, item 4):
// head-averaged attention maps of the extra forward passes and the Attention
// Rollout (Abnar and Zuidema, 2020) flow into the masked positions.
//
// softmax_accumulate: A[i, :] (+)= w * softmax(scale * S[i, :T]) for one head;
//   heads are added in a fixed order by successive launches.
// rollout_step: out = (A^T v + v) / 2, i.e. v^T (A + I) / 2, one output per
//   thread summing i in ascending order.
#include "kernels.h"

namespace dlmc {
namespace {

constexpr int SB = 256;

__device__ __forceinline__ float block_reduce(float x, float* lds, bool is_max) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float y = __shfl_xor(x, o);
    x = is_max ? fmaxf(x, y) : x + y;
  }
  if (lane == 0) lds[wave] = x;
  __syncthreads();
  float r = lds[0];
  for (int w = 1; w < SB / 64; ++w) r = is_max ? fmaxf(r, lds[w]) : r + lds[w];
  __syncthreads();
  return r;
}

__global__ void __launch_bounds__(SB)
softmax_accumulate_kernel(const float* __restrict__ S, float* __restrict__ A, int T, float scale,
                          float w, int first) {
  __shared__ float lds[SB / 64];
  const size_t i = blockIdx.x;
  const float* s = S + i * T;
  float* a = A + i * T;
  float m = -INFINITY;
  for (int j = threadIdx.x; j < T; j += SB) m = fmaxf(m, s[j]);
  m = block_reduce(m, lds, true);
  float z = 0.0f;
  for (int j = threadIdx.x; j < T; j += SB) z += expf((s[j] - m) * scale);
  z = block_reduce(z, lds, false);
  const float k = w / z;
  for (int j = threadIdx.x; j < T; j += SB) {
    const float p = expf((s[j] - m) * scale) * k;
    a[j] = first ? p : a[j] + p;
  }
}

__global__ void __launch_bounds__(SB)
rollout_step_kernel(const float* __restrict__ A, const float* __restrict__ v, float* __restrict__ out,
                    int T) {
  const int j = blockIdx.x * SB + threadIdx.x;
  if (j >= T) return;
  float acc = 0.0f;
  for (int i = 0; i < T; ++i) acc += v[i] * A[(size_t)i * T + j];
  out[j] = 0.5f * acc + 0.5f * v[j];
}

}  // namespace

void softmax_accumulate(hipStream_t st, const float* S, float* A, int T, float scale, float w,
                        bool first) {
  if (T <= 0) return;
  softmax_accumulate_kernel<<<T, SB, 0, st>>>(S, A, T, scale, w, first ? 1 : 0);
  DLMC_HIP(hipGetLastError());
}

void rollout_step(hipStream_t st, const float* A, const float* v, float* out, int T) {
  if (T <= 0) return;
  rollout_step_kernel<<<ceil_div(T, SB), SB, 0, st>>>(A, v, out, T);
  DLMC_HIP(hipGetLastError());
}

}  // namespace dlmc
