// Shared host/device definitions of libdlmc (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <stdexcept>
#include <string>

#include "../../include/dlmc.h"

namespace dlmc {

typedef uint16_t bf16_t;  // bf16 bit pattern in memory

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// An error carrying a dlmc_status across internal C++ code; converted to a
// status code at the ABI boundary.
struct Error : std::runtime_error {
  dlmc_status code;
  Error(dlmc_status c, const std::string& m) : std::runtime_error(m), code(c) {}
};

#define DLMC_HIP(expr)                                                                   \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess)                                                                \
      throw ::dlmc::Error(DLMC_E_DEVICE, std::string(#expr ": ") + hipGetErrorString(e_)); \
  } while (0)

#define DLMC_CHECK(cond, code, msg)                  \
  do {                                               \
    if (!(cond)) throw ::dlmc::Error((code), (msg)); \
  } while (0)

__host__ __device__ inline float bf16_to_f32(bf16_t b) {
  return __builtin_bit_cast(float, (uint32_t)b << 16);
}
// round to nearest even (inputs here are never NaN)
__host__ __device__ inline bf16_t f32_to_bf16(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

constexpr int ceil_div(int a, int b) { return (a + b - 1) / b; }
constexpr int round_up(int a, int b) { return ceil_div(a, b) * b; }

}  // namespace dlmc
