// Shared device helpers for the WeDLM decode-step kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wedlm.h"

#define WEDLM_VERSION_NUMBER 100  // 0.1.0

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float floatx16_t __attribute__((ext_vector_type(16)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8_t __attribute__((ext_vector_type(8)));
typedef uint16_t u16x4_t __attribute__((ext_vector_type(4)));

namespace wedlm {

constexpr int kWave = 64;
constexpr int kPage = WEDLM_PAGE_SIZE;
constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ uint64_t ballot(bool p) {
  return __ballot(p);
}

// Lane index within the wave.
__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// Element (t, k) of an activation matrix with K columns (a multiple of 64)
// in the packed MFMA tile layout of the projections: tile (t/32, k/64) at
// 2048 * (t/32 * K/64 + k/64), then MFMA j = k%32 / 8 (512 elements each),
// lane t%32 + 32 * (k%64 / 32), element k%8.  Eight consecutive k from a
// multiple of 8 are 16 contiguous bytes.
__device__ __forceinline__ int64_t packed_off(int64_t t, int k, int K) {
  return ((t / 32 * (K / 64) + k / 64) * 4 + (k & 31) / 8) * 512 +
         ((t & 31) + 32 * ((k & 63) / 32)) * 8 + (k & 7);
}

}  // namespace wedlm

// Host-side launch check.
#define WEDLM_LAUNCH_CHECK()                      \
  do {                                            \
    if (hipGetLastError() != hipSuccess)          \
      return WEDLM_E_LAUNCH;                      \
  } while (0)
