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

typedef __attribute__((address_space(3))) void lds_void_t;
typedef int i32x4_t __attribute__((ext_vector_type(4)));

// Word 3 of a raw buffer resource on gfx950 (32-bit data format, no
// swizzle); reads past num_records return zero.
constexpr int kBufferFlags = 0x00020000;

// Raw buffer resource (stride 0) over num_bytes at base.
__device__ __forceinline__ i32x4_t buffer_rsrc(const void* base,
                                               int num_bytes) {
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  i32x4_t r;
  r[0] = __builtin_amdgcn_readfirstlane(static_cast<int>(p & 0xffffffffu));
  r[1] = __builtin_amdgcn_readfirstlane(static_cast<int>((p >> 32) & 0xffffu));
  r[2] = num_bytes;
  r[3] = kBufferFlags;
  return r;
}

// 16 bytes per lane from a raw buffer straight into LDS: lane l's data
// lands at LDS byte lds_addr + 16*l (lds_addr is passed in M0).  Issued
// through inline asm so the compiler does not guard every later LDS read
// with a wait for these loads (it cannot tell which slot they write); the
// kernel waits for them explicitly (wait_vmcnt) before the barrier that
// publishes a slot.  NT: the non-temporal hint (a stream read once).
template <bool NT = true>
__device__ __forceinline__ void load_to_lds16(i32x4_t rsrc, int voff,
                                              uint32_t lds_addr) {
  if constexpr (NT)
    asm volatile("buffer_load_dwordx4 %0, %1, 0 offen nt lds"
                 :
                 : "v"(voff), "s"(rsrc), "{m0}"(lds_addr));
  else
    asm volatile("buffer_load_dwordx4 %0, %1, 0 offen lds"
                 :
                 : "v"(voff), "s"(rsrc), "{m0}"(lds_addr));
}

// s_waitcnt with only the vector-memory counter bounded by N.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (((N >> 4) & 3) << 14) | (7 << 4) |
                             (0xF << 8));
}

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
