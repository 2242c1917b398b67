// Device helpers shared by the HIP kernels of libpagedweight.so (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

#include "pw.h"

namespace pw {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// 16-bit float helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf16_val(uint32_t h) { return __uint_as_float(h << 16); }
__device__ __forceinline__ float f16_val(uint32_t h) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(h)));
}
__device__ __forceinline__ float val16(uint32_t h, int fmt) {
  return fmt == PW_BF16 ? bf16_val(h & 0xFFFFu) : f16_val(h & 0xFFFFu);
}
// round to nearest even (finite inputs)
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ uint32_t f16_rne(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f));
}
__device__ __forceinline__ uint32_t rne16(float f, int fmt) {
  return fmt == PW_BF16 ? bf16_rne(f) : f16_rne(f);
}

// Directed rounding of an fp32 value to bf16: truncation moves toward zero,
// so it rounds down for positive inputs and up for negative ones.
__device__ __forceinline__ uint32_t bf16_down(float x) {
  if (x == 0.0f) return 0u;
  const uint32_t u = __float_as_uint(x), t = u >> 16;
  if ((u & 0xFFFFu) == 0u) return t;
  return (u >> 31) ? t + 1u : t;
}
__device__ __forceinline__ uint32_t bf16_up(float x) {
  if (x == 0.0f) return 0u;
  const uint32_t u = __float_as_uint(x), t = u >> 16;
  if ((u & 0xFFFFu) == 0u) return t;
  const uint32_t r = (u >> 31) ? t : t + 1u;
  return r == 0x8000u ? 0u : r;
}
// fp16: convert to nearest, then step one ulp if it landed on the wrong side.
__device__ __forceinline__ uint32_t f16_step(uint32_t h, bool up) {
  if ((h & 0x7FFFu) == 0u) return up ? 0x0001u : 0x8001u;
  const bool neg = (h >> 15) != 0;
  return (neg != up) ? h + 1u : h - 1u;
}
__device__ __forceinline__ uint32_t f16_down(float x) {
  if (x == 0.0f) return 0u;
  uint32_t h = f16_rne(x);
  if (f16_val(h) > x) h = f16_step(h, false);
  return (h & 0x7FFFu) == 0u ? 0u : h;
}
__device__ __forceinline__ uint32_t f16_up(float x) {
  if (x == 0.0f) return 0u;
  uint32_t h = f16_rne(x);
  if (f16_val(h) < x) h = f16_step(h, true);
  return (h & 0x7FFFu) == 0u ? 0u : h;
}
__device__ __forceinline__ uint32_t round_down16(float x, int fmt) {
  return fmt == PW_BF16 ? bf16_down(x) : f16_down(x);
}
__device__ __forceinline__ uint32_t round_up16(float x, int fmt) {
  return fmt == PW_BF16 ? bf16_up(x) : f16_up(x);
}

__device__ __forceinline__ int lane_id() {
  return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

template <int ACT>
__device__ __forceinline__ f32x4 mma(u32x4 a, u32x4 b, f32x4 c) {
  if constexpr (ACT == PW_BF16)
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

template <int ACT>
__device__ __forceinline__ u32x4 ones_op() {
  const uint32_t one = ACT == PW_BF16 ? 0x3F803F80u : 0x3C003C00u;
  return u32x4{one, one, one, one};
}

__device__ __forceinline__ u32x4 ld16(const uint8_t* p) { return *reinterpret_cast<const u32x4*>(p); }
// Weights are streamed once: nontemporal loads.
__device__ __forceinline__ u32x4 ld16_nt(const uint8_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

// Bytes of one 16-row x 128-value tile of a page at `B` bits.
template <int B> constexpr int tile_bytes() { return B == 16 ? 4096 : B == 8 ? 2048 : 1024; }

}  // namespace
}  // namespace pw
