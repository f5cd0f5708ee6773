// Shared device-side types and helpers of the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kNumXcd = 8;       // MI355X: 8 accelerator complex dies, 32 CUs each
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Workgroups are handed to the XCDs round-robin by id.  Remap so that each XCD
// receives one contiguous range of logical ids: neighbouring tiles (same chunk
// and head) then share that XCD's L2.
__device__ __forceinline__ int xcd_remap(int bid, int total) {
  const int xcd = bid % kNumXcd;
  const int idx = bid / kNumXcd;
  const int per = total / kNumXcd;
  const int rem = total % kNumXcd;
  return xcd * per + (xcd < rem ? xcd : rem) + idx;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}

// Round-to-nearest-even fp32 -> bf16 (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  __bf16 b = (__bf16)f;
  return __builtin_bit_cast(uint16_t, b);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Index checks of the checking build (compiled with PD_CHECK_INDICES): a kept
// chunk outside 0..N-1 or a kept slot outside 1..C (slot 0, the BOS row, is
// implied) is replaced by slot 0 of chunk 0 before anything is read, and every
// output that depended on it is written as NaN.  Release builds trust the
// indices, which the selection kernels produce in range.
#ifdef PD_CHECK_INDICES
constexpr bool kCheckIndices = true;
#else
constexpr bool kCheckIndices = false;
#endif
constexpr uint32_t kNanWord = 0x7FC07FC0u;   // a NaN as fp32 and as two bf16
__device__ __forceinline__ bool kept_row_ok(int chunk, int slot, bool bos, int N, int C) {
  return chunk >= 0 && chunk < N && (bos ? slot == 0 : (slot >= 1 && slot <= C));
}

// Monotone map of an fp32 value to uint32 (ascending order preserved; -0 == +0).
__device__ __forceinline__ uint32_t float_order_key(float f) {
  if (f == 0.0f) f = 0.0f;
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace pd
