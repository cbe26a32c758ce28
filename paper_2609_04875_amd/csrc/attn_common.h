// Vector types and lane helpers shared by the bf16 MFMA attention kernels
// (prefill and decode) on gfx950.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace pgsr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ constexpr bf16x2 kOnes = {(__bf16)1.0f, (__bf16)1.0f};

// Value of the lane 32 apart (same query row, other half of the wave):
// v_permlane32_swap exchanges the upper half of its first operand with the
// lower half of its second, so with both operands = x the low lanes find the
// partner's x in the second result and the high lanes in the first.
__device__ inline float xor32(float x) {
  const int xi = __builtin_bit_cast(int, x);
  const auto r = __builtin_amdgcn_permlane32_swap(xi, xi, false, false);
  return __builtin_bit_cast(float, (threadIdx.x & 32) ? r[0] : r[1]);
}

// Zero 16-bit elements e (0..7) of a 16-byte chunk for which pos0 + e >= limit.
__device__ inline u32x4 zero_tail(u32x4 v, int pos0, int limit) {
  const int keep = limit - pos0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const int e0 = 2 * w;
    uint32_t m = 0;
    if (e0 < keep) m |= 0x0000FFFFu;
    if (e0 + 1 < keep) m |= 0xFFFF0000u;
    v[w] &= m;
  }
  return v;
}

// Eight E4M3 codes (byte e = element e) as eight bf16 values, exactly (a
// code has at most 4 significant bits and an exponent inside bf16's range):
// the scaled pair conversion with scale 1 widens two codes per instruction
// (bytes 0-1 or 2-3 of a word).  On all 65536 pairs of codes it gives the
// bits of the fp32 pair conversion's upper halves, NaNs included.
__device__ inline u32x4 widen_fp8(u32x2 w) {
  u32x4 r;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    r[2 * h] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[h], 1.0f, false));
    r[2 * h + 1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[h], 1.0f, true));
  }
  return r;
}

}  // namespace
}  // namespace pgsr
