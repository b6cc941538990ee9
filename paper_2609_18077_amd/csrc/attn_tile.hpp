// Device helpers shared by the attention forward kernels (dense and short-key
// forms): matrix instruction, lane-half reductions, the transposing LDS read,
// the query/output staging layout and waitcnt immediates.
#pragma once

#include "common.hpp"

namespace vidax {
namespace tile {

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr;

constexpr int kBufferFlags = 0x00020000;                  // raw buffer, 32-bit data format
constexpr float kSumLimit = 18446744073709551616.0f;      // 2^64
constexpr uint32_t kOnesBf16x2 = 0x3f803f80u;             // bf16 (1, 1)

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// lanes l and l ^ 32 hold the same query: combine their partial max / sum
__device__ __forceinline__ float wave_half_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float wave_half_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// gfx950 transposing LDS read: 4 consecutive 16-bit rows of one column per lane
__device__ __forceinline__ i16x4 lds_read_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
}

// c + a.lo * b.lo + a.hi * b.hi on packed bf16 pairs, fp32 accumulate
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

// Slot of 16-byte chunk c of staging row r (an involution in c).  For any 16
// consecutive rows and one chunk, and for any 4 rows x 4 chunks aligned by 4,
// the slots are distinct, so the staging accesses are free of bank conflicts.
__device__ __forceinline__ int stage_slot(int c, int r) {
  const int x = r & 15;
  return c ^ (((x & 3) << 2) | (x >> 2));
}

// s_waitcnt immediates (gfx9 encoding): at most n vector memory operations
// outstanding (expcnt and lgkmcnt not waited for); all LDS/scalar operations
// done (vector memory not waited for).
constexpr int wait_vm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }
constexpr int kWaitLgkm0 = 0xc07f;

}  // namespace tile
}  // namespace vidax
