// Shared device/host definitions of the gfx950 kernels (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vidax {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kHeadDim = 128;
// Entries (cos, sin) of the per-workgroup rotary table kept in LDS.
constexpr int kRopeTableMax = 4096;
// The attention kernel's table has one extra identity position per axis and
// packs a token's (t, h, w) into one word (w, h in 11-bit fields, t in 10).
constexpr int kAttnTableMax = 4096;
constexpr int kAttnGridHWMax = 1023;
constexpr int kAttnGridTMax = 1023;

// Rotary parameters in the form the kernels consume (derived from
// vidax_rope3d_desc by the host).
struct RopeParams {
  int enabled;
  int gt, gh, gw;      // token grid
  int dt, dh, dw;      // channel widths of the t, h, w blocks
  int pair_mode;       // 0 interleaved, 1 half split
  int keys_prerotated; // attention: keys arrive already rotated
  int inverse;         // standalone rotation: rotate by -angle (the transpose)
  int n_rot;           // gt * gh * gw
  int base1, base2;    // first table entry of the h and w axes
  int n_entries;       // table entries: gt*dt/2 + gh*dh/2 + gw*dw/2
  float log2_theta;
};

// ---------------------------------------------------------------- device ----

__device__ __forceinline__ float bf16lo_to_f32(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16hi_to_f32(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two fp32 -> packed bf16 pair (lo in bits 0-15), round to nearest even:
// one v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Angle of table entry e: the entries of axis a are laid out [pos][j] with
// d_a/2 entries per position; frequency theta^(-2j/d_a).
__device__ __forceinline__ float2 rope_table_entry(const RopeParams& r, int e) {
  int pos, j, da;
  if (e < r.base1) {
    int half = r.dt >> 1; pos = e / half; j = e - pos * half; da = r.dt;
  } else if (e < r.base2) {
    int half = r.dh >> 1; int f = e - r.base1; pos = f / half; j = f - pos * half; da = r.dh;
  } else {
    int half = r.dw >> 1; int f = e - r.base2; pos = f / half; j = f - pos * half; da = r.dw;
  }
  float omega = exp2f(-((float)(2 * j) / (float)da) * r.log2_theta);
  float s, c;
  sincosf((float)pos * omega, &s, &c);
  return make_float2(c, s);
}

// Table entry of channel pair `pi` (interleaved numbering, pi in [0, 64)) at
// coordinates (t, h, w): base of the pair's axis + pos * (d_a/2) + j.
struct PairSlot {
  int axis;   // 0, 1, 2
  int base;   // base_a + j
  int stride; // d_a / 2
};

__host__ __device__ inline PairSlot pair_slot(const RopeParams& r, int pi) {
  PairSlot s;
  int ht = r.dt >> 1, hh = r.dh >> 1;
  if (pi < ht) {
    s.axis = 0; s.base = pi; s.stride = ht;
  } else if (pi < ht + hh) {
    s.axis = 1; s.base = r.base1 + (pi - ht); s.stride = hh;
  } else {
    s.axis = 2; s.base = r.base2 + (pi - ht - hh); s.stride = r.dw >> 1;
  }
  return s;
}

}  // namespace vidax
