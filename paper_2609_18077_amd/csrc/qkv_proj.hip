// Q/K/V projection of a video DiT attention block with the Q/K prologue in
// its epilogue, for gfx950: y = x W^T + bias (bf16 operands, fp32
// accumulation), split into the q, k and v heads; every q and k head of every
// token is RMS-normalised over its 128 channels, multiplied by a per-channel
// gain and rotated by the 3D rotary embedding, then all three are rounded to
// bf16 once and written as [B, L, H, 128].  (Section 2, "3D RoPE, 3D VAEs,
// and flash attention", and Section 3, "Supported Models", for the models
// whose attention inputs these are.)
//
// The product is computed transposed, y^T = W x^T, so that a lane holds one
// token and its registers hold output channels (the accumulator layout of
// v_mfma_f32_32x32x16_bf16: lane = column, registers = rows): the per-head
// sum of squares is then a register sum plus one swap between the lane
// halves, and the two channels of a rotary pair sit in neighbouring
// registers of the same lane.
//
// Workgroup: 8 waves, 256 output channels (two heads) x 256 tokens; wave
// (i, j) owns head i of the two (128 channels, 4 blocks of 32) for tokens
// 64 j .. 64 j + 63 (2 blocks of 32): 8 accumulators.  The reduction over
// the C input channels runs in stages of 64: each stage copies the W and x
// tiles (256 rows x 64 channels each, 32 KB) straight from global memory into
// LDS in MFMA operand order, double buffered, one barrier per stage; per
// stage a wave issues 32 matrix instructions.  After the last stage the LDS
// holds the rotary (cos, sin) table for the epilogue.
#include "launch.hpp"

namespace vidax {
namespace {

constexpr int D = kHeadDim;
constexpr int NW = 8, NT = NW * 64;
constexpr int BNC = 256;  // output channels per workgroup
constexpr int BMT = 256;  // tokens per workgroup
constexpr int BK = 64;    // input channels per stage
constexpr int TILE = 256 * BK;  // elements of one staged tile
constexpr int BLK = 512;        // elements per operand block (1 KB)
constexpr int kBufferFlags = 0x00020000;  // raw buffer, 32-bit data format

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr;

struct QkvArgs {
  const uint16_t* x;   // [M, C]
  const uint16_t* w;   // [N, C], N = 3 H 128
  const float* bias;   // [N] or null
  const float* gain_q; // [128] or null
  const float* gain_k; // [128] or null
  uint16_t* out[3];    // q, k, v: [M, H 128]
  float eps;
  int M, C, N, H, L;
  int ntn, ntm;        // workgroup tiles along channels and tokens
  int nwg;
  RopeParams rp;
};

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float half_swap_sum(float x) {
  // lanes l and l ^ 32 hold the same token
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__global__ __launch_bounds__(NT) void qkv_proj_kernel(QkvArgs a) {
  // tile layout (K order, as the attention kernel's keys): block 8 st + rb
  // holds, for lane l, the 16 bytes of row 32 rb + (l & 31), input channels
  // 16 st + 8 (l >> 5) .. + 7 of the stage
  __shared__ __attribute__((aligned(16))) uint16_t W0[TILE], W1[TILE], X0[TILE], X1[TILE];
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int lid;
  {  // workgroups go round-robin over the 8 XCDs: contiguous ranges per XCD
    const int i = blockIdx.x, n = a.nwg;
    const int per = n >> 3, rem = n & 7, xcd = i & 7, kk = i >> 3;
    lid = xcd < rem ? xcd * (per + 1) + kk : rem * (per + 1) + (xcd - rem) * per + kk;
  }
  // Groups of GM token tiles, token tiles fastest inside a group: the 32
  // workgroups an XCD runs at a time then cover 8 token tiles x 4 channel
  // tiles, whose weight rows (4 x 768 KB at C = 1536) stay in that XCD's L2.
  constexpr int GM = 8;
  const int g = lid / (GM * a.ntn), r = lid - g * GM * a.ntn;
  const int gm = min(GM, a.ntm - g * GM);
  const int tn = r / gm, tm = g * GM + (r - (r / gm) * gm);
  const int n0 = tn * BNC, m0 = tm * BMT;
  const int wh = wave & 1, wt = wave >> 1;  // the wave's head (of two) and token group

  const int rows_w = min(BNC, a.N - n0), rows_x = min(BMT, a.M - m0);
  const int cbytes = a.C * 2;
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.w + (size_t)n0 * a.C), (short)0, rows_w * cbytes, kBufferFlags);
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.x + (size_t)m0 * a.C), (short)0, rows_x * cbytes, kBufferFlags);
  // staging: wave w copies blocks 4 w .. 4 w + 3 of each tile
  int goff[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int b = 4 * wave + u, st = b >> 3, rb = b & 7;
    goff[u] = (32 * rb + l32) * cbytes + (16 * st + 8 * hi) * 2;
  }
  auto stage = [&](int s, uint16_t* wb, uint16_t* xb) __attribute__((always_inline)) {
    const int koff = s * BK * 2;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int b = 4 * wave + u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr)(wb + b * BLK), 16, goff[u] + koff, 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_ptr)(xb + b * BLK), 16, goff[u] + koff, 0, 0, 0);
    }
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int cb = 0; cb < 4; ++cb) acc[cb][0] = acc[cb][1] = f32x16{};
  // one stage: 4 k-steps x (4 channel blocks x 2 token blocks)
  auto compute = [&](const uint16_t* wb, const uint16_t* xb) __attribute__((always_inline)) {
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      bf16x8 av[4], bv[2];
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
        av[cb] = *reinterpret_cast<const bf16x8*>(wb + (8 * st + 4 * wh + cb) * BLK + lane * 8);
#pragma unroll
      for (int tb = 0; tb < 2; ++tb)
        bv[tb] = *reinterpret_cast<const bf16x8*>(xb + (8 * st + 2 * wt + tb) * BLK + lane * 8);
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int tb = 0; tb < 2; ++tb) acc[cb][tb] = mfma32(av[cb], bv[tb], acc[cb][tb]);
    }
  };

  const int ns = a.C / BK;
  stage(0, W0, X0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  int s = 0;
  for (; s + 1 < ns; s += 2) {
    stage(s + 1, W1, X1);
    compute(W0, X0);
    __builtin_amdgcn_s_waitcnt(0);  // this wave's copies have landed
    __syncthreads();
    if (s + 2 < ns) stage(s + 2, W0, X0);
    compute(W1, X1);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  if (s < ns) {
    compute(W0, X0);
    __syncthreads();
  }

  // ---- epilogue.  Register i of acc[cb][tb] holds channel 32 cb + 8 (i >> 2)
  // + 4 hi + (i & 3) of the wave's head, token m0 + 64 wt + 32 tb + l32.
  const RopeParams& rp = a.rp;
  float2* tab = reinterpret_cast<float2*>(W0);  // the stage buffers are free now (32 KB)
  if (rp.enabled) {
    for (int e = tid; e < rp.n_entries; e += NT) tab[e] = rope_table_entry(rp, e);
    __syncthreads();
  }
  const int hg = n0 / D + wh;        // global head index over q, k, v
  if (hg >= 3 * a.H) return;         // uniform: past the last head (no barrier follows)
  const int part = hg / a.H, head = hg - part * a.H;
  uint16_t* outp = a.out[part];
  const int chan0 = hg * D;          // first row of this head in W

  const float* gain = part == 0 ? a.gain_q : a.gain_k;

#pragma unroll
  for (int tb = 0; tb < 2; ++tb) {
    const int m = m0 + 64 * wt + 32 * tb + l32;
    // bias (4 consecutive channels per (cb, g), one 16-byte load)
    if (a.bias) {
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const float4 bb = *reinterpret_cast<const float4*>(a.bias + chan0 + 32 * cb + 8 * g + 4 * hi);
          acc[cb][tb][4 * g + 0] += bb.x;
          acc[cb][tb][4 * g + 1] += bb.y;
          acc[cb][tb][4 * g + 2] += bb.z;
          acc[cb][tb][4 * g + 3] += bb.w;
        }
    }
    if (part < 2) {
      float ss = 0.f;
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int i = 0; i < 16; ++i) ss = fmaf(acc[cb][tb][i], acc[cb][tb][i], ss);
      ss = half_swap_sum(ss);
      const float r = __builtin_amdgcn_rsqf(ss * (1.0f / D) + a.eps);
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float4 gg = make_float4(r, r, r, r);
          if (gain) {
            gg = *reinterpret_cast<const float4*>(gain + 32 * cb + 8 * g + 4 * hi);
            gg.x *= r; gg.y *= r; gg.z *= r; gg.w *= r;
          }
          acc[cb][tb][4 * g + 0] *= gg.x;
          acc[cb][tb][4 * g + 1] *= gg.y;
          acc[cb][tb][4 * g + 2] *= gg.z;
          acc[cb][tb][4 * g + 3] *= gg.w;
        }
      const int n = m % a.L;  // position in the sequence
      if (rp.enabled && n < rp.n_rot) {
        const int t = n / (rp.gh * rp.gw);
        const int rr = n - t * rp.gh * rp.gw;
        const int hh = rr / rp.gw;
        const int ww = rr - hh * rp.gw;
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
#pragma unroll
          for (int i = 0; i < 16; i += 2) {
            const int c = 32 * cb + 8 * (i >> 2) + 4 * hi + (i & 3);  // even: pair c / 2
            const PairSlot sl = pair_slot(rp, c >> 1);
            const int pos = sl.axis == 0 ? t : (sl.axis == 1 ? hh : ww);
            const float2 e = tab[sl.base + pos * sl.stride];
            const float x0 = acc[cb][tb][i], x1 = acc[cb][tb][i + 1];
            acc[cb][tb][i] = fmaf(x0, e.x, -x1 * e.y);
            acc[cb][tb][i + 1] = fmaf(x0, e.y, x1 * e.x);
          }
      }
    }
    if (m < a.M) {
      uint16_t* op = outp + (size_t)m * a.H * D + (size_t)head * D;
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          uint2 pk;
          pk.x = pack_bf16x2(acc[cb][tb][4 * g + 0], acc[cb][tb][4 * g + 1]);
          pk.y = pack_bf16x2(acc[cb][tb][4 * g + 2], acc[cb][tb][4 * g + 3]);
          *reinterpret_cast<uint2*>(op + 32 * cb + 8 * g + 4 * hi) = pk;
        }
    }
  }
}

}  // namespace

hipError_t launch_qkv_proj(const uint16_t* x, const uint16_t* w, const float* bias, const float* gain_q,
                           const float* gain_k, float eps, uint16_t* q, uint16_t* k, uint16_t* v, int B, int L, int H,
                           int C, const RopeParams& rp, hipStream_t stream) {
  QkvArgs a;
  a.x = x; a.w = w; a.bias = bias; a.gain_q = gain_q; a.gain_k = gain_k;
  a.out[0] = q; a.out[1] = k; a.out[2] = v;
  a.eps = eps;
  a.M = B * L; a.C = C; a.N = 3 * H * D; a.H = H; a.L = L;
  a.ntn = (a.N + BNC - 1) / BNC;
  a.ntm = (a.M + BMT - 1) / BMT;
  a.nwg = a.ntn * a.ntm;
  a.rp = rp;
  hipLaunchKernelGGL(qkv_proj_kernel, dim3((unsigned)a.nwg), dim3(NT), 0, stream, a);
  return hipGetLastError();
}

}  // namespace vidax
