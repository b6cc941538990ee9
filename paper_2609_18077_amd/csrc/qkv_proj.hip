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
// tiles (256 rows x 64 channels each) straight from global memory into LDS,
// double buffered, one barrier per stage; per stage a wave issues 32 matrix
// instructions.  In LDS a tile row (128 bytes) is followed by 16 bytes of
// padding: every copy instruction then fetches whole rows with its lanes in
// address order (coalesced; the pad lane reads past the buffer's records:
// zero, no memory access), and
// the operand reads (16 rows x one 16-byte chunk per 16 lanes, rows 144 bytes
// apart) are free of bank conflicts.  After the last stage the LDS holds the
// rotary (cos, sin) table for the epilogue.
#include "launch.hpp"

namespace vidax {
namespace {

constexpr int D = kHeadDim;
constexpr int NW = 8, NT = NW * 64;
constexpr int BNC = 256;  // output channels per workgroup
constexpr int BMT = 256;  // tokens per workgroup
constexpr int BK = 64;    // input channels per stage
constexpr int kPitch = BK + 8;    // elements per staged row: 64 channels + 16 bytes of padding
constexpr int TILE = 256 * kPitch;  // elements of one staged tile (36 KB)
constexpr int kCopies = TILE * 2 / 1024;  // 1 KB copy instructions per tile (36)
static_assert(kCopies == 36, "the copy split over the waves assumes 36 copies per tile");
static_assert(kRopeTableMax * 8 <= TILE * 2, "the rotary table must fit in one stage buffer");
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

// Output staging: slot of 16-byte chunk c of staging row r (an involution in
// c); for 16 consecutive rows and one chunk, and for 4 rows x 4 chunks aligned
// by 4, the slots are distinct (no LDS bank conflicts).
__device__ __forceinline__ int out_slot(int c, int r) {
  const int x = r & 15;
  return c ^ (((x & 3) << 2) | (x >> 2));
}

__device__ __forceinline__ float half_swap_sum(float x) {
  // lanes l and l ^ 32 hold the same token
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// HALF: half-split rotary pairs (channel o_a + j with o_a + j + d_a / 2)
template <bool HALF>
__global__ __launch_bounds__(NT) void qkv_proj_kernel(QkvArgs a) {
  // tile layout: row r at element r * kPitch, 16-byte chunk c of the stage's
  // 64 input channels at + 8 c
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
  // staging: copy j (of kCopies per tile) fills 16-byte slots 64 j .. 64 j + 63
  // of the tile, lane l slot s = 64 j + l = row s / 9, chunk s % 9 (chunk 8 is
  // the padding: its offset lies past the records, so it reads zero without
  // a memory access).  Waves 0..3 issue copies 5 w .. 5 w + 4, waves 4..7
  // copies 20 + 4 (w - 4) .. + 3.
  const int cfirst = wave < 4 ? 5 * wave : 20 + 4 * (wave - 4);
  const int ccount = wave < 4 ? 5 : 4;
  int goff[5];
#pragma unroll
  for (int u = 0; u < 5; ++u) {
    const int sl = 64 * (cfirst + u) + lane, r = sl / 9, c = sl - 9 * r;
    goff[u] = c < 8 ? r * cbytes + c * 16 : 0x7ffff000;
  }
  auto stage = [&](int s, uint16_t* wb, uint16_t* xb) __attribute__((always_inline)) {
    const int koff = __builtin_amdgcn_readfirstlane(s * BK * 2);
#pragma unroll
    for (int u = 0; u < 5; ++u) {
      if (u < ccount) {
        const int j = cfirst + u;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr)(wb + j * 512), 16, goff[u], koff, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_ptr)(xb + j * 512), 16, goff[u], koff, 0, 0);
      }
    }
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int cb = 0; cb < 4; ++cb) acc[cb][0] = acc[cb][1] = f32x16{};
  // one stage: 4 k-steps x (4 channel blocks x 2 token blocks); the A operand
  // of channel block cb, k-step st: row 128 wh + 32 cb + l32, chunk 2 st + hi
  const int abase = (128 * wh + l32) * kPitch + 8 * hi;
  const int bbase = (64 * wt + l32) * kPitch + 8 * hi;
  auto compute = [&](const uint16_t* wb, const uint16_t* xb) __attribute__((always_inline)) {
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      bf16x8 av[4], bv[2];
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
        av[cb] = *reinterpret_cast<const bf16x8*>(wb + abase + 32 * cb * kPitch + 16 * st);
#pragma unroll
      for (int tb = 0; tb < 2; ++tb)
        bv[tb] = *reinterpret_cast<const bf16x8*>(xb + bbase + 32 * tb * kPitch + 16 * st);
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
  float2* tab = reinterpret_cast<float2*>(W0);  // the stage buffers are free now (36 KB)
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
  // the wave's 8 KB output staging area (32 tokens x 128 channels), in the
  // stage buffers W1 and X0 that are free now: the results leave as whole
  // 256-byte head rows, 4 tokens per store instruction
  uint16_t* const ostage = (wave < 4 ? W1 : X0) + (wave & 3) * 32 * D;

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
      if (HALF) {
        // A channel's partner lies d_a / 2 further in its axis block, in
        // another register or the other lane half: the token's values go
        // through wave-private fp32 rows in X1 (free now), an eighth of the
        // wave's tokens at a time: the two lanes of a token write their
        // halves to row x, rotate their channels from row x into row y in a
        // plain loop, and read row y back (one wave, in order: no barrier).
        float* const xrow = reinterpret_cast<float*>(X1) + (wave * 8 + (l32 & 3)) * D;
        float* const yrow = xrow + 4 * D;
        const bool rot = n < rp.n_rot;
        const int t = n / (rp.gh * rp.gw);
        const int rr = n - t * rp.gh * rp.gw;
        const int hh = rr / rp.gw;
        const int ww = rr - hh * rp.gw;
        const int ht = rp.dt >> 1, hd = rp.dh >> 1;
        for (int pass = 0; pass < 8; ++pass) {
          if ((l32 >> 2) != pass || !rot) continue;
#pragma unroll
          for (int cb = 0; cb < 4; ++cb)
#pragma unroll
            for (int g = 0; g < 4; ++g)
              *reinterpret_cast<float4*>(xrow + 32 * cb + 8 * g + 4 * hi) =
                  make_float4(acc[cb][tb][4 * g], acc[cb][tb][4 * g + 1], acc[cb][tb][4 * g + 2], acc[cb][tb][4 * g + 3]);
#pragma unroll 1
          for (int k = 0; k < 64; ++k) {
            const int ch = 32 * (k >> 4) + 8 * ((k >> 2) & 3) + 4 * hi + (k & 3);
            int o, hl, pb;
            if (ch < rp.dt) { o = 0; hl = ht; pb = 0; }
            else if (ch < rp.dt + rp.dh) { o = rp.dt; hl = hd; pb = ht; }
            else { o = rp.dt + rp.dh; hl = rp.dw >> 1; pb = ht + hd; }
            const bool first = ch - o < hl;
            const int j = first ? ch - o : ch - o - hl;
            const PairSlot sl = pair_slot(rp, pb + j);
            const int pos = sl.axis == 0 ? t : (sl.axis == 1 ? hh : ww);
            const float2 e = tab[sl.base + pos * sl.stride];
            const float x = xrow[ch], xp = xrow[first ? ch + hl : ch - hl];
            yrow[ch] = first ? fmaf(x, e.x, -xp * e.y) : fmaf(xp, e.y, x * e.x);
          }
#pragma unroll
          for (int cb = 0; cb < 4; ++cb)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const float4 y = *reinterpret_cast<const float4*>(yrow + 32 * cb + 8 * g + 4 * hi);
              acc[cb][tb][4 * g] = y.x;
              acc[cb][tb][4 * g + 1] = y.y;
              acc[cb][tb][4 * g + 2] = y.z;
              acc[cb][tb][4 * g + 3] = y.w;
            }
        }
      } else if (rp.enabled && n < rp.n_rot) {
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
    // the lane's token l32, channels 32 cb + 8 g + 4 hi .. + 3: half hi of chunk 4 cb + g
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint2 pk;
        pk.x = pack_bf16x2(acc[cb][tb][4 * g + 0], acc[cb][tb][4 * g + 1]);
        pk.y = pack_bf16x2(acc[cb][tb][4 * g + 2], acc[cb][tb][4 * g + 3]);
        *reinterpret_cast<uint2*>(ostage + l32 * D + out_slot(4 * cb + g, l32) * 8 + 4 * hi) = pk;
      }
    // whole rows out: slot lane & 15 of row 4 i + (lane >> 4) holds chunk out_slot(lane & 15, row)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = 4 * i + (lane >> 4);
      const uint4 v = *reinterpret_cast<const uint4*>(ostage + r * D + (lane & 15) * 8);
      const int mm = m0 + 64 * wt + 32 * tb + r;
      if (mm < a.M)
        *reinterpret_cast<uint4*>(outp + (size_t)mm * a.H * D + (size_t)head * D + out_slot(lane & 15, r) * 8) = v;
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
  return rp.enabled && rp.pair_mode ? launch_kernel(qkv_proj_kernel<true>, (unsigned)a.nwg, (unsigned)NT, stream, a)
                                     : launch_kernel(qkv_proj_kernel<false>, (unsigned)a.nwg, (unsigned)NT, stream, a);
}

}  // namespace vidax
