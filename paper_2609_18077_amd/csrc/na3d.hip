// 3D neighbourhood attention forward for gfx950 (the windowed attention of a
// video VAE decoder, Section 2 and the porting-bug table of the paper): each
// query (t, h, w) of a T x Hp x Wp token grid attends to the keys of its own
// window, a box of kt x kh x kw positions around it (clipped to the grid, or
// moved inward at the border), with a softmax over that key set.  bf16 in/out,
// fp32 accumulation, head dim 128.
//
// One wave owns a 2 x 4 x 4 block of 32 queries (t, h, w).  The union of
// their windows is a box of at most (kt + 1) x (kh + 3) x (kw + 3) keys; the
// wave walks it as runs of 16 keys along w (one run per (t', h') row of the
// box, starting at an even w), two runs per 32-key score block:
//
//   S^T [32 keys x 32 queries] = K Q^T     8 x v_mfma_f32_32x32x16_bf16
//   P^T = exp2(S^T c - m), zero outside each query's window
//   O^T [128 x 32] += V^T P^T              8 x v_mfma_f32_32x32x16_bf16
//
// as in the dense forward kernel (score tile transposed so that a lane holds
// one query; P taken from the accumulator layout as the B operand; the
// softmax reference m reset only when a block's row sum leaves [0, 2^64)).
// Waves are independent (no LDS, no barriers): the K operand is read straight
// from global memory (a lane's 16 bytes are one key row's d-chunk), and the
// V^T operand from a transposed copy of V written by the first launch,
// [B, H, 128, T*Hp, Wps] with the w rows padded with zeros to Wps (a multiple
// of 8), so a lane's 4 consecutive keys of one channel are one aligned 8-byte
// load.  Out-of-range rows read as zero through buffer resources.
#include "common.hpp"

namespace vidax {
namespace {

constexpr int D = kHeadDim;
constexpr int QT = 2, QH = 4, QW = 4;  // query block of one wave
constexpr int NWV = 4;                 // waves per workgroup
constexpr int kBufferFlags = 0x00020000;  // raw buffer, 32-bit data format
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kSumLimit = 18446744073709551616.0f;  // 2^64

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

struct NaArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* vt;
  uint16_t* o;
  float* lse;
  int B, H, T, Hp, Wp, L;
  int Wps;    // padded row length of the transposed V
  int plane;  // T * Hp * Wps: elements of one channel of one (b, h) in vt
  int kt, kh, kw;
  int shift;       // border: 0 clip, 1 shift
  float c;         // |scale| log2(e)
  uint32_t qsign;  // 0x80008000 when scale < 0: queries enter negated
  int nbt, nbh, nbw;
  int nblk;  // wave blocks: B * H * nbt * nbh * nbw
  int nwg;
};

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float wave_half_max(float x) {
  // lanes l and l ^ 32 hold the same query
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float wave_half_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

// Inclusive window [lo, hi] on an axis of N positions for a query at c
// (window size K odd): clipped to the axis, or moved inward to keep K.
__device__ __forceinline__ int2 axis_window(int c, int N, int K, int shift) {
  const int r = (K - 1) >> 1;
  if (!shift) return make_int2(max(0, c - r), min(N - 1, c + r));
  if (N <= K) return make_int2(0, N - 1);
  const int lo = min(max(c - r, 0), N - K);
  return make_int2(lo, lo + K - 1);
}

// ---- vt[b][h][c][row][w] = v[b][row * Wp + w][h][c] (rows = T * Hp), zero
// for Wp <= w < Wps.  Workgroup: one (b, h, row) and 64 positions of w.
__global__ __launch_bounds__(256) void na3d_transpose_v_kernel(const uint16_t* __restrict__ v,
                                                               uint16_t* __restrict__ vt, NaArgs a) {
  __shared__ uint16_t tile[64][D + 8];
  const int nwc = (a.Wps + 63) >> 6;
  int x = blockIdx.x;
  const int wc = x % nwc;
  x /= nwc;
  const int row = x % (a.T * a.Hp);
  x /= a.T * a.Hp;
  const int h = x % a.H, b = x / a.H;
  const int w0 = wc * 64;
  const int tid = threadIdx.x;
  const size_t tok = (size_t)a.H * D;
  // load 64 tokens x 128 channels, 16 bytes per thread and pass
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int e = p * 256 + tid;  // chunk index: token e >> 4, chunk e & 15
    const int wl = e >> 4, ch = e & 15;
    const int w = w0 + wl;
    uint4 val = make_uint4(0, 0, 0, 0);
    if (w < a.Wp) val = *reinterpret_cast<const uint4*>(v + ((size_t)b * a.L + (size_t)row * a.Wp + w) * tok + (size_t)h * D + ch * 8);
    *reinterpret_cast<uint4*>(&tile[wl][ch * 8]) = val;
  }
  __syncthreads();
  // write 128 channels x 64 positions, 4 positions (8 bytes) per thread and pass
  uint16_t* out = vt + ((size_t)b * a.H + h) * D * a.plane + (size_t)row * a.Wps;
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    const int e = p * 256 + tid;  // channel e >> 4, positions 4 (e & 15) ..
    const int c = e >> 4, wl = 4 * (e & 15);
    if (w0 + wl < a.Wps) {  // Wps is a multiple of 8: all four positions are in the row
      uint2 pk;
      pk.x = (uint32_t)tile[wl][c] | ((uint32_t)tile[wl + 1][c] << 16);
      pk.y = (uint32_t)tile[wl + 2][c] | ((uint32_t)tile[wl + 3][c] << 16);
      *reinterpret_cast<uint2*>(out + (size_t)c * a.plane + w0 + wl) = pk;
    }
  }
}

// ---- the attention: one wave per 2 x 4 x 4 query block.
__global__ __launch_bounds__(NWV * 64) __attribute__((amdgpu_waves_per_eu(2))) void na3d_fwd_kernel(NaArgs a) {
  const int lane = threadIdx.x & 63, l32 = lane & 31, hi = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int lid;
  {  // workgroups go round-robin over the 8 XCDs: contiguous ranges per XCD
    const int i = blockIdx.x, n = a.nwg;
    const int per = n >> 3, rem = n & 7, xcd = i & 7, kk = i >> 3;
    lid = xcd < rem ? xcd * (per + 1) + kk : rem * (per + 1) + (xcd - rem) * per + kk;
  }
  const int blk = lid * NWV + wave;
  if (blk >= a.nblk) return;  // whole wave; there are no barriers
  int x = blk;
  const int bw = x % a.nbw;
  x /= a.nbw;
  const int bh = x % a.nbh;
  x /= a.nbh;
  const int bt = x % a.nbt;
  x /= a.nbt;
  const int h = x % a.H, b = x / a.H;
  const int t0 = bt * QT, h0 = bh * QH, w0 = bw * QW;

  // the lane's query and its window
  const int qt = t0 + (l32 >> 4), qh = h0 + ((l32 >> 2) & 3), qw = w0 + (l32 & 3);
  const bool qlive = qt < a.T && qh < a.Hp && qw < a.Wp;
  const int2 wt = axis_window(min(qt, a.T - 1), a.T, a.kt, a.shift);
  const int2 wh = axis_window(min(qh, a.Hp - 1), a.Hp, a.kh, a.shift);
  const int2 ww = axis_window(min(qw, a.Wp - 1), a.Wp, a.kw, a.shift);

  // the block's key box (windows are monotone in the query coordinate)
  const int bt0 = axis_window(t0, a.T, a.kt, a.shift).x;
  const int bt1 = axis_window(min(t0 + QT - 1, a.T - 1), a.T, a.kt, a.shift).y;
  const int bh0 = axis_window(h0, a.Hp, a.kh, a.shift).x;
  const int bh1 = axis_window(min(h0 + QH - 1, a.Hp - 1), a.Hp, a.kh, a.shift).y;
  const int a0 = axis_window(w0, a.Wp, a.kw, a.shift).x & ~1;  // run start (even)
  const int nrh = bh1 - bh0 + 1;
  const int nruns = (bt1 - bt0 + 1) * nrh;
  const int nsb = (nruns + 1) >> 1;

  // register i of a score accumulator holds key row 8 (i >> 2) + 4 hi + (i & 3)
  // of the block: run i >> 3, position j(i) = 8 ((i >> 2) & 1) + 4 hi + (i & 3)
  bool wok[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int w = a0 + 8 * ((i >> 2) & 1) + 4 * hi + (i & 3);
    wok[i] = w >= ww.x && w <= ww.y;
  }

  const int tok = a.H * D, rbytes = tok * 2;
  const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.q + (size_t)b * a.L * tok), (short)0, a.L * rbytes, kBufferFlags);
  const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.k + (size_t)b * a.L * tok), (short)0, a.L * rbytes, kBufferFlags);
  const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.vt + ((size_t)b * a.H + h) * D * a.plane), (short)0, D * a.plane * 2, kBufferFlags);

  // Q as the B operand: lane = query, d-chunk 2 st + hi of k-step st
  bf16x8 qop[8];
  {
    const uint32_t qoff = qlive ? (uint32_t)(((qt * a.Hp + qh) * a.Wp + qw) * rbytes + h * D * 2) : 0xfffff000u;
#pragma unroll
    for (int st = 0; st < 8; ++st) {
      u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rq, qoff + (2 * st + hi) * 16, 0, 0);
      v ^= a.qsign;
      qop[st] = __builtin_bit_cast(bf16x8, v);
    }
  }

  f32x16 oacc[4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) oacc[mb] = f32x16{};
  float mref = -INFINITY, lsum = 0.f;
  const uint32_t ones = 0x3f803f80u;  // bf16 (1, 1)

  // runs r0, r1 of score block p: (t', h') rows of the box
  auto run_row = [&](int r) __attribute__((always_inline)) {
    const int tk = bt0 + r / nrh, hk = bh0 + r % nrh;
    return make_int2(tk, hk);
  };
  auto load_k = [&](int p, u32x4 kreg[8]) __attribute__((always_inline)) {
    const int r = min(2 * p + (l32 >> 4), nruns - 1);
    const int2 rk2 = run_row(r);
    const uint32_t koff = (uint32_t)(((rk2.x * a.Hp + rk2.y) * a.Wp + a0 + (l32 & 15)) * rbytes + h * D * 2);
#pragma unroll
    for (int st = 0; st < 8; ++st) kreg[st] = __builtin_amdgcn_raw_buffer_load_b128(rk, koff + (2 * st + hi) * 16, 0, 0);
  };

  u32x4 kcur[8];
  if (nsb > 0) load_k(0, kcur);
  for (int p = 0; p < nsb; ++p) {
    const int r0 = 2 * p, r1 = min(2 * p + 1, nruns - 1);
    const bool real1 = 2 * p + 1 < nruns;
    const int2 row0 = run_row(r0), row1 = run_row(r1);
    // V^T operand of both runs: lane = channel 32 mb + l32, keys 4 hi .. +3 and 8 + 4 hi .. +3
    u32x2 vlo[2][4], vhi[2][4];
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const int2 rw = k2 ? row1 : row0;
      const uint32_t base = (uint32_t)(((rw.x * a.Hp + rw.y) * a.Wps + a0 + 4 * hi) * 2);
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const uint32_t off = base + (uint32_t)((32 * mb + l32) * a.plane) * 2u;
        vlo[k2][mb] = __builtin_amdgcn_raw_buffer_load_b64(rv, off, 0, 0);
        vhi[k2][mb] = __builtin_amdgcn_raw_buffer_load_b64(rv, off + 16, 0, 0);
      }
    }
    // scores of this block
    f32x16 s = f32x16{};
#pragma unroll
    for (int st = 0; st < 8; ++st) s = mfma32(__builtin_bit_cast(bf16x8, kcur[st]), qop[st], s);
    if (p + 1 < nsb) load_k(p + 1, kcur);

    // the lane's query sees run r (rows t', h') and, within it, positions wok
    const bool ok0 = qlive && row0.x >= wt.x && row0.x <= wt.y && row0.y >= wh.x && row0.y <= wh.y;
    const bool ok1 = qlive && real1 && row1.x >= wt.x && row1.x <= wt.y && row1.y >= wh.x && row1.y <= wh.y;
    bf16x8 pop[2];
    auto probs = [&]() __attribute__((always_inline)) {
      const float nm0 = ok0 ? -mref : -INFINITY, nm1 = ok1 ? -mref : -INFINITY;
      float tsum = 0.f;
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        uint32_t pw[4];
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const int i = 8 * k2 + e;
          const float p0 = wok[i] ? __builtin_amdgcn_exp2f(fmaf(s[i], a.c, k2 ? nm1 : nm0)) : 0.f;
          const float p1 = wok[i + 1] ? __builtin_amdgcn_exp2f(fmaf(s[i + 1], a.c, k2 ? nm1 : nm0)) : 0.f;
          pw[e >> 1] = pack_bf16x2(p0, p1);
          tsum = dot2(pw[e >> 1], ones, tsum);
        }
        pop[k2] = __builtin_bit_cast(bf16x8, make_uint4(pw[0], pw[1], pw[2], pw[3]));
      }
      return tsum;
    };
    float tsum = probs();
    if (__builtin_amdgcn_ballot_w64(!(tsum < kSumLimit)) != 0) {
      // reset the reference to the running max of the valid scores
      float m = -INFINITY;
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (wok[i] && (i < 8 ? ok0 : ok1)) m = fmaxf(m, s[i]);
      const float m2 = wave_half_max(m);
      const float mnew = fmaxf(mref, m2 == -INFINITY ? -INFINITY : m2 * a.c);
      const float alpha = mnew == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(mref - mnew);
      lsum *= alpha;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[mb][i] *= alpha;
      mref = mnew;
      tsum = probs();
    }
    lsum += tsum;
    // O^T += V^T P^T
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const u32x4 w4 = {vlo[k2][mb][0], vlo[k2][mb][1], vhi[k2][mb][0], vhi[k2][mb][1]};
        oacc[mb] = mfma32(__builtin_bit_cast(bf16x8, w4), pop[k2], oacc[mb]);
      }
  }

  // ---- output: O = O^T / l, lse = (m + log2 l) ln 2; lane holds its query,
  // d = 32 mb + 8 g + 4 hi + (0..3)
  const float l = wave_half_sum(lsum);
  const float inv = l > 0.f ? 1.0f / l : 0.f;
  const int qn = (qt * a.Hp + qh) * a.Wp + qw;
  if (qlive) {
    uint16_t* op = a.o + ((size_t)b * a.L + qn) * tok + (size_t)h * D;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint2 pk;
        pk.x = pack_bf16x2(oacc[mb][4 * g + 0] * inv, oacc[mb][4 * g + 1] * inv);
        pk.y = pack_bf16x2(oacc[mb][4 * g + 2] * inv, oacc[mb][4 * g + 3] * inv);
        *reinterpret_cast<uint2*>(op + mb * 32 + 8 * g + 4 * hi) = pk;
      }
    if (a.lse && hi == 0) a.lse[((size_t)b * a.H + h) * a.L + qn] = (mref + __log2f(l)) * 0.69314718055994531f;
  }
}

}  // namespace

size_t na3d_workspace_elems(int B, int H, int T, int Hp, int Wp) {
  const size_t wps = ((size_t)Wp + 7) / 8 * 8;
  return (size_t)B * H * D * T * Hp * wps;
}

hipError_t launch_na3d_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v, uint16_t* o, float* lse,
                           uint16_t* vt, int B, int H, int T, int Hp, int Wp, int kt, int kh, int kw, int shift,
                           float scale, hipStream_t stream) {
  NaArgs a;
  a.q = q; a.k = k; a.vt = vt; a.o = o; a.lse = lse;
  a.B = B; a.H = H; a.T = T; a.Hp = Hp; a.Wp = Wp; a.L = T * Hp * Wp;
  a.Wps = (Wp + 7) / 8 * 8;
  a.plane = T * Hp * a.Wps;
  a.kt = kt; a.kh = kh; a.kw = kw; a.shift = shift;
  a.c = fabsf(scale) * kLog2e;
  a.qsign = scale < 0.f ? 0x80008000u : 0u;
  a.nbt = (T + QT - 1) / QT;
  a.nbh = (Hp + QH - 1) / QH;
  a.nbw = (Wp + QW - 1) / QW;
  a.nblk = B * H * a.nbt * a.nbh * a.nbw;
  a.nwg = (a.nblk + NWV - 1) / NWV;
  const int ntr = B * H * T * Hp * ((a.Wps + 63) / 64);
  hipLaunchKernelGGL(na3d_transpose_v_kernel, dim3((unsigned)ntr), dim3(256), 0, stream, v, vt, a);
  hipLaunchKernelGGL(na3d_fwd_kernel, dim3((unsigned)a.nwg), dim3(NWV * 64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace vidax
