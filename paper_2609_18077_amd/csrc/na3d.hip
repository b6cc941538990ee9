// 3D neighbourhood attention forward for gfx950 (the windowed attention of a
// video VAE decoder, Section 2 and the porting-bug table of the paper): each
// query (t, h, w) of a T x Hp x Wp token grid attends to the keys of its own
// window, a box of kt x kh x kw positions around it (clipped to the grid, or
// moved inward at the border), with a softmax over that key set.  bf16 in/out,
// fp32 accumulation, head dim 128.
//
// A workgroup of 4 waves owns a 2 x 4 x 16 block of queries (t, h, w); wave
// j owns the 2 x 4 x 4 sub-block at w offset 4 j, 32 queries, so every row
// of the workgroup's key box lies in every wave's windows along t and h (with
// 8 waves over a 2 x 8 x 16 block, each wave sat out the steps of the rows
// outside its own h range, a fifth of them).  The union of the workgroup's
// windows is a box of rows (t', h') times at most 26 consecutive w.  The
// workgroup streams that box two rows at a time: each step copies the two
// rows' keys and values (32 w positions each, from an even start) straight
// from global memory into LDS, double buffered, one barrier per step; two
// workgroups (64 KB of LDS each) share a CU.  Each wave computes one 32-key
// score block per step -- 16 keys of each row, at its own offset along w --
// as in the dense forward kernel:
//
//   S^T [32 keys x 32 queries] = K Q^T     8 x v_mfma_f32_32x32x16_bf16
//   P^T = exp2(S^T c - m), zero outside each query's window
//   O^T [128 x 32] += V^T P^T              8 x v_mfma_f32_32x32x16_bf16
//
// (score tile transposed so that a lane holds one query; P taken from the
// accumulator layout as the B operand; V^T read by ds_read_b64_tr_b16; the
// softmax reference m reset only when a block's row sum leaves [0, 2^64)).
// LDS holds the staged keys row-major, 256 bytes a key, with the 16-byte
// chunk c of key x stored at chunk c ^ f(x mod 16), f(x) = 4 (x mod 4) +
// x / 4: any 16 consecutive keys put one chunk in 16 different places (the
// score reads), and any 4 consecutive keys put a 64-byte span in 4 different
// quarters of the banks (the transposing reads).  Each 1 KB direct copy
// fills 4 whole keys, 256 contiguous bytes of global memory each.
#include "launch.hpp"

namespace vidax {
namespace {

constexpr int D = kHeadDim;
constexpr int QT = 2, QH = 4, QW = 4;  // query block of one wave
constexpr int WH = 1, WW = 4;          // waves of a workgroup along h and w
constexpr int NW = WH * WW, NT = NW * 64;
constexpr int ROWK = 32;               // staged keys per row
constexpr int STEPK = 2 * ROWK;        // keys per step (two rows)
constexpr int BUF = STEPK * D;         // elements of one staged tensor
constexpr int kBufferFlags = 0x00020000;  // raw buffer, 32-bit data format
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kSumLimit = 18446744073709551616.0f;  // 2^64

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr;

struct NaArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  int B, H, T, Hp, Wp, L;
  int kt, kh, kw;
  int shift;       // border: 0 clip, 1 shift
  float c;         // |scale| log2(e)
  uint32_t qsign;  // 0x80008000 when scale < 0: queries enter negated
  int nbt, nbh, nbw;  // workgroup blocks per axis
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

__device__ __forceinline__ i16x4 lds_read_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
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

// 16-byte chunk slot of chunk c of staged key x (an involution in c)
__device__ __forceinline__ int chunk_slot(int x, int c) {
  const int m = x & 15;
  return c ^ (((m & 3) << 2) | (m >> 2));
}

__global__ __launch_bounds__(NT, 2) void na3d_fwd_kernel(NaArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t K0[BUF], K1[BUF], V0[BUF], V1[BUF];
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int lid;
  {  // workgroups go round-robin over the 8 XCDs: contiguous ranges per XCD
    const int i = blockIdx.x, n = a.nwg;
    const int per = n >> 3, rem = n & 7, xcd = i & 7, kk = i >> 3;
    lid = xcd < rem ? xcd * (per + 1) + kk : rem * (per + 1) + (xcd - rem) * per + kk;
  }
  int x = lid;
  const int bw = x % a.nbw;
  x /= a.nbw;
  const int bh = x % a.nbh;
  x /= a.nbh;
  const int bt = x % a.nbt;
  x /= a.nbt;
  const int h = x % a.H, b = x / a.H;
  const int t0 = bt * QT, h0 = bh * QH * WH, w0 = bw * QW * WW;
  const int wi = wave / WW, wj = wave % WW;         // the wave's sub-block
  const int sh0 = h0 + QH * wi, sw0 = w0 + QW * wj;
  const bool wlive = sh0 < a.Hp && sw0 < a.Wp;       // uniform

  // the lane's query and its window
  const int qt = t0 + (l32 >> 4), qh = sh0 + ((l32 >> 2) & 3), qw = sw0 + (l32 & 3);
  const bool qlive = qt < a.T && qh < a.Hp && qw < a.Wp;
  const int2 wt = axis_window(min(qt, a.T - 1), a.T, a.kt, a.shift);
  const int2 wh = axis_window(min(qh, a.Hp - 1), a.Hp, a.kh, a.shift);
  const int2 ww = axis_window(min(qw, a.Wp - 1), a.Wp, a.kw, a.shift);

  // the workgroup's key box (windows are monotone in the query coordinate):
  // rows (t', h') and the staged w range [A0, A0 + 32)
  const int bt0 = axis_window(t0, a.T, a.kt, a.shift).x;
  const int bt1 = axis_window(min(t0 + QT - 1, a.T - 1), a.T, a.kt, a.shift).y;
  const int bh0 = axis_window(h0, a.Hp, a.kh, a.shift).x;
  const int bh1 = axis_window(min(h0 + QH * WH - 1, a.Hp - 1), a.Hp, a.kh, a.shift).y;
  const int A0 = axis_window(w0, a.Wp, a.kw, a.shift).x & ~1;
  const int nrh = bh1 - bh0 + 1;
  const int nrows = (bt1 - bt0 + 1) * nrh;
  const int nsteps = (nrows + 1) >> 1;
  // the wave's rows h' and its 16-key run [a0, a0 + 16) of each staged row
  const int wh0 = axis_window(min(sh0, a.Hp - 1), a.Hp, a.kh, a.shift).x;
  const int wh1 = axis_window(min(sh0 + QH - 1, a.Hp - 1), a.Hp, a.kh, a.shift).y;
  const int a0 = axis_window(min(sw0, a.Wp - 1), a.Wp, a.kw, a.shift).x & ~1;
  const int off = a0 - A0;  // 0 .. 13

  // register i of a score accumulator holds key row 8 (i >> 2) + 4 hi + (i & 3)
  // of the block: row i >> 3 of the step, run position j(i) = 8 ((i >> 2) & 1)
  // + 4 hi + (i & 3)
  bool wok[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int w = a0 + 8 * ((i >> 2) & 1) + 4 * hi + (i & 3);
    wok[i] = w >= ww.x && w <= ww.y;
  }

  const int tok = a.H * D, rbytes = tok * 2;
  const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.k + (size_t)b * a.L * tok), (short)0, a.L * rbytes, kBufferFlags);
  const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.v + (size_t)b * a.L * tok), (short)0, a.L * rbytes, kBufferFlags);

  // Rows (t', h') of the box are walked in order, two per step; a cursor
  // holds the coordinates of the first row of a step.
  auto advance = [&](int2 r, int n) __attribute__((always_inline)) {
    r.y += n;
    while (r.y > bh1) {
      r.y -= nrh;
      r.x += 1;
    }
    return r;
  };
  // staging: wave w copies 1 KB blocks 4 w .. 4 w + 3 of each tensor, 4 keys
  // a block (keys 0 .. 31 from the step's first row -- waves 0, 1 --, 32 .. 63
  // from its second -- waves 2, 3 --, at w positions A0 .. A0 + 31; a missing
  // second row repeats the first); lane i fills slot i & 15 of key
  // 4 blk + (i >> 4).  The lane's byte offset within the staged row span is
  // fixed (cg); the row's base is a uniform offset.
  const bool second = wave >= 2;  // uniform
  int cg[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int kx = 16 * wave + (lane >> 4) + 4 * u;
    cg[u] = (kx & 31) * rbytes + h * D * 2 + chunk_slot(kx, lane & 15) * 16;
  }
  auto stage = [&](int stp, int2 rowA, uint16_t* kb, uint16_t* vb) __attribute__((always_inline)) {
    const int2 rw = second && 2 * stp + 1 < nrows ? advance(rowA, 1) : rowA;
    const int rbase = __builtin_amdgcn_readfirstlane(((rw.x * a.Hp + rw.y) * a.Wp + A0) * rbytes);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int blk = 4 * wave + u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_ptr)(kb + blk * 512), 16, cg[u], rbase, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_ptr)(vb + blk * 512), 16, cg[u], rbase, 0, 0);
    }
  };

  // Q as the B operand: lane = query, d-chunk 2 st + hi of k-step st
  bf16x8 qop[8];
  {
    const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(a.q + (size_t)b * a.L * tok), (short)0, a.L * rbytes, kBufferFlags);
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

  // per-lane LDS element offsets: score operand (key row l32 of the block,
  // chunk 2 st + hi) and transposing V reads (as in the dense kernel's V
  // order: key 8 r + 4 hi + ((l & 15) >> 2) of a 16-key step, channels
  // 32 mb + 16 ((l >> 4) & 1) + 4 (l & 3) .. + 3); the second row's keys are
  // 32 further (same slot map), an immediate offset
  int koffs[8], voffs[4][2];
  {
    const int kx = 32 * (l32 >> 4) + off + (l32 & 15);
#pragma unroll
    for (int st = 0; st < 8; ++st) koffs[st] = kx * D + chunk_slot(kx, 2 * st + hi) * 8;
    const int vd = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int kk = off + 8 * r + 4 * hi + ((lane & 15) >> 2);
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const int d = 32 * mb + vd;
        voffs[mb][r] = kk * D + chunk_slot(kk, d >> 3) * 8 + (d & 7);
      }
    }
  }

  auto step = [&](int2 rowA, bool realB, const uint16_t* kb, const uint16_t* vb) __attribute__((always_inline)) {
    const int2 rowB = realB ? advance(rowA, 1) : rowA;
    const bool useA = wlive && rowA.y >= wh0 && rowA.y <= wh1;
    const bool useB = wlive && realB && rowB.y >= wh0 && rowB.y <= wh1;
    if (!(useA || useB)) return;  // uniform: nothing of this step is in the wave's windows
    f32x16 sc = f32x16{};
#pragma unroll
    for (int st = 0; st < 8; ++st) {
      const bf16x8 kop = *reinterpret_cast<const bf16x8*>(kb + koffs[st]);
      sc = mfma32(kop, qop[st], sc);
    }
    const bool ok0 = qlive && useA && rowA.x >= wt.x && rowA.x <= wt.y && rowA.y >= wh.x && rowA.y <= wh.y;
    const bool ok1 = qlive && useB && rowB.x >= wt.x && rowB.x <= wt.y && rowB.y >= wh.x && rowB.y <= wh.y;
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
          const float p0 = wok[i] ? __builtin_amdgcn_exp2f(fmaf(sc[i], a.c, k2 ? nm1 : nm0)) : 0.f;
          const float p1 = wok[i + 1] ? __builtin_amdgcn_exp2f(fmaf(sc[i + 1], a.c, k2 ? nm1 : nm0)) : 0.f;
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
        if (wok[i] && (i < 8 ? ok0 : ok1)) m = fmaxf(m, sc[i]);
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
    // O^T += V^T P^T, one 16-key step per staged row
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        i16x4 part[2];
#pragma unroll
        for (int r = 0; r < 2; ++r) part[r] = lds_read_tr16(vb + voffs[mb][r] + 32 * k2 * D);
        const bf16x8 vop = __builtin_bit_cast(bf16x8, __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7));
        oacc[mb] = mfma32(vop, pop[k2], oacc[mb]);
      }
  };

  int2 cur = make_int2(bt0, bh0);  // first row of step s
  stage(0, cur, K0, V0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  int s = 0;
  for (; s + 1 < nsteps; s += 2) {
    const int2 nxt = advance(cur, 2);
    stage(s + 1, nxt, K1, V1);
    step(cur, 2 * s + 1 < nrows, K0, V0);
    __builtin_amdgcn_s_waitcnt(0);  // this wave's copies have landed
    __syncthreads();
    cur = advance(nxt, 2);
    if (s + 2 < nsteps) stage(s + 2, cur, K0, V0);
    step(nxt, 2 * s + 3 < nrows, K1, V1);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  if (s < nsteps) step(cur, 2 * s + 1 < nrows, K0, V0);

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

hipError_t launch_na3d_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v, uint16_t* o, float* lse, int B,
                           int H, int T, int Hp, int Wp, int kt, int kh, int kw, int shift, float scale,
                           hipStream_t stream) {
  NaArgs a;
  a.q = q; a.k = k; a.v = v; a.o = o; a.lse = lse;
  a.B = B; a.H = H; a.T = T; a.Hp = Hp; a.Wp = Wp; a.L = T * Hp * Wp;
  a.kt = kt; a.kh = kh; a.kw = kw; a.shift = shift;
  a.c = fabsf(scale) * kLog2e;
  a.qsign = scale < 0.f ? 0x80008000u : 0u;
  a.nbt = (T + QT - 1) / QT;
  a.nbh = (Hp + QH * WH - 1) / (QH * WH);
  a.nbw = (Wp + QW * WW - 1) / (QW * WW);
  a.nwg = B * H * a.nbt * a.nbh * a.nbw;
  return launch_kernel(na3d_fwd_kernel, (unsigned)a.nwg, (unsigned)NT, stream, a);
}

}  // namespace vidax
