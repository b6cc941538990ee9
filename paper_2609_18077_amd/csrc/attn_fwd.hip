// Flash-attention forward for gfx950: bf16 MFMA (32x32x16) with fp32
// accumulation, streaming softmax, fused 3D rotary embedding, per-batch
// valid-key prefix.  Head dim 128.
//
// Work decomposition
//   One workgroup = 8 waves = 256 query rows of one (batch, head); each wave
//   owns 32 query rows.  Keys/values stream through LDS in tiles of 64, two
//   buffers each.  The loop is software pipelined: while the softmax of tile j
//   runs on the vector ALUs, the matrix cores already compute the scores of
//   tile j+1; while the PV products of tile j run, the threads write the next
//   K tile (rotated) and V tile into the free buffers.  One barrier per tile.
//
// Matrix-core formulation (per wave, per key tile)
//   S^T[64 keys x 32 queries] = K_tile * Q^T   (16 MFMAs: 2 key blocks x 8 d-steps)
//   O^T[128 d x 32 queries]  += V^T * P^T      (16 MFMAs: 4 d blocks x 4 key-steps)
//   Computing the transposed scores puts one query column in each lane, so the
//   softmax row max/sum are register-local plus one swap between the two lane
//   halves, and the fp32 scores convert in place into the bf16 B operand of
//   the PV product (no shuffles).  The key order inside a 16-key step is the
//   accumulator's natural order.  V stays row-major in LDS; its V^T operands
//   are read with the gfx950 transposing LDS load (ds_read_b64_tr_b16), which
//   hands each lane 4 keys of one d column per read.
//
// Softmax: p = exp2(s * c - m) with c = |scale| * log2 e in one FMA (the
// rotated query is rounded to bf16 unscaled; a negative scale negates it, a
// zero scale zeroes it).  The output/sum rescale is skipped until some row's
// tile max exceeds its reference max by more than 8 (factor 256), which keeps
// every exponent <= 2^8 and the result exact up to rounding.  Row sums add
// the bf16-rounded p actually fed to the PV product (v_dot2 with ones).
//
// LDS (per workgroup): K tiles 2 x 16 KB and V tiles 2 x 16 KB (row-major,
// 16-byte chunks XOR swizzled by row), rotary table <= 32 KB.
#include "common.hpp"

namespace vidax {
namespace {

constexpr int D = kHeadDim;
constexpr int BM = 256;
constexpr int BN = 64;
constexpr int NW = 8;
constexpr int NT = NW * 64;
constexpr float kRescaleThreshold = 8.0f;

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  const int32_t* kv_valid_len;
  int B, H, Lq, Lk;
  int nqt;      // query tiles per (b, h)
  int nwg;      // total workgroups
  float c2;     // |scale| * log2(e), or 1 when scale == 0
  float qsign;  // +1, -1, or 0 (scale == 0) applied to the rotated query
  RopeParams rp;
  // mixed-radix increment of a key token index by BN: (dt, dh, dw) digits
  int step_t, step_h, step_w;
};

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float wave_half_max(float x) {
  // lanes l and l^32 hold the same query: combine their partial maxima
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float wave_half_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Rotates the 4 interleaved pairs of one 16-byte chunk with table entries.
__device__ __forceinline__ uint4 rotate_chunk(uint4 v, const float2* __restrict__ tab, const int idx[4]) {
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const float2 cs = tab[idx[p]];
    const float x0 = bf16lo_to_f32(w[p]);
    const float x1 = bf16hi_to_f32(w[p]);
    w[p] = pack_bf16x2(fmaf(x0, cs.x, -x1 * cs.y), fmaf(x0, cs.y, x1 * cs.x));
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

__device__ __forceinline__ int sel_pos(int axis, int t, int h, int w) {
  return axis == 0 ? t : (axis == 1 ? h : w);
}

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ i16x4 lds_read_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
}

// 16-byte chunk c of row r of a K tile / V tile
__device__ __forceinline__ int k_off(int r, int c) { return r * D + ((c ^ (r & 15)) << 3); }
__device__ __forceinline__ int v_off(int r, int c) { return r * D + ((c ^ ((r & 3) << 2)) << 3); }

template <bool ROPE>
__global__ __launch_bounds__(NT) void attn_fwd_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][BN * D];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[2][BN * D];
  // rotary table plus one identity entry (cos 1, sin 0) for unrotated tokens
  __shared__ float2 tab[ROPE ? kRopeTableMax + 1 : 1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31;
  const int hi = lane >> 5;

  // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
  // contiguous range of logical tiles so the query tiles of one (b, h) share
  // that XCD's L2 for the K/V stream.
  int lid;
  {
    const int i = blockIdx.x, n = a.nwg;
    const int per = n >> 3, rem = n & 7, xcd = i & 7, kk = i >> 3;
    lid = xcd < rem ? xcd * (per + 1) + kk : rem * (per + 1) + (xcd - rem) * per + kk;
  }
  const int qt = lid % a.nqt;
  const int bh = lid / a.nqt;
  const int h = bh % a.H;
  const int b = bh / a.H;

  int lv = a.Lk;
  if (a.kv_valid_len) lv = min(max(a.kv_valid_len[b], 0), a.Lk);

  const size_t tok = (size_t)a.H * D;
  const uint16_t* qbh = a.q + (size_t)b * a.Lq * tok + (size_t)h * D;
  const uint16_t* kbh = a.k + (size_t)b * a.Lk * tok + (size_t)h * D;
  const uint16_t* vbh = a.v + (size_t)b * a.Lk * tok + (size_t)h * D;
  uint16_t* obh = a.o + (size_t)b * a.Lq * tok + (size_t)h * D;

  const int qrow = qt * BM + wave * 32 + l32;
  const bool qlive = qrow < a.Lq;

  if (lv == 0) {
    // no valid key: output 0, lse -inf
    if (qlive) {
#pragma unroll
      for (int s = 0; s < 8; ++s)
        *reinterpret_cast<uint4*>(obh + (size_t)qrow * tok + (2 * s + hi) * 8) = make_uint4(0, 0, 0, 0);
      if (a.lse && hi == 0) a.lse[((size_t)b * a.H + h) * a.Lq + qrow] = -INFINITY;
    }
    return;
  }

  if (ROPE) {
    for (int e = tid; e < a.rp.n_entries; e += NT) tab[e] = rope_table_entry(a.rp, e);
    if (tid == 0) tab[a.rp.n_entries] = make_float2(1.f, 0.f);
    __syncthreads();
  }

  // ---- Q: lane holds query qrow, d-chunks 2s + hi (s = 0..7) as MFMA B operands
  bf16x8 qreg[8];
  {
    int t = 0, hh = 0, w = 0;
    const bool qrot = ROPE && qlive && qrow < a.rp.n_rot;
    if (qrot) {
      t = qrow / (a.rp.gh * a.rp.gw);
      const int r = qrow - t * a.rp.gh * a.rp.gw;
      hh = r / a.rp.gw;
      w = r - hh * a.rp.gw;
    }
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int c = 2 * s + hi;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (qlive) v = *reinterpret_cast<const uint4*>(qbh + (size_t)qrow * tok + c * 8);
      uint32_t wq[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        float x0 = bf16lo_to_f32(wq[p]);
        float x1 = bf16hi_to_f32(wq[p]);
        if (qrot) {
          const PairSlot sl = pair_slot(a.rp, 4 * c + p);
          const float2 cs = tab[sl.base + sel_pos(sl.axis, t, hh, w) * sl.stride];
          const float y0 = fmaf(x0, cs.x, -x1 * cs.y);
          const float y1 = fmaf(x0, cs.y, x1 * cs.x);
          x0 = y0;
          x1 = y1;
        }
        wq[p] = pack_bf16x2(x0 * a.qsign, x1 * a.qsign);
      }
      qreg[s] = __builtin_bit_cast(bf16x8, make_uint4(wq[0], wq[1], wq[2], wq[3]));
    }
  }

  // ---- staging: thread owns chunk kc of rows kr0 and kr0 + 32 of every K and V tile
  const int kc = lane & 15;
  const int kr0 = (lane >> 4) + 4 * wave;

  // rotary state of the two K rows (token index kr0 + 32 r + BN * tile)
  int kslot_base[4], kslot_stride[4], kslot_axis[4];
  int kt[2] = {0, 0}, kh[2] = {0, 0}, kw[2] = {0, 0};
  if (ROPE) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const PairSlot sl = pair_slot(a.rp, 4 * kc + p);
      kslot_base[p] = sl.base;
      kslot_stride[p] = sl.stride;
      kslot_axis[p] = sl.axis;
    }
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int n = kr0 + 32 * r;
      kt[r] = n / (a.rp.gh * a.rp.gw);
      const int rr = n - kt[r] * a.rp.gh * a.rp.gw;
      kh[r] = rr / a.rp.gw;
      kw[r] = rr - kh[r] * a.rp.gw;
    }
  }

  const int ntiles = (lv + BN - 1) / BN;

  // Rows at or beyond lv read row lv - 1 (always valid) and are zeroed, so the
  // loads carry no branch; tiles past the end are staged but never used.
  auto load_rows = [&](const uint16_t* base, int tile, uint4 reg[2]) {
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int n = tile * BN + kr0 + 32 * r;
      const uint4 v = *reinterpret_cast<const uint4*>(base + (size_t)min(n, lv - 1) * tok + kc * 8);
      const bool ok = n < lv;
      reg[r] = make_uint4(ok ? v.x : 0u, ok ? v.y : 0u, ok ? v.z : 0u, ok ? v.w : 0u);
    }
  };

  auto store_k = [&](int tile, uint16_t* buf, const uint4 reg[2]) {
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int row = kr0 + 32 * r;
      uint4 kv = reg[r];
      if (ROPE) {
        const bool rot = tile * BN + row < a.rp.n_rot;
        int idx[4];
#pragma unroll
        for (int p = 0; p < 4; ++p)
          idx[p] = rot ? kslot_base[p] + sel_pos(kslot_axis[p], kt[r], kh[r], kw[r]) * kslot_stride[p]
                       : a.rp.n_entries;
        kv = rotate_chunk(kv, tab, idx);
        // advance this row's coordinates by BN tokens for the next tile
        kw[r] += a.step_w;
        kh[r] += a.step_h;
        kt[r] += a.step_t;
        if (kw[r] >= a.rp.gw) { kw[r] -= a.rp.gw; kh[r] += 1; }
        if (kh[r] >= a.rp.gh) { kh[r] -= a.rp.gh; kt[r] += 1; }
      }
      *reinterpret_cast<uint4*>(buf + k_off(row, kc)) = kv;
    }
  };

  auto store_v = [&](uint16_t* buf, const uint4 reg[2]) {
#pragma unroll
    for (int r = 0; r < 2; ++r) *reinterpret_cast<uint4*>(buf + v_off(kr0 + 32 * r, kc)) = reg[r];
  };

  // per-lane LDS element offsets of the MFMA operands
  int koff[8];
#pragma unroll
  for (int st = 0; st < 8; ++st) koff[st] = k_off(l32, 2 * st + hi);
  // V^T via transposing reads: lane (h, g, i) = (hi, (lane >> 4) & 1, lane & 15)
  // reads 4 d-values of key row 16 ks + 8 r + 4 h + i/4 at d = 32 mb + 16 g + 4 (i & 3).
  const int vi = lane & 15;
  const int vg = (lane >> 4) & 1;
  const int vrow = 4 * hi + (vi >> 2);
  int voff[4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) voff[mb] = v_off(vrow, 4 * mb + 2 * vg + ((vi & 3) >> 1)) + 4 * (vi & 1);

  auto qk = [&](const uint16_t* kb, f32x16 s[2]) {
    s[0] = f32x16{};
    s[1] = f32x16{};
#pragma unroll
    for (int st = 0; st < 8; ++st) {
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) {
        const bf16x8 kop = *reinterpret_cast<const bf16x8*>(kb + koff[st] + blk * 32 * D);
        s[blk] = mfma32(kop, qreg[st], s[blk]);
      }
    }
  };

  f32x16 oacc[4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) oacc[mb] = f32x16{};
  float mref = -INFINITY;  // reference max (log2 units), identical in both lane halves
  float lsum = 0.f;        // this lane half's partial sum of p
  const float c2 = a.c2;
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  // row max of a score tile, rescale of the running output when it grew
  auto update_max = [&](const f32x16 s[2]) {
    float mx = fmaxf(s[0][0], s[0][1]);
#pragma unroll
    for (int i = 2; i < 16; ++i) mx = fmaxf(mx, s[0][i]);
#pragma unroll
    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[1][i]);
    mx = wave_half_max(mx) * c2;
    if (__builtin_amdgcn_ballot_w64(mx > mref + kRescaleThreshold) != 0) {
      const float mnew = fmaxf(mref, mx);
      const float alpha = __builtin_amdgcn_exp2f(mref - mnew);
      lsum *= alpha;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[mb][i] *= alpha;
      mref = mnew;
    }
  };

  auto softmax_p = [&](const f32x16 s[2], bf16x8 pop[4]) {
    const float nm = -mref;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      uint32_t pw[4];
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(s[ks >> 1][8 * (ks & 1) + e], c2, nm));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(s[ks >> 1][8 * (ks & 1) + e + 1], c2, nm));
        pw[e >> 1] = pack_bf16x2(p0, p1);
        lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw[e >> 1]), ones, lsum, false);
      }
      pop[ks] = __builtin_bit_cast(bf16x8, make_uint4(pw[0], pw[1], pw[2], pw[3]));
    }
  };

  auto pv = [&](const uint16_t* vb, const bf16x8 pop[4]) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const i16x4 lo = lds_read_tr16(vb + voff[mb] + (16 * ks) * D);
        const i16x4 hi4 = lds_read_tr16(vb + voff[mb] + (16 * ks + 8) * D);
        const bf16x8 vop = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi4, 0, 1, 2, 3, 4, 5, 6, 7));
        oacc[mb] = mfma32(vop, pop[ks], oacc[mb]);
      }
    }
  };

  // ---- prologue: K0, V0 and K1 in LDS, scores of tile 0
  {
    uint4 k0[2], v0[2], k1[2];
    load_rows(kbh, 0, k0);
    load_rows(vbh, 0, v0);
    load_rows(kbh, 1, k1);
    store_k(0, Ks[0], k0);
    store_v(Vs[0], v0);
    store_k(1, Ks[1], k1);
  }
  __syncthreads();

  f32x16 sa[2], sb[2];
  qk(Ks[0], sa);

  // one pipelined step: tile j's softmax + PV while tile j+1's scores run,
  // staging K_{j+2} and V_{j+1}
  auto step = [&](int j, f32x16 scur[2], f32x16 snext[2]) {
    uint4 kn[2], vn[2];
    load_rows(kbh, j + 2, kn);
    load_rows(vbh, j + 1, vn);
    update_max(scur);
    bf16x8 pop[4];
    qk(Ks[(j + 1) & 1], snext);
    softmax_p(scur, pop);
    pv(Vs[j & 1], pop);
    store_k(j + 2, Ks[j & 1], kn);
    store_v(Vs[(j + 1) & 1], vn);
    __syncthreads();
  };

  int j = 0;
  for (; j + 2 < ntiles; j += 2) {
    step(j, sa, sb);
    step(j + 1, sb, sa);
  }
  f32x16* slast = sa;
  if (j + 1 < ntiles) {
    step(j, sa, sb);
    ++j;
    slast = sb;
  }

  // ---- last tile: mask keys >= lv, softmax, PV
  {
    f32x16 s[2] = {slast[0], slast[1]};
    if (j * BN + BN > lv) {
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = j * BN + blk * 32 + 8 * (i >> 2) + 4 * hi + (i & 3);
          if (key >= lv) s[blk][i] = -INFINITY;
        }
    }
    update_max(s);
    bf16x8 pop[4];
    softmax_p(s, pop);
    pv(Vs[j & 1], pop);
  }

  // ---- epilogue: O = O^T / l, lane holds query qrow, d = 32 mb + 8 g + 4 hi + (0..3)
  const float l = wave_half_sum(lsum);
  const float inv = 1.0f / l;
  if (qlive) {
    uint16_t* orow = obh + (size_t)qrow * tok;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = mb * 32 + 8 * g + 4 * hi;
        uint2 pk;
        pk.x = pack_bf16x2(oacc[mb][4 * g + 0] * inv, oacc[mb][4 * g + 1] * inv);
        pk.y = pack_bf16x2(oacc[mb][4 * g + 2] * inv, oacc[mb][4 * g + 3] * inv);
        *reinterpret_cast<uint2*>(orow + d) = pk;
      }
    if (a.lse && hi == 0)
      a.lse[((size_t)b * a.H + h) * a.Lq + qrow] = (mref + __log2f(l)) * 0.69314718055994531f;
  }
}

}  // namespace

hipError_t launch_attn_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v, uint16_t* o,
                           float* lse, int B, int H, int Lq, int Lk, float scale,
                           const int32_t* kv_valid_len, const RopeParams& rp, hipStream_t stream) {
  AttnArgs a;
  a.q = q; a.k = k; a.v = v; a.o = o; a.lse = lse; a.kv_valid_len = kv_valid_len;
  a.B = B; a.H = H; a.Lq = Lq; a.Lk = Lk;
  a.nqt = (Lq + BM - 1) / BM;
  const long nwg = (long)a.nqt * B * H;
  a.nwg = (int)nwg;
  // p = exp2(c2 * (qsign q).k - m): |scale| goes into the exponent, its sign into q
  a.c2 = scale == 0.f ? 1.f : fabsf(scale) * 1.4426950408889634f;
  a.qsign = scale > 0.f ? 1.f : (scale < 0.f ? -1.f : 0.f);
  a.rp = rp;
  a.step_t = a.step_h = a.step_w = 0;
  if (rp.enabled) {
    a.step_w = BN % rp.gw;
    a.step_h = (BN / rp.gw) % rp.gh;
    a.step_t = BN / (rp.gw * rp.gh);
  }
  if (rp.enabled)
    hipLaunchKernelGGL(attn_fwd_kernel<true>, dim3((unsigned)nwg), dim3(NT), 0, stream, a);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<false>, dim3((unsigned)nwg), dim3(NT), 0, stream, a);
  return hipGetLastError();
}

}  // namespace vidax
