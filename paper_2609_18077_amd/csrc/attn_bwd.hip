// Attention backward for gfx950: the gradient of o = softmax(scale q k^T) v
// (non-causal, per-batch valid-key prefix) for a given dO, from the forward's
// output O and natural-log sum-exp.  bf16 in/out, fp32 accumulation, head
// dim 128.  With P = exp(scale q k^T - lse):
//
//   D_i = <dO_i, O_i>            dq kernel, from the own rows' dO (loaded
//                                  anyway) and O; written for the dkdv kernel
//   dQ  = scale dS K             dq kernel: one query tile per workgroup,
//                                  streaming K and V tiles
//   dV  = P^T dO, dK = scale dS^T Q   dkdv kernel: one key tile per
//                                  workgroup, streaming Q and dO tiles
//   dS  = P * (dO V^T - D)
//
// Both matrix kernels stream tiles of 64 rows straight from global memory
// into LDS (buffer loads with the LDS flag), two buffers per tensor, one
// barrier per tile, and keep the tiles as 256-byte rows with XOR-permuted
// 16-byte chunks (the row layout at the dq kernel), which every operand read
// -- 16-byte row reads and the transposing ds_read_b64_tr_b16 -- hits without
// bank conflicts.  The dq kernel follows the forward kernel's formulation:
// a wave's 32 own queries (q and dO) stay in registers as the B operand of
// v_mfma_f32_32x32x16_bf16, the K and V rows are the A operand, S^T and dP^T
// land in accumulators whose lanes each hold one query, and dS^T, converted
// to bf16 in place, is the B operand of dQ^T += K^T dS^T with K^T from the
// transposing read of the same K tile, in the matching key order.  The dkdv
// kernel computes both key gradients from one pass over the queries with 16
// own keys per wave and 16 x 16 x 32 products (both accumulators then fit a
// wave's registers at two waves per SIMD); its description is at the kernel.
#include <type_traits>

#include <mutex>

#include "launch.hpp"

namespace vidax {
namespace {

constexpr int D = kHeadDim;
constexpr int BN = 64;        // rows per streamed tile
constexpr int NW = 8;         // waves of a dkdv workgroup
constexpr int NT = NW * 64;   // its threads
constexpr int kBufferFlags = 0x00020000;  // raw buffer, 32-bit data format
constexpr float kLog2e = 1.4426950408889634f;

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr;

struct BwdArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* o;
  const uint16_t* dout;
  const float* lse;
  float* delta;
  uint16_t* dq;
  uint16_t* dk;
  uint16_t* dv;
  const int32_t* kv_valid_len;
  int B, H, Lq, Lk;
  float scale;
  float c;    // scale * log2(e)
  int ntile;  // own-row tiles per (b, h) of the launched kernel
  int nwg;    // workgroups of the launched kernel
  // key-side kernels: the query stream is cut into qsplit runs of qper
  // 64-row tiles, one workgroup each; with qsplit > 1 each writes its fp32
  // partial dK or dV to part ([qsplit][B][Lk][H][d], dV after dK) and the
  // reduce kernel sums them
  int qsplit, qper;
  float* part;
};

[[maybe_unused]] __device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ i16x4 lds_read_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
}

// Sum over lanes l and l ^ 32.
__device__ __forceinline__ float half_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Workgroups are dispatched round-robin over the 8 XCDs: give each XCD a
// contiguous range of logical tiles (own-row tiles of one (b, h) together).
__device__ __forceinline__ int logical_tile(int i, int n) {
  const int per = n >> 3, rem = n & 7, xcd = i & 7, kk = i >> 3;
  return xcd < rem ? xcd * (per + 1) + kk : rem * (per + 1) + (xcd - rem) * per + kk;
}

// Lv of batch b (uniform).
__device__ __forceinline__ int valid_keys(const BwdArgs& a, int b) {
  int lv = a.Lk;
  if (a.kv_valid_len) lv = min(max(a.kv_valid_len[b], 0), a.Lk);
  return __builtin_amdgcn_readfirstlane(lv);
}

// Buffer resource of 64-row tile `tile` of rows [0, limit): later rows read
// as zero (and land in LDS as zero).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const uint16_t* base, int tile, int limit, int tok) {
  const int rows = min(max(limit - tile * BN, 0), BN);
  const int nbytes = __builtin_amdgcn_readfirstlane(rows * tok * 2);
  return __builtin_amdgcn_make_buffer_rsrc((void*)(base + (size_t)tile * BN * tok), (short)0, nbytes, kBufferFlags);
}

// B operand of the wave's own row: chunks 2 s + hi (s = 0..7) of the row at
// p (zero when !live).
__device__ __forceinline__ void own_operand(const uint16_t* p, bool live, int hi, bf16x8 op[8]) {
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    uint4 x = make_uint4(0, 0, 0, 0);
    if (live) x = *reinterpret_cast<const uint4*>(p + (2 * s + hi) * 8);
    op[s] = __builtin_bit_cast(bf16x8, x);
  }
}

// A 32 x 32 fp32 accumulator (tile rows x own rows) -> two bf16 B operands of
// 16 tile rows each, in the accumulator's row order.
[[maybe_unused]] __device__ __forceinline__ void pack_ops(const f32x16& x, bf16x8 op[2]) {
#pragma unroll
  for (int k2 = 0; k2 < 2; ++k2) {
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 8; e += 2) w[e >> 1] = pack_bf16x2(x[8 * k2 + e], x[8 * k2 + e + 1]);
    op[k2] = __builtin_bit_cast(bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
  }
}

// Tile row (0..63) of register i of accumulator blk for lane half hi.
[[maybe_unused]] __device__ __forceinline__ int acc_row(int blk, int i, int hi) { return 32 * blk + 8 * (i >> 2) + 4 * hi + (i & 3); }

// Own row `row` of the wave (lane holds it), d = 32 mb + 8 g + 4 hi + (0..3):
// acc^T * mul -> bf16, 8-byte stores.
__device__ __forceinline__ void store_own(uint16_t* p, const f32x16 acc[4], float mul, int hi) {
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint2 pk;
      pk.x = pack_bf16x2(acc[mb][4 * g + 0] * mul, acc[mb][4 * g + 1] * mul);
      pk.y = pack_bf16x2(acc[mb][4 * g + 2] * mul, acc[mb][4 * g + 3] * mul);
      *reinterpret_cast<uint2*>(p + mb * 32 + 8 * g + 4 * hi) = pk;
    }
}

// ---- dQ: one tile of 32 NWQ queries of one (b, h) per workgroup of NWQ
// waves: 8 for long key sequences, 4 for short ones (two workgroups then
// share a CU, so that one's start and end overlap the other's products --
// with few key tiles per workgroup those dominate).  K and V tiles of 64 keys
// in the swizzled row layout (see below), double-buffered:
//   S^T = K Q^T, dP^T = V dO^T (A: key rows, one 16-byte read), P^T =
//   exp2(S^T c - lse log2 e), dS^T = P^T (dP^T - D), dQ^T += K^T dS^T (A: the
//   transposing read of the same K tile: 4 keys x 16 d per 16-lane group, in
//   the key order of the dS^T operand taken from the accumulator).
constexpr int STILE = BN * D;  // elements of a swizzled tile
// key tiles at or below which the dq workgroups have 4 waves instead of 8
constexpr int kDqShortTiles = 16;

// Tiles of 64 rows sit in LDS as 256-byte rows whose 16-byte chunks are
// permuted: chunk c of row r at position c ^ swz(r), swz linear in the bits
// of r & 15 (bit 0 -> 2, bit 1 -> 4, bit 2 -> 9, bit 3 -> 8), found by
// exhaustive search: the rows of every operand read of the dq and dkdv
// kernels then fall on distinct banks, whether the LDS serves 128 or 256
// bytes a cycle.  Copy j of a tile fills rows 4 j .. 4 j + 3: lane l writes
// position l & 15 of row 4 j + (l >> 4), fetching its chunk (l & 15) ^
// swz(row) (each row read whole, 256 contiguous bytes).
__device__ __forceinline__ int swz(int r) { return ((r & 3) << 1) ^ ((r & 4) ? 9 : 0) ^ (r & 8); }

template <int NWQ>
__device__ __forceinline__ void dq_body(const BwdArgs& a) {
  constexpr int BWQ = NWQ * 32;       // queries per workgroup
  constexpr int NCOPY = 16 / NWQ;     // copies per wave of a tile (16 of 4 rows)
  __shared__ __attribute__((aligned(16))) uint16_t K0[STILE], K1[STILE], V0[STILE], V1[STILE];
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lid = logical_tile(blockIdx.x, a.nwg);
  const int qt = lid % a.ntile, bh = lid / a.ntile, h = bh % a.H, b = bh / a.H;
  const int tok = a.H * D, rbytes = tok * 2;
  const int lv = valid_keys(a, b);
  const int qrow = qt * BWQ + wave * 32 + l32;
  const bool qlive = qrow < a.Lq;
  const size_t rowoff = ((size_t)b * a.Lq + (qlive ? qrow : 0)) * tok + (size_t)h * D;
  uint16_t* dqp = a.dq + rowoff;
  const size_t lrow = ((size_t)b * a.H + h) * a.Lq + (qlive ? qrow : 0);
  bf16x8 dop[8];
  own_operand(a.dout + rowoff, qlive, hi, dop);
  // D of the own row: this lane half's 64 products <dO, O>, then the other
  // half's; stored for the dkdv kernel (every row, also without valid keys)
  float dl;
  {
    bf16x8 oop[8];
    own_operand(a.o + rowoff, qlive, hi, oop);
    // packed bf16 pair products, two fp32 chains
    float sum[2] = {0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const uint4 x = __builtin_bit_cast(uint4, dop[s]), y = __builtin_bit_cast(uint4, oop[s]);
      const uint32_t xw[4] = {x.x, x.y, x.z, x.w}, yw[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
      for (int p = 0; p < 4; ++p)
        sum[p & 1] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, xw[p]), __builtin_bit_cast(bf16x2, yw[p]),
                                                     sum[p & 1], false);
    }
    dl = half_sum(sum[0] + sum[1]);
    if (qlive && hi == 0) a.delta[lrow] = dl;
  }
  f32x16 acc[4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) acc[mb] = f32x16{};
  if (lv == 0) {  // no valid key: dQ = 0
    if (qlive) store_own(dqp, acc, 0.f, hi);
    return;
  }
  bf16x8 qop[8];
  own_operand(a.q + rowoff, qlive, hi, qop);
  const float lse2 = qlive ? a.lse[lrow] * kLog2e : INFINITY;  // dead rows: P = 0

  const uint16_t* kbh = a.k + (size_t)b * a.Lk * tok + (size_t)h * D;
  const uint16_t* vbh = a.v + (size_t)b * a.Lk * tok + (size_t)h * D;
  const int ntiles = (lv + BN - 1) / BN;
  // the wave's copies NCOPY wave .. + NCOPY - 1 of a tile: byte offsets from its first row
  int cg[NCOPY];
#pragma unroll
  for (int u = 0; u < NCOPY; ++u) {
    const int row = 4 * (NCOPY * wave + u) + (lane >> 4);
    cg[u] = row * rbytes + ((lane & 15) ^ swz(row)) * 16;
  }
  auto copies = [&](int j, uint16_t* kb, uint16_t* vb) __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t rk = tile_rsrc(kbh, j, lv, tok);
    const __amdgpu_buffer_rsrc_t rv = tile_rsrc(vbh, j, lv, tok);
#pragma unroll
    for (int u = 0; u < NCOPY; ++u) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_ptr)(kb + (NCOPY * wave + u) * 512), 16, cg[u], 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_ptr)(vb + (NCOPY * wave + u) * 512), 16, cg[u], 0, 0, 0);
    }
  };
  // per-lane LDS element offsets:
  //   key-row operand, key row l32 (+ 32 blk), d = 16 st + 8 hi: chunk 2 st +
  //     hi at 2 (st ^ (swz >> 1)) + (hi ^ (swz & 1));
  //   K^T operand (transposing reads h = 0, 1 of 16-key step ks), key row
  //     16 ks + 8 h + 4 hi + (w >> 2), d = 32 mb + 16 (g & 1) + 4 (w & 3) for
  //     lane l = 16 g + w.
  int rk[8], tk[2][4];
  {
    const int fr = swz(l32);
#pragma unroll
    for (int st = 0; st < 8; ++st) rk[st] = l32 * D + 8 * (hi ^ (fr & 1)) + 16 * (st ^ (fr >> 1));
    const int g = lane >> 4, w = lane & 15, cc = w & 3;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int row = 8 * hh + 4 * hi + (w >> 2), ft = swz(row);
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
        tk[hh][mb] = row * D + 32 * (mb ^ (ft >> 2)) + 8 * ((2 * (g & 1) + (cc >> 1)) ^ (ft & 3)) + 4 * (cc & 1);
    }
  }
  copies(0, K0, V0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  auto step = [&](auto par, int j) __attribute__((always_inline)) {
    constexpr int P = decltype(par)::value;
    const uint16_t* kt = P ? K1 : K0;
    const uint16_t* vt = P ? V1 : V0;
    if (j + 1 < ntiles) copies(j + 1, P ? K0 : K1, P ? V0 : V1);
    const bool tail = j * BN + BN > lv;
    // one 32-key block at a time: fewer live registers, and the products of
    // the second block overlap the first block's exponentials
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
      for (int st = 0; st < 8; ++st) {
        s = mfma32(*reinterpret_cast<const bf16x8*>(kt + 32 * blk * D + rk[st]), qop[st], s);
        dp = mfma32(*reinterpret_cast<const bf16x8*>(vt + 32 * blk * D + rk[st]), dop[st], dp);
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) s[i] = __builtin_amdgcn_exp2f(fmaf(s[i], a.c, -lse2)) * (dp[i] - dl);
      if (tail) {  // uniform: only the last, ragged key tile; keys past Lv get dS = 0
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (j * BN + acc_row(blk, i, hi) >= lv) s[i] = 0.f;
      }
      bf16x8 dsop[2];
      pack_ops(s, dsop);
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const int ks = 2 * blk + k2;
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
          const i16x4 lo = lds_read_tr16(kt + 16 * ks * D + tk[0][mb]);
          const i16x4 up = lds_read_tr16(kt + 16 * ks * D + tk[1][mb]);
          acc[mb] = mfma32(__builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, up, 0, 1, 2, 3, 4, 5, 6, 7)),
                           dsop[k2], acc[mb]);
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0);  // this wave's copies have landed
    __syncthreads();
  };
  using even = std::integral_constant<int, 0>;
  using odd = std::integral_constant<int, 1>;
  int j = 0;
  for (; j + 1 < ntiles; j += 2) {
    step(even(), j);
    step(odd(), j + 1);
  }
  if (j < ntiles) step(even(), j);
  if (qlive) store_own(dqp, acc, a.scale, hi);
}

// 4 waves (128 queries) a workgroup where the key sequence is short, 8
// waves (256 queries) otherwise.
__global__ __launch_bounds__(256, 2) void bwd_dq4_kernel(BwdArgs a) { dq_body<4>(a); }
__global__ __launch_bounds__(512) void bwd_dq8_kernel(BwdArgs a) { dq_body<8>(a); }

// ---- dK and dV together: one tile of 128 keys of one (b, h) per workgroup,
// 16 keys per wave, with v_mfma_f32_16x16x32_bf16 (A: lane l holds row l % 16,
// k = 8 (l / 16) .. + 7; B: column l % 16, the same k; C: column l % 16, rows
// 4 (l / 16) .. + 3).  Per 64-query tile and query block r (16 queries):
//   S[r] = Q K^T, dP[r] = dO V^T  (A: Q / dO rows from the padded row tile,
//     one 16-byte read; B: the wave's own k / v rows in registers)
//   P = exp2(S c - lse log2 e), dS = P (dP - D)   (lane: key column, 4 queries)
//   dV^T += dO^T P, dK^T += Q^T dS over k-steps of 32 queries  (A: the
//     transposing read of the same padded row tile, 4 queries x 16 d per
//     16-lane group; B: P / dS, whose k order -- queries 32 s + 4 g .. + 3,
//     then 32 s + 16 + 4 g .. + 3 for lane group g -- the two reads match).
// Both accumulators (64 registers) and k, v (32) fit in a wave's 256
// registers at two waves per SIMD; each query tile is copied once per
// tensor.
// Tiles of 64 query rows in the swizzled row layout of the dq kernel.
constexpr int BK = 128;  // keys per workgroup
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__global__ __launch_bounds__(NT) void bwd_dkdv_kernel(BwdArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t Qk0[STILE], Qk1[STILE], Ok0[STILE], Ok1[STILE];
  __shared__ __attribute__((aligned(16))) float Lt[2][BN], Dt[2][BN];
  const int tid = threadIdx.x, lane = tid & 63, c16 = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lid = logical_tile(blockIdx.x, a.nwg);
  const int kt = lid % a.ntile, sbh = lid / a.ntile, sp = sbh % a.qsplit, bh = sbh / a.qsplit;
  const int h = bh % a.H, b = bh / a.H;
  const int tok = a.H * D, rbytes = tok * 2;
  const int lv = valid_keys(a, b);
  const int krow = kt * BK + wave * 16 + c16;
  const bool klive = krow < a.Lk;
  const bool kvalid = krow < lv;
  const bool wlive = kt * BK + wave * 16 < lv;  // uniform
  const size_t rowoff = ((size_t)b * a.Lk + (klive ? krow : 0)) * tok + (size_t)h * D;
  f32x4 dk[8], dv[8];
#pragma unroll
  for (int mb = 0; mb < 8; ++mb) dk[mb] = dv[mb] = f32x4{};
  // own row: lane holds key krow, d = 16 mb + 4 g .. + 3 of block mb
  auto finish = [&](float mulk) __attribute__((always_inline)) {
    if (!klive) return;
    if (a.qsplit > 1) {
      const size_t n = (size_t)a.B * a.Lk * tok;
      float* pk = a.part + (size_t)sp * n + rowoff;
      float* pv = a.part + (size_t)(a.qsplit + sp) * n + rowoff;
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) {
        *reinterpret_cast<float4*>(pk + 16 * mb + 4 * g) = make_float4(dk[mb][0], dk[mb][1], dk[mb][2], dk[mb][3]);
        *reinterpret_cast<float4*>(pv + 16 * mb + 4 * g) = make_float4(dv[mb][0], dv[mb][1], dv[mb][2], dv[mb][3]);
      }
    } else {
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) {
        uint2 x, y;
        x.x = pack_bf16x2(dk[mb][0] * mulk, dk[mb][1] * mulk);
        x.y = pack_bf16x2(dk[mb][2] * mulk, dk[mb][3] * mulk);
        y.x = pack_bf16x2(dv[mb][0], dv[mb][1]);
        y.y = pack_bf16x2(dv[mb][2], dv[mb][3]);
        *reinterpret_cast<uint2*>(a.dk + rowoff + 16 * mb + 4 * g) = x;
        *reinterpret_cast<uint2*>(a.dv + rowoff + 16 * mb + 4 * g) = y;
      }
    }
  };
  if (kt * BK >= lv) {  // no valid key in this workgroup: zero gradient
    finish(0.f);
    return;
  }
  // own k, v as B operands: lane holds key krow, d = 32 st + 8 g .. + 7
  bf16x8 kop[4], vop[4];
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    uint4 x = make_uint4(0, 0, 0, 0), y = x;
    if (klive) {
      x = *reinterpret_cast<const uint4*>(a.k + rowoff + 32 * st + 8 * g);
      y = *reinterpret_cast<const uint4*>(a.v + rowoff + 32 * st + 8 * g);
    }
    kop[st] = __builtin_bit_cast(bf16x8, x);
    vop[st] = __builtin_bit_cast(bf16x8, y);
  }

  const uint16_t* qbh = a.q + (size_t)b * a.Lq * tok + (size_t)h * D;
  const uint16_t* obh = a.dout + (size_t)b * a.Lq * tok + (size_t)h * D;
  const float* lseb = a.lse + ((size_t)b * a.H + h) * a.Lq;
  const float* delb = a.delta + ((size_t)b * a.H + h) * a.Lq;
  // the wave's copies 2 wave, 2 wave + 1 of a tile: byte offsets from its first row
  int cg[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int row = 4 * (2 * wave + u) + (lane >> 4);
    cg[u] = row * rbytes + (c16 ^ swz(row)) * 16;
  }
  auto copy_tile = [&](__amdgpu_buffer_rsrc_t rs, uint16_t* buf) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 2; ++u)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr)(buf + (2 * wave + u) * 512), 16, cg[u], 0, 0, 0);
  };
  const int t0 = sp * a.qper;
  const int t1 = min(t0 + a.qper, (a.Lq + BN - 1) / BN);
  float lrow = INFINITY, drow = 0.f;
  auto copies = [&](int t, uint16_t* qk, uint16_t* ok) __attribute__((always_inline)) {
    copy_tile(tile_rsrc(qbh, t, a.Lq, tok), qk);
    copy_tile(tile_rsrc(obh, t, a.Lq, tok), ok);
    if (tid < BN) {
      const int r = t * BN + tid;
      lrow = r < a.Lq ? lseb[r] : INFINITY;
      drow = r < a.Lq ? delb[r] : 0.f;
    }
  };
  auto put_rows = [&](int buf) __attribute__((always_inline)) {
    if (tid < BN) {
      Lt[buf][tid] = lrow * kLog2e;
      Dt[buf][tid] = drow;
    }
  };
  if (t0 >= t1) {
    finish(0.f);
    return;
  }
  copies(t0, Qk0, Ok0);
  put_rows(0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // per-lane LDS element offsets (rows of a 16-row block share swz):
  //   row operand, query row 16 r + c16, d = 32 st + 8 g: chunk 4 st + g,
  //     placed at 4 (st ^ (swz >> 2)) + ((g ^ swz) & 3);
  //   transposing read, query row 4 g + (c16 >> 2) of a 16-row block, d =
  //     16 mb + 4 (c16 & 3): 8 bytes of chunk pair mb, placed at pair
  //     mb ^ (swz >> 1), chunk ((c16 >> 1) & 1) ^ (swz & 1) of the pair.
  int roff[4], toff[8];
  {
    const int fr = swz(c16);
#pragma unroll
    for (int st = 0; st < 4; ++st) roff[st] = c16 * D + 8 * (4 * (st ^ (fr >> 2)) + ((g ^ fr) & 3));
    const int tr = 4 * g + (c16 >> 2), ft = swz(tr), cc = c16 & 3;
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) toff[mb] = tr * D + 16 * (mb ^ (ft >> 1)) + 8 * ((cc >> 1) ^ (ft & 1)) + 4 * (cc & 1);
  }
  auto step = [&](auto par, int t) __attribute__((always_inline)) {
    constexpr int P = decltype(par)::value;
    const uint16_t* qt = P ? Qk1 : Qk0;
    const uint16_t* ot = P ? Ok1 : Ok0;
    if (t + 1 < t1) copies(t + 1, P ? Qk0 : Qk1, P ? Ok0 : Ok1);
    if (wlive) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        f32x4 sc[2], dp[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int r = 2 * s + u;
          sc[u] = dp[u] = f32x4{};
#pragma unroll
          for (int st = 0; st < 4; ++st) {
            const bf16x8 qa = *reinterpret_cast<const bf16x8*>(qt + 16 * r * D + roff[st]);
            const bf16x8 oa = *reinterpret_cast<const bf16x8*>(ot + 16 * r * D + roff[st]);
            sc[u] = mfma16(qa, kop[st], sc[u]);
            dp[u] = mfma16(oa, vop[st], dp[u]);
          }
        }
        // P and dS of queries 16 r + 4 g + i (i = 0..3), r = 2 s + u
        uint32_t pw[4], dw[4];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int r0 = 16 * (2 * s + u) + 4 * g;
          const float4 l4 = *reinterpret_cast<const float4*>(&Lt[P][r0]);
          const float4 d4 = *reinterpret_cast<const float4*>(&Dt[P][r0]);
          const float lr[4] = {l4.x, l4.y, l4.z, l4.w}, dr[4] = {d4.x, d4.y, d4.z, d4.w};
          float pp[4], dd[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            pp[i] = kvalid ? __builtin_amdgcn_exp2f(fmaf(sc[u][i], a.c, -lr[i])) : 0.f;
            dd[i] = pp[i] * (dp[u][i] - dr[i]);
          }
          pw[2 * u] = pack_bf16x2(pp[0], pp[1]);
          pw[2 * u + 1] = pack_bf16x2(pp[2], pp[3]);
          dw[2 * u] = pack_bf16x2(dd[0], dd[1]);
          dw[2 * u + 1] = pack_bf16x2(dd[2], dd[3]);
        }
        const bf16x8 pb = __builtin_bit_cast(bf16x8, make_uint4(pw[0], pw[1], pw[2], pw[3]));
        const bf16x8 db = __builtin_bit_cast(bf16x8, make_uint4(dw[0], dw[1], dw[2], dw[3]));
        // dV^T += dO^T P, dK^T += Q^T dS over queries 32 s .. 32 s + 31
#pragma unroll
        for (int mb = 0; mb < 8; ++mb) {
          const int o0 = 32 * s * D + toff[mb];
          const i16x4 olo = lds_read_tr16(ot + o0), ohi = lds_read_tr16(ot + o0 + 16 * D);
          const i16x4 qlo = lds_read_tr16(qt + o0), qhi = lds_read_tr16(qt + o0 + 16 * D);
          dv[mb] = mfma16(__builtin_bit_cast(bf16x8, __builtin_shufflevector(olo, ohi, 0, 1, 2, 3, 4, 5, 6, 7)), pb, dv[mb]);
          dk[mb] = mfma16(__builtin_bit_cast(bf16x8, __builtin_shufflevector(qlo, qhi, 0, 1, 2, 3, 4, 5, 6, 7)), db, dk[mb]);
        }
      }
    }
    if (t + 1 < t1) put_rows(1 - P);
    __builtin_amdgcn_s_waitcnt(0);  // this wave's copies have landed
    __syncthreads();
  };
  using even = std::integral_constant<int, 0>;
  using odd = std::integral_constant<int, 1>;
  int t = t0;
  for (; t + 1 < t1; t += 2) {
    step(even(), t);
    step(odd(), t + 1);
  }
  if (t < t1) step(even(), t);
  finish(a.scale);
}

// ---- dK = scale * sum of the partials, dV = sum of the partials (qsplit >
// 1): 8 consecutive d values of one (b, key, h) row per thread.
__global__ __launch_bounds__(256) void bwd_reduce_kernel(BwdArgs a) {
  const size_t n = (size_t)a.B * a.Lk * a.H * D;  // elements per gradient
  const size_t groups = n / 8;
  for (size_t g = (size_t)blockIdx.x * 256 + threadIdx.x; g < 2 * groups; g += (size_t)gridDim.x * 256) {
    const bool isk = g < groups;
    const size_t e = (isk ? g : g - groups) * 8;
    const float* src = a.part + (isk ? 0 : (size_t)a.qsplit * n) + e;
    float4 x0 = make_float4(0.f, 0.f, 0.f, 0.f), x1 = x0;
    for (int sp = 0; sp < a.qsplit; ++sp) {
      const float4 u = *reinterpret_cast<const float4*>(src + (size_t)sp * n);
      const float4 v = *reinterpret_cast<const float4*>(src + (size_t)sp * n + 4);
      x0.x += u.x; x0.y += u.y; x0.z += u.z; x0.w += u.w;
      x1.x += v.x; x1.y += v.y; x1.z += v.z; x1.w += v.w;
    }
    const float mul = isk ? a.scale : 1.f;
    uint4 o;
    o.x = pack_bf16x2(x0.x * mul, x0.y * mul);
    o.y = pack_bf16x2(x0.z * mul, x0.w * mul);
    o.z = pack_bf16x2(x1.x * mul, x1.y * mul);
    o.w = pack_bf16x2(x1.z * mul, x1.w * mul);
    *reinterpret_cast<uint4*>((isk ? a.dk : a.dv) + e) = o;
  }
}

}  // namespace

// Compute units of the current device (queried once per device).
int device_cu_count() {
  static std::mutex mu;
  static int counts[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  std::lock_guard<std::mutex> lock(mu);
  if (counts[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    counts[dev] = n;
  }
  return counts[dev];
}

hipError_t launch_attn_bwd(const uint16_t* q, const uint16_t* k, const uint16_t* v, const uint16_t* o,
                           const uint16_t* dout, const float* lse, float* ws, size_t ws_floats, uint16_t* dq,
                           uint16_t* dk, uint16_t* dv, int B, int H, int Lq, int Lk, float scale,
                           const int32_t* kv_valid_len, hipStream_t stream) {
  BwdArgs a;
  a.q = q; a.k = k; a.v = v; a.o = o; a.dout = dout; a.lse = lse; a.delta = ws;
  a.dq = dq; a.dk = dk; a.dv = dv; a.kv_valid_len = kv_valid_len;
  a.B = B; a.H = H; a.Lq = Lq; a.Lk = Lk;
  a.scale = scale;
  a.c = scale * kLog2e;
  BwdSplit sp = attn_bwd_split(B, H, Lq, Lk, device_cu_count());
  if (ws_floats < sp.floats) {  // too small a workspace for the split: run unsplit
    sp.qsplit = 1;
    sp.qper = (Lq + BN - 1) / BN;
  }
  a.qsplit = sp.qsplit;
  a.qper = sp.qper;
  a.part = sp.qsplit > 1 ? ws + sp.part_offset : nullptr;
  hipError_t e = hipSuccess;
  if (Lq > 0) {
    const bool short_keys = (Lk + BN - 1) / BN <= kDqShortTiles;
    const int nwq = short_keys ? 4 : 8;
    a.ntile = (Lq + 32 * nwq - 1) / (32 * nwq);
    a.nwg = a.ntile * B * H;
    e = short_keys ? launch_kernel(bwd_dq4_kernel, (unsigned)a.nwg, 256u, stream, a)
                   : launch_kernel(bwd_dq8_kernel, (unsigned)a.nwg, 512u, stream, a);
    if (e != hipSuccess) return e;
  }
  if (Lk > 0) {
    a.ntile = (Lk + BK - 1) / BK;
    a.nwg = a.ntile * B * H * a.qsplit;
    e = launch_kernel(bwd_dkdv_kernel, (unsigned)a.nwg, (unsigned)NT, stream, a);
    if (e != hipSuccess) return e;
    if (a.qsplit > 1) {
      const size_t groups = 2 * (size_t)B * Lk * H * D / 8;
      size_t g = (groups + 255) / 256;
      if (g > 16384) g = 16384;
      e = launch_kernel(bwd_reduce_kernel, (unsigned)g, 256u, stream, a);
    }
  }
  return e;
}

// ---- allocation-free backward ------------------------------------------
//
// D of the allocation-free entry point lives in this fixed array instead of a
// caller workspace: kNoAllocRows fp32 values (16 MiB), one copy per GPU the
// library runs on, held until the process ends.  In host code `scratch` is
// only a stand-in for the symbol; its device address (different on every
// GPU) is looked up once per device and only that address is handed to the
// kernels.  Calls that overlap on one GPU share the array and race; the dq
// kernel writes every value the dkdv kernel then reads, so nothing is
// cleared.
static __device__ __align__(256) float scratch[kNoAllocRows];

constexpr int kMaxDevices = 64;

// Device address of `scratch` on the current device (looked up on the first
// call made with that device current).
static hipError_t scratch_address(float** out) {
  static std::mutex mu;
  static float* addr[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    addr[dev] = static_cast<float*>(ptr);
  }
  *out = addr[dev];
  return hipSuccess;
}

hipError_t launch_attn_bwd_noalloc(const uint16_t* q, const uint16_t* k, const uint16_t* v, const uint16_t* o,
                                   const uint16_t* dout, const float* lse, uint16_t* dq, uint16_t* dk, uint16_t* dv,
                                   int B, int H, int Lq, int Lk, float scale, const int32_t* kv_valid_len,
                                   hipStream_t stream) {
  if ((long)B * H * Lq > kNoAllocRows) return hipErrorInvalidValue;  // the entry point rejects this first
  float* delta = nullptr;
  const hipError_t e = scratch_address(&delta);
  if (e != hipSuccess) return e;
  // D only (the array holds no room for split partials): unsplit
  return launch_attn_bwd(q, k, v, o, dout, lse, delta, (size_t)B * H * Lq, dq, dk, dv, B, H, Lq, Lk, scale,
                         kv_valid_len, stream);
}

}  // namespace vidax
