// Attention backward for gfx950: the gradient of o = softmax(scale q k^T) v
// (non-causal, per-batch valid-key prefix) for a given dO, from the forward's
// output O and natural-log sum-exp.  bf16 in/out, fp32 accumulation, head
// dim 128.  With P = exp(scale q k^T - lse):
//
//   D_i = <dO_i, O_i>            delta kernel (HBM-bound, one pass over dO, O)
//   dQ  = scale dS K             dq kernel: one query tile per workgroup,
//                                  streaming K and V tiles
//   dV  = P^T dO                 dv kernel: one key tile per workgroup,
//   dK  = scale dS^T Q           dk kernel:   streaming Q and dO tiles
//   dS  = P * (dO V^T - D)
//
// Each kernel has the forward kernel's shape and layouts: eight waves of 32
// own rows, tiles of 64 streamed rows copied straight into LDS (buffer loads
// with the LDS flag), two buffers per tile kind, one barrier per tile.  Tiles
// read row-wise are kept as padded rows (whole-row copies, lanes in address
// order); tiles read transposed are kept in MFMA operand order.  The own rows' vectors (q and dO in the dq kernel, k and
// v in the dk/dv kernels) stay in registers as the B operand of
// v_mfma_f32_32x32x16_bf16; the streamed tile is the A operand, read either
// row-wise (K order) or transposed by ds_read_b64_tr_b16 (V order).  The
// products of a 64-row tile with the wave's 32 own rows land in two 32 x 32
// accumulators whose lanes each hold one own row; converted to bf16 they are
// directly the B operand of the next product (P or dS against the other
// tile), with the row order inside each 16-row step matched by the
// transposing read -- as in the forward.  dK and dV have their own kernels
// because keeping both accumulators (and k, v, S, dP) in one wave needs more
// than the 256 registers a wave has at two waves per SIMD.
#include <type_traits>

#include <mutex>

#include "launch.hpp"

namespace vidax {
namespace {

constexpr int D = kHeadDim;
constexpr int BN = 64;        // rows per streamed tile
constexpr int NW = 8;         // waves per workgroup
constexpr int NT = NW * 64;   // threads
constexpr int BW = NW * 32;   // own rows per workgroup
constexpr int TILE = BN * D;  // elements per streamed tile in V order
constexpr int kRowPitch = 17 * 8;  // elements per row of a K-order tile (16 chunks + 1 padding)
constexpr int KTILE = BN * kRowPitch;  // elements per streamed tile in K order (17 KB)
constexpr int BLK = 512;      // elements per operand block (1 KB)
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
  int ntile;  // own-row tiles (of BW rows) per (b, h) of the launched kernel
  int nwg;    // workgroups of the launched kernel
  // key-side kernels: the query stream is cut into qsplit runs of qper
  // 64-row tiles, one workgroup each; with qsplit > 1 each writes its fp32
  // partial dK or dV to part ([qsplit][B][Lk][H][d], dV after dK) and the
  // reduce kernel sums them
  int qsplit, qper;
  float* part;
};

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ i16x4 lds_read_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
}

// Sum over the 16 lanes of a row (row rotations, then quad permutations).
__device__ __forceinline__ float row16_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x124, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4e, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xb1, 0xf, 0xf, false));
  return v;
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

// ---- streamed tiles (64 rows of a [B, L, H, 128] tensor for one (b, h)).
//   K order (read row-wise): row by row, each 256-byte row followed by 16
//     bytes of padding, so that every direct copy (64 lanes x 16 bytes into
//     consecutive slots) fetches whole rows with its lanes in address order
//     (coalesced; the padding slot reads past the records: zero, no memory
//     access) and the operand reads -- lane l: row 32 blk + (l & 31), chunk
//     2 st + (l >> 5) -- fall on distinct banks (rows 17 chunks apart).
// V order, in MFMA operand order, 16 blocks of 1 KB:
//   V order, block 4 ks + mb, half r: lane l's 8 bytes = row
//     16 ks + 8 r + 4 (l >> 5) + ((l & 15) >> 2), d = 32 mb + 16 ((l >> 4) & 1)
//     + 4 (l & 3) .. + 3  (what the transposing read of lane l fetches for
//     the A^T operand of d block mb, rows 16 ks .. 16 ks + 15)
// V order: wave w copies blocks 2w, 2w + 1 of a tile.  K order: copy j (of
// 17 a tile) fills 16-byte slots 64 j .. 64 j + 63, lane l slot s = 64 j + l =
// row s / 17, chunk s % 17 (16: padding); wave 0 issues copies 0..2, wave
// w > 0 copies 2 w + 1, 2 w + 2.  Lane offsets in bytes from the tile's first
// row:
struct Staging {
  int r[3];        // K-order copies
  int rfirst, rn;  // the wave's first K-order copy and their number
  int v0, v1;      // V-order blocks
};

__device__ __forceinline__ Staging staging(int wave, int lane, int rbytes) {
  const int hi = lane >> 5;
  Staging s;
  s.rfirst = wave == 0 ? 0 : 2 * wave + 1;
  s.rn = wave == 0 ? 3 : 2;
#pragma unroll
  for (int u = 0; u < 3; ++u) {
    const int sl = 64 * (s.rfirst + u) + lane, row = sl / 17, c = sl - 17 * row;
    s.r[u] = c < 16 ? row * rbytes + c * 16 : 0x7ffffff0;
  }
  const int vrow = 8 * hi + 4 * ((lane >> 4) & 1) + ((lane & 7) >> 1);
  const int vd = 16 * ((lane >> 3) & 1) + 8 * (lane & 1);
  const int b0 = 2 * wave, b1 = 2 * wave + 1;  // V blocks (ks, mb) = (b >> 2, b & 3)
  s.v0 = (vrow + 16 * (b0 >> 2)) * rbytes + 2 * (vd + 32 * (b0 & 3));
  s.v1 = (vrow + 16 * (b1 >> 2)) * rbytes + 2 * (vd + 32 * (b1 & 3));
  return s;
}

// Buffer resource of 64-row tile `tile` of rows [0, limit): later rows read
// as zero (and land in LDS as zero).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const uint16_t* base, int tile, int limit, int tok) {
  const int rows = min(max(limit - tile * BN, 0), BN);
  const int nbytes = __builtin_amdgcn_readfirstlane(rows * tok * 2);
  return __builtin_amdgcn_make_buffer_rsrc((void*)(base + (size_t)tile * BN * tok), (short)0, nbytes, kBufferFlags);
}

__device__ __forceinline__ void copy_blocks(__amdgpu_buffer_rsrc_t rs, uint16_t* buf, int wave, int g0, int g1) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr)(buf + (2 * wave) * BLK), 16, g0, 0, 0, 0);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr)(buf + (2 * wave + 1) * BLK), 16, g1, 0, 0, 0);
}

// the wave's K-order copies of a tile
__device__ __forceinline__ void copy_rows(__amdgpu_buffer_rsrc_t rs, uint16_t* buf, const Staging& sg) {
#pragma unroll
  for (int u = 0; u < 3; ++u)
    if (u < sg.rn)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr)(buf + (sg.rfirst + u) * 512), 16, sg.r[u], 0, 0, 0);
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

// acc = (tile rows 32 blk .. 32 blk + 31) x (own rows)^T over d, from a
// K-order tile.
__device__ __forceinline__ f32x16 rows_x_own(const uint16_t* t, const bf16x8 own[8], int blk, int lane) {
  f32x16 acc = f32x16{};
  const uint16_t* base = t + (32 * blk + (lane & 31)) * kRowPitch + 8 * (lane >> 5);
#pragma unroll
  for (int st = 0; st < 8; ++st) {
    const bf16x8 a = *reinterpret_cast<const bf16x8*>(base + 16 * st);
    acc = mfma32(a, own[st], acc);
  }
  return acc;
}

// acc[mb] += (tile^T, d block mb) x op over tile rows 32 blk .. 32 blk + 31,
// from a V-order tile (op[k2] holds rows 32 blk + 16 k2 .. + 15).
__device__ __forceinline__ void tr_x_op(const uint16_t* t, const bf16x8 op[2], int blk, f32x16 acc[4], int lane) {
#pragma unroll
  for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
      const int ks = 2 * blk + k2;
      const i16x4 lo = lds_read_tr16(t + (4 * ks + mb) * BLK + lane * 4);
      const i16x4 hi4 = lds_read_tr16(t + (4 * ks + mb) * BLK + BLK / 2 + lane * 4);
      const bf16x8 a = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi4, 0, 1, 2, 3, 4, 5, 6, 7));
      acc[mb] = mfma32(a, op[k2], acc[mb]);
    }
}

// A 32 x 32 fp32 accumulator (tile rows x own rows) -> two bf16 B operands of
// 16 tile rows each, in the accumulator's row order.
__device__ __forceinline__ void pack_ops(const f32x16& x, bf16x8 op[2]) {
#pragma unroll
  for (int k2 = 0; k2 < 2; ++k2) {
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 8; e += 2) w[e >> 1] = pack_bf16x2(x[8 * k2 + e], x[8 * k2 + e + 1]);
    op[k2] = __builtin_bit_cast(bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
  }
}

// Tile row (0..63) of register i of accumulator blk for lane half hi.
__device__ __forceinline__ int acc_row(int blk, int i, int hi) { return 32 * blk + 8 * (i >> 2) + 4 * hi + (i & 3); }

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

// Own row as fp32 (partial of a split run): 16-byte stores.
__device__ __forceinline__ void store_own_f32(float* p, const f32x16 acc[4], int hi) {
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int g = 0; g < 4; ++g)
      *reinterpret_cast<float4*>(p + mb * 32 + 8 * g + 4 * hi) =
          make_float4(acc[mb][4 * g + 0], acc[mb][4 * g + 1], acc[mb][4 * g + 2], acc[mb][4 * g + 3]);
}

// ---- D_i = <dO_i, O_i>: 16 lanes per row, fp32.  A workgroup takes 64
// consecutive rows i of one (b, h) (the order of D, so that 16 consecutive
// rows' results are one contiguous store), four rows per thread in flight.
constexpr int kDeltaRows = 4;
constexpr int kDeltaBlock = 16 * kDeltaRows;  // rows per workgroup
__global__ __launch_bounds__(256) void bwd_delta_kernel(BwdArgs a) {
  const int c = threadIdx.x & 15;
  const int nblk = (a.Lq + kDeltaBlock - 1) / kDeltaBlock;
  const int bh = blockIdx.x / nblk;
  const int i0 = (blockIdx.x - bh * nblk) * kDeltaBlock + (threadIdx.x >> 4);
  const int h = bh % a.H, b = bh / a.H;
  const size_t tok = (size_t)a.H * D;
  const uint16_t* dob = a.dout + (size_t)b * a.Lq * tok + (size_t)h * D + c * 8;
  const uint16_t* ob = a.o + (size_t)b * a.Lq * tok + (size_t)h * D + c * 8;
  uint4 x[kDeltaRows], y[kDeltaRows];
#pragma unroll
  for (int u = 0; u < kDeltaRows; ++u) {
    const int i = i0 + 16 * u;
    x[u] = y[u] = make_uint4(0, 0, 0, 0);
    if (i < a.Lq) {
      x[u] = *reinterpret_cast<const uint4*>(dob + (size_t)i * tok);
      y[u] = *reinterpret_cast<const uint4*>(ob + (size_t)i * tok);
    }
  }
#pragma unroll
  for (int u = 0; u < kDeltaRows; ++u) {
    const uint32_t xw[4] = {x[u].x, x[u].y, x[u].z, x[u].w}, yw[4] = {y[u].x, y[u].y, y[u].z, y[u].w};
    float sum = 0.f;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      sum = fmaf(bf16lo_to_f32(xw[p]), bf16lo_to_f32(yw[p]), sum);
      sum = fmaf(bf16hi_to_f32(xw[p]), bf16hi_to_f32(yw[p]), sum);
    }
    sum = row16_sum(sum);
    const int i = i0 + 16 * u;
    if (c == 0 && i < a.Lq) a.delta[(size_t)bh * a.Lq + i] = sum;
  }
}

// ---- dQ: one tile of 256 queries of one (b, h) per workgroup.
//   S^T = K Q^T, dP^T = V dO^T (K, V tiles in K order), P^T = exp2(S^T c -
//   lse log2 e), dS^T = P^T (dP^T - D), dQ^T += K^T dS^T (K tile in V order).
__global__ __launch_bounds__(NT) void bwd_dq_kernel(BwdArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t Kk0[KTILE], Kk1[KTILE], Vk0[KTILE], Vk1[KTILE], Kv0[TILE], Kv1[TILE];
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lid = logical_tile(blockIdx.x, a.nwg);
  const int qt = lid % a.ntile, bh = lid / a.ntile, h = bh % a.H, b = bh / a.H;
  const int tok = a.H * D, rbytes = tok * 2;
  const int lv = valid_keys(a, b);
  const int qrow = qt * BW + wave * 32 + l32;
  const bool qlive = qrow < a.Lq;
  const size_t rowoff = ((size_t)b * a.Lq + (qlive ? qrow : 0)) * tok + (size_t)h * D;
  uint16_t* dqp = a.dq + rowoff;
  f32x16 acc[4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) acc[mb] = f32x16{};
  if (lv == 0) {  // no valid key: dQ = 0
    if (qlive) store_own(dqp, acc, 0.f, hi);
    return;
  }
  bf16x8 qop[8], dop[8];
  own_operand(a.q + rowoff, qlive, hi, qop);
  own_operand(a.dout + rowoff, qlive, hi, dop);
  const size_t lrow = ((size_t)b * a.H + h) * a.Lq + (qlive ? qrow : 0);
  const float lse2 = qlive ? a.lse[lrow] * kLog2e : INFINITY;  // dead rows: P = 0
  const float dl = qlive ? a.delta[lrow] : 0.f;

  const uint16_t* kbh = a.k + (size_t)b * a.Lk * tok + (size_t)h * D;
  const uint16_t* vbh = a.v + (size_t)b * a.Lk * tok + (size_t)h * D;
  const Staging sg = staging(wave, lane, rbytes);
  const int ntiles = (lv + BN - 1) / BN;
  auto copies = [&](int j, uint16_t* kk, uint16_t* vk, uint16_t* kv) __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t rk = tile_rsrc(kbh, j, lv, tok);
    const __amdgpu_buffer_rsrc_t rv = tile_rsrc(vbh, j, lv, tok);
    copy_rows(rk, kk, sg);
    copy_rows(rv, vk, sg);
    copy_blocks(rk, kv, wave, sg.v0, sg.v1);
  };
  copies(0, Kk0, Vk0, Kv0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  auto step = [&](auto par, int j) __attribute__((always_inline)) {
    constexpr int P = decltype(par)::value;
    if (j + 1 < ntiles) copies(j + 1, P ? Kk0 : Kk1, P ? Vk0 : Vk1, P ? Kv0 : Kv1);
    const bool tail = j * BN + BN > lv;
    // one 32-key block at a time: fewer live registers, and the products of
    // the second block overlap the first block's exponentials
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      f32x16 s = rows_x_own(P ? Kk1 : Kk0, qop, blk, lane);
      const f32x16 dp = rows_x_own(P ? Vk1 : Vk0, dop, blk, lane);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float p = __builtin_amdgcn_exp2f(fmaf(s[i], a.c, -lse2));
        if (tail && j * BN + acc_row(blk, i, hi) >= lv) p = 0.f;
        s[i] = p * (dp[i] - dl);
      }
      bf16x8 dsop[2];
      pack_ops(s, dsop);
      tr_x_op(P ? Kv1 : Kv0, dsop, blk, acc, lane);
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

// ---- dK (DK) or dV (!DK): one tile of 256 keys of one (b, h) per workgroup.
//   S = Q K^T (Q tile in K order), P = exp2(S c - lse log2 e) (per query row),
//   dV^T += dO^T P (dO tile in V order); dP = dO V^T (dO tile in K order),
//   dS = P (dP - D), dK^T += Q^T dS (Q tile in V order).  Keys at or beyond
//   Lv get P = 0 and so zero gradient.
template <bool DK>
__global__ __launch_bounds__(NT) void bwd_kv_kernel(BwdArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t Qk0[KTILE], Qk1[KTILE], Tv0[TILE], Tv1[TILE];
  __shared__ __attribute__((aligned(16))) uint16_t Ok0[DK ? KTILE : 8], Ok1[DK ? KTILE : 8];
  __shared__ __attribute__((aligned(16))) float Lt[2][BN], Dt[2][BN];
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // logical order: key tiles innermost, so the workgroups streaming one
  // query run of one (b, h) are neighbours (same XCD, shared L2)
  const int lid = logical_tile(blockIdx.x, a.nwg);
  const int kt = lid % a.ntile, sbh = lid / a.ntile, sp = sbh % a.qsplit, bh = sbh / a.qsplit;
  const int h = bh % a.H, b = bh / a.H;
  const int tok = a.H * D, rbytes = tok * 2;
  const int lv = valid_keys(a, b);
  const int krow = kt * BW + wave * 32 + l32;
  const bool klive = krow < a.Lk;
  const bool kvalid = krow < lv;
  // a wave none of whose 32 keys is valid does its share of the copies and
  // barriers but no products
  const bool wlive = kt * BW + wave * 32 < lv;
  const size_t rowoff = ((size_t)b * a.Lk + (klive ? krow : 0)) * tok + (size_t)h * D;
  uint16_t* outp = (DK ? a.dk : a.dv) + rowoff;
  // fp32 partial of this run: [qsplit][B][Lk][H][d], dV's after dK's
  float* partp =
      a.qsplit > 1 ? a.part + ((size_t)(DK ? 0 : a.qsplit) + sp) * ((size_t)a.B * a.Lk * tok) + rowoff : nullptr;
  f32x16 acc[4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) acc[mb] = f32x16{};
  auto finish = [&](float mul) __attribute__((always_inline)) {
    if (!klive) return;
    if (a.qsplit > 1) store_own_f32(partp, acc, hi);
    else store_own(outp, acc, mul, hi);
  };
  if (kt * BW >= lv) {  // no valid key in this workgroup: zero gradient
    finish(0.f);
    return;
  }
  bf16x8 kop[8], vop[8];
  own_operand(a.k + rowoff, klive, hi, kop);
  if (DK) own_operand(a.v + rowoff, klive, hi, vop);

  const uint16_t* qbh = a.q + (size_t)b * a.Lq * tok + (size_t)h * D;
  const uint16_t* obh = a.dout + (size_t)b * a.Lq * tok + (size_t)h * D;
  const float* lseb = a.lse + ((size_t)b * a.H + h) * a.Lq;
  const float* delb = a.delta + ((size_t)b * a.H + h) * a.Lq;
  const Staging sg = staging(wave, lane, rbytes);
  // this workgroup's run of query tiles [t0, t1)
  const int t0 = sp * a.qper;
  const int t1 = min(t0 + a.qper, (a.Lq + BN - 1) / BN);
  // copies of query tile t, and its per-row lse and D into registers (rows
  // past Lq: P = 0); put_rows stores those into LDS.  The stores come at the
  // end of a step, where the step waits for its copies anyway: a wave's
  // vector memory operations complete in issue order, so an LDS store right
  // after the loads would make the wave wait for the tile copies too.
  float lrow = INFINITY, drow = 0.f;
  auto copies = [&](int t, uint16_t* qk, uint16_t* tv, uint16_t* ok) __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t rq = tile_rsrc(qbh, t, a.Lq, tok);
    const __amdgpu_buffer_rsrc_t ro = tile_rsrc(obh, t, a.Lq, tok);
    copy_rows(rq, qk, sg);
    if (DK) {
      copy_blocks(rq, tv, wave, sg.v0, sg.v1);
      copy_rows(ro, ok, sg);
    } else {
      copy_blocks(ro, tv, wave, sg.v0, sg.v1);
    }
    if (tid < BN) {
      const int r = t * BN + tid;
      lrow = r < a.Lq ? lseb[r] : INFINITY;
      if (DK) drow = r < a.Lq ? delb[r] : 0.f;
    }
  };
  auto put_rows = [&](int buf) __attribute__((always_inline)) {
    if (tid < BN) {
      Lt[buf][tid] = lrow * kLog2e;
      if (DK) Dt[buf][tid] = drow;
    }
  };
  if (t0 >= t1) {  // empty run
    finish(0.f);
    return;
  }
  copies(t0, Qk0, Tv0, Ok0);
  put_rows(0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  auto step = [&](auto par, int t) __attribute__((always_inline)) {
    constexpr int P = decltype(par)::value;
    if (t + 1 < t1) copies(t + 1, P ? Qk0 : Qk1, P ? Tv0 : Tv1, P ? Ok0 : Ok1);
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      if (!wlive) break;
      f32x16 s = rows_x_own(P ? Qk1 : Qk0, kop, blk, lane);
      f32x16 dp;
      if (DK) dp = rows_x_own(P ? Ok1 : Ok0, vop, blk, lane);
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int r0 = acc_row(blk, 4 * i4, hi);  // four consecutive rows
        const float4 l4 = *reinterpret_cast<const float4*>(&Lt[P][r0]);
        const float lr[4] = {l4.x, l4.y, l4.z, l4.w};
        float dr[4] = {0.f, 0.f, 0.f, 0.f};
        if (DK) {
          const float4 d4 = *reinterpret_cast<const float4*>(&Dt[P][r0]);
          dr[0] = d4.x; dr[1] = d4.y; dr[2] = d4.z; dr[3] = d4.w;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = 4 * i4 + e;
          const float p = kvalid ? __builtin_amdgcn_exp2f(fmaf(s[i], a.c, -lr[e])) : 0.f;
          s[i] = DK ? p * (dp[i] - dr[e]) : p;
        }
      }
      bf16x8 op[2];
      pack_ops(s, op);
      tr_x_op(P ? Tv1 : Tv0, op, blk, acc, lane);
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
  finish(DK ? a.scale : 1.f);
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
    const long g = (long)B * H * ((Lq + kDeltaBlock - 1) / kDeltaBlock);
    e = launch_kernel(bwd_delta_kernel, (unsigned)g, 256u, stream, a);
    if (e != hipSuccess) return e;
    a.ntile = (Lq + BW - 1) / BW;
    a.nwg = a.ntile * B * H;
    e = launch_kernel(bwd_dq_kernel, (unsigned)a.nwg, (unsigned)NT, stream, a);
    if (e != hipSuccess) return e;
  }
  if (Lk > 0) {
    a.ntile = (Lk + BW - 1) / BW;
    a.nwg = a.ntile * B * H * a.qsplit;
    e = launch_kernel(bwd_kv_kernel<false>, (unsigned)a.nwg, (unsigned)NT, stream, a);
    if (e != hipSuccess) return e;
    e = launch_kernel(bwd_kv_kernel<true>, (unsigned)a.nwg, (unsigned)NT, stream, a);
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
// kernels.  Calls that overlap on one GPU share the array and race; the
// delta kernel rewrites every value a call reads, so nothing is cleared.
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
