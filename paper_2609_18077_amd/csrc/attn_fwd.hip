// Flash-attention forward for gfx950: bf16 MFMA (32x32x16) with fp32
// accumulation, streaming softmax, 3D rotary embedding, per-batch valid-key
// prefix.  Head dim 128.
//
// Work decomposition
//   One workgroup = 8 waves = 256 query rows of one (batch, head); each wave
//   owns 32 query rows, and the two waves sharing a SIMD overlap each other's
//   matrix and vector work.  Keys/values stream through LDS in tiles of 64,
//   two buffers each, one barrier per tile.  Step j is software pipelined:
//   the matrix cores compute the scores of tile j + 1 while the vector ALUs
//   turn the first key block (32 keys) of tile j into probabilities; the PV
//   products of that block run while the second block's probabilities are
//   computed; then the second block's PV products.  Meanwhile K_{j+2} and
//   V_{j+1} are copied from global memory straight into LDS (buffer loads
//   with the LDS flag: no registers, no LDS store instructions).
//
// Matrix-core formulation (per wave, per key tile)
//   S^T[64 keys x 32 queries] = K_tile * Q^T   (16 MFMAs: 2 key blocks x 8 d-steps)
//   O^T[128 d x 32 queries]  += V^T * P^T      (16 MFMAs: 4 d blocks x 4 key-steps)
//   Computing the transposed scores puts one query column in each lane, so the
//   softmax row max/sum are register-local plus one swap between the two lane
//   halves, and the fp32 scores convert in place into the bf16 B operand of
//   the PV product (no shuffles).  The key order inside a 16-key step is the
//   accumulator's natural order.  The V^T operands come from the gfx950
//   transposing LDS read (ds_read_b64_tr_b16), which hands each lane 4 keys
//   of one d column per read.
//
// Softmax: the query is multiplied by scale * log2 e (in fp32, after the
// rotation) and rounded to bf16 once, so the products are scores in log2
// units; and the score accumulators of a tile start at -m instead of zero, so
// the matrix cores hand out s - m and p = exp2 of it takes no vector
// arithmetic besides the exponential.  The reference m of a row is not the
// running max but the max of the block that last reset it: no per-tile max is
// computed.  The first block of a row (its sum starts at +inf) and any key
// block whose row sum of p reaches 2^64 or is not finite reset m to the
// running max, rescale the output and sum, shift the scores already computed
// from the old m (the other block of the tile, the next tile), and recompute
// the block's p.  p therefore never exceeds 2^64, so the bf16 P, fp32 sums
// and fp32 output accumulators cannot overflow, and the result equals the
// usual online softmax up to rounding.  Row sums add the bf16-rounded p
// actually fed to the PV product (v_dot2 with ones).

// Rotary embedding: each workgroup builds an fp32 (cos, sin) table per (axis,
// position, frequency) in LDS; each axis has one extra identity position used
// by unrotated tokens.  Queries are rotated as they are loaded.  Keys either
// arrive rotated (rotated once by the standalone rotary kernel, which costs
// less than rotating every key tile once per query tile) or are rotated here:
// then K goes through registers instead of the direct copy, the coefficients
// of the rows staged next are fetched at the start of a step, and the rotated
// rows are written to LDS after the PV products.
//
// Global loads use buffer resources whose record count ends at the last valid
// key, so rows past kv_valid_len read as zero (and land in LDS as zero)
// without any per-lane test.
//
// Query rows are loaded and output rows stored whole (coalesced), through a
// per-wave staging area in LDS that converts to and from the layout in which
// a lane holds one query.
//
// LDS (per workgroup): K and V tiles 2 x 16 KB each, stored in MFMA operand
// order (see below); rotary table <= 32 KB; query/output staging in the K/V
// buffers (free before the first copies and after the last tile).
//
// Short key sequences without rotation (text cross-attention) go to the
// persistent short-key kernel instead (xattn_fwd.hip).
#include <type_traits>

#include "attn_tile.hpp"
#include "launch.hpp"

namespace vidax {
namespace {

using namespace tile;

constexpr int D = kHeadDim;
constexpr int BM = 256;
constexpr int BN = 64;
constexpr int NW = 8;
constexpr int NT = NW * 64;
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
  float qmul;   // scale * log2(e): the rotated query is multiplied by it before rounding to bf16
  float c2;     // unrotated query: |scale| * log2(e) (1 when scale == 0), applied in the exponent
  float qsign;  // unrotated query: +1, -1 or 0 (scale == 0) applied to the query
  RopeParams rp;
  // attention rotary table: axis a holds (G_a + 1) positions x d_a/2 pairs
  int tbase1, tbase2, tentries;
  uint32_t pos_step;  // packed (t, h, w) increment of BN tokens
  uint32_t pos_sent;  // packed identity position (gt, gh, gw)
};

// Rotates one interleaved bf16 pair (x0 low, x1 high) by (cos, sin) in fp32.
__device__ __forceinline__ uint32_t rotate_pair(uint32_t x, float2 cs) {
  const float x0 = bf16lo_to_f32(x), x1 = bf16hi_to_f32(x);
  return pack_bf16x2(fmaf(x0, cs.x, -x1 * cs.y), fmaf(x0, cs.y, x1 * cs.x));
}

// Table entry e of the attention kernel (see AttnArgs): position G_a of each
// axis is the identity.
__device__ float2 attn_table_entry(const AttnArgs& a, int e) {
  const RopeParams& r = a.rp;
  int f, half, da, g;
  if (e < a.tbase1) { f = e; half = r.dt >> 1; da = r.dt; g = r.gt; }
  else if (e < a.tbase2) { f = e - a.tbase1; half = r.dh >> 1; da = r.dh; g = r.gh; }
  else { f = e - a.tbase2; half = r.dw >> 1; da = r.dw; g = r.gw; }
  const int pos = f / half;
  const int j = f - pos * half;
  float c = 1.f, s = 0.f;
  if (pos < g) {
    const float omega = exp2f(-((float)(2 * j) / (float)da) * r.log2_theta);
    sincosf((float)pos * omega, &s, &c);
  }
  return make_float2(c, s);
}

// Per channel pair: byte offset of its first table entry, byte stride per
// position, and which coordinate of the packed (t << 22 | h << 11 | w)
// position selects the row.  The w and h fields have one spare bit so a
// BN-token step plus carry never overflows them.
struct PairIdx {
  int base, stride, shift;
};
constexpr int kEntryBytes = 8;

__device__ __forceinline__ PairIdx pair_idx(const AttnArgs& a, int pi) {
  const RopeParams& r = a.rp;
  const int ht = r.dt >> 1, hh = r.dh >> 1;
  PairIdx p;
  if (pi < ht) { p.base = pi; p.stride = ht; p.shift = 22; }
  else if (pi < ht + hh) { p.base = a.tbase1 + pi - ht; p.stride = hh; p.shift = 11; }
  else { p.base = a.tbase2 + pi - ht - hh; p.stride = r.dw >> 1; p.shift = 0; }
  p.base *= kEntryBytes;
  p.stride *= kEntryBytes;
  return p;
}

// Table entry of pair p at packed position pos (24-bit multiply-add).
__device__ __forceinline__ float2 table_entry(const float2* tab, const PairIdx& p, uint32_t pos) {
  // the t field is the top 10 bits, so an 11-bit extract at offset 22 is exact
  const uint32_t off = __umul24(__builtin_amdgcn_ubfe(pos, p.shift, 11), (uint32_t)p.stride) + (uint32_t)p.base;
  return *reinterpret_cast<const float2*>(reinterpret_cast<const char*>(tab) + off);
}

__device__ __forceinline__ uint32_t packed_pos(const AttnArgs& a, int n) {
  if (n >= a.rp.n_rot) return a.pos_sent;
  const int t = n / (a.rp.gh * a.rp.gw);
  const int rem = n - t * a.rp.gh * a.rp.gw;
  const int h = rem / a.rp.gw;
  return ((uint32_t)t << 22) | ((uint32_t)h << 11) | (uint32_t)(rem - h * a.rp.gw);
}

// K and V tiles sit in LDS in MFMA operand order: 16 blocks of 1 KB, each
// holding exactly what one wave reads for one matrix instruction, lane by lane.
//   K block 2 st + blk: lane l's 16 bytes = key row 32 blk + (l & 31),
//     d = 16 st + 8 (l >> 5) .. + 7 (A operand of S^T = K Q^T, d-step st).
//   V block 4 ks + mb, half r (512 bytes): lane l's 8 bytes = key row
//     16 ks + 8 r + 4 (l >> 5) + ((l & 15) >> 2), d = 32 mb + 16 ((l >> 4) & 1)
//     + 4 (l & 3) .. + 3 (what the transposing read of lane l fetches for the
//     V^T operand of d block mb, keys 16 ks .. 16 ks + 15).
// Every operand read is one contiguous, bank-conflict-free 1 KB (K) or 512 B
// (V) access at an offset that is a constant of the instruction, and each
// block is filled by one direct 1 KB global -> LDS copy.
constexpr int TILE = BN * D;  // elements per K or V tile
constexpr int BLK = 512;      // elements per operand block
// Short key sequences without rotation: at or below this many keys (and with
// enough query tiles to fill the chip) the persistent short-key kernel runs.
constexpr int kAttnShortKeys = 1024;

// ROPE: rotate the queries (and build the table); ROPE_K: also rotate the keys
// while staging them (false when the caller passes pre-rotated keys).
// HALF: half-split pairs (queries only; ROPE_K is then false).
template <bool ROPE, bool ROPE_K, bool HALF = false>
__global__ __launch_bounds__(NT) void attn_fwd_kernel(AttnArgs a) {
  // Two K and two V buffers, each its own LDS object so that the compiler can
  // tell the direct copies into one buffer from the operand reads of another
  // (and does not wait for the copies before those reads).
  __shared__ __attribute__((aligned(16))) uint16_t K0[TILE], K1[TILE], V0[TILE], V1[TILE];
  __shared__ float2 tab[ROPE ? kAttnTableMax : 1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  const int tok = a.H * D;     // elements between consecutive tokens
  const int rbytes = tok * 2;  // bytes between consecutive tokens

  // ---- state of the current query tile (logical tile lid: query tile
  // lid % nqt of (b, h) = (lid / nqt / H, lid / nqt % H))
  int b = 0, h = 0, qrow = 0, lv = 0, ntiles = 0;
  bool qlive = false;
  const uint16_t* kbh = a.k;
  const uint16_t* vbh = a.v;
  // Tile order: the query tiles of one (b, h) are consecutive (the K/V
  // stream of that head is then shared in L2).
  auto tile_of = [&](int lid, int& qt, int& bh) __attribute__((always_inline)) {
    qt = lid % a.nqt;
    bh = lid / a.nqt;
  };
  auto begin_tile = [&](int lid) __attribute__((always_inline)) {
    int qt, bh;
    tile_of(lid, qt, bh);
    h = bh % a.H;
    b = bh / a.H;
    int l = a.Lk;
    if (a.kv_valid_len) l = min(max(a.kv_valid_len[b], 0), a.Lk);
    lv = __builtin_amdgcn_readfirstlane(l);  // uniform: keeps buffer descriptors in SGPRs
    kbh = a.k + (size_t)b * a.Lk * tok + (size_t)h * D;
    vbh = a.v + (size_t)b * a.Lk * tok + (size_t)h * D;
    qrow = qt * BM + wave * 32 + l32;
    qlive = qrow < a.Lq;
    ntiles = (lv + BN - 1) / BN;
  };

  // Query rows come in and output rows go out whole: each 16-lane group of a
  // wave moves one 256-byte row (coalesced), and the wave's 8 KB staging area
  // in LDS (32 rows x 16 chunks of 16 bytes, chunk c of row r at slot
  // stage_slot(c, r)) converts between that layout and the operand layout in
  // which a lane holds one query.  It borrows the K/V buffers (free before
  // the first copies and after the last tile).
  uint16_t* const stage = (wave < 2 ? K0 : wave < 4 ? K1 : wave < 6 ? V0 : V1) + (wave & 1) * 32 * D;

  // The wave's 32 query rows of tile lid into its staging area: copy i brings
  // rows 4 i .. 4 i + 3, lane l the chunk that belongs in slot l & 15 of row
  // 4 i + (l >> 4).  Rows past Lq read as zero.  Exactly 8 copies a wave.
  auto dma_q = [&](int lid) __attribute__((always_inline)) {
    int qt, bh;
    tile_of(lid, qt, bh);
    const int row0 = qt * BM + wave * 32;
    const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(a.q + (size_t)(bh / a.H) * a.Lq * tok + (size_t)(bh % a.H) * D), (short)0, a.Lq * rbytes,
        kBufferFlags);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = 4 * i + (lane >> 4);
      const int off = row0 + r < a.Lq ? (row0 + r) * rbytes + stage_slot(lane & 15, r) * 16 : 0x7ffffff0;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rq, (lds_ptr)(stage + 4 * i * D), 16, off, 0, 0, 0);
    }
  };

  // raw[s] = chunk 2 s + hi of the lane's own query row l32, from the staging area
  auto read_q = [&](uint4 raw[8]) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < 8; ++s)
      raw[s] = *reinterpret_cast<const uint4*>(stage + l32 * D + stage_slot(2 * s + hi, l32) * 8);
  };

  // ---- Q: lane holds query qrow, d-chunks 2s + hi (s = 0..7) as MFMA B operands
  bf16x8 qreg[8];
  // Half-split pairs (keys then come rotated by vidax_rope3d): pair j of the
  // block of axis a (offset o_a, width d_a) is channels o_a + j and
  // o_a + j + d_a / 2, which different lanes read out.  So the staged query
  // row is rotated and scaled in place first, the two lanes of a row taking
  // 32 pairs each (one rounding, as in the interleaved path), and make_q then
  // takes the values as they are.
  auto rotate_staged_half_split = [&]() __attribute__((always_inline)) {
    const RopeParams& r = a.rp;
    const uint32_t qpos = packed_pos(a, qlive ? qrow : r.n_rot);
    const float qm = a.qmul;
    uint16_t* const row = stage + l32 * D;
    const int ht = r.dt >> 1, hh = r.dh >> 1;
#pragma unroll 1
    for (int pi = 32 * hi; pi < 32 * hi + 32; ++pi) {
      int o, hl, j;
      if (pi < ht) { o = 0; hl = ht; j = pi; }
      else if (pi < ht + hh) { o = r.dt; hl = hh; j = pi - ht; }
      else { o = r.dt + r.dh; hl = r.dw >> 1; j = pi - ht - hh; }
      const int c0 = o + j, c1 = c0 + hl;
      uint16_t* const p0 = row + stage_slot(c0 >> 3, l32) * 8 + (c0 & 7);
      uint16_t* const p1 = row + stage_slot(c1 >> 3, l32) * 8 + (c1 & 7);
      const float x0 = __uint_as_float((uint32_t)*p0 << 16), x1 = __uint_as_float((uint32_t)*p1 << 16);
      const float2 cs = table_entry(tab, pair_idx(a, pi), qpos);
      const uint32_t y = pack_bf16x2(fmaf(x0, cs.x, -x1 * cs.y) * qm, fmaf(x0, cs.y, x1 * cs.x) * qm);
      *p0 = (uint16_t)(y & 0xffffu);
      *p1 = (uint16_t)(y >> 16);
    }
  };
  auto make_q = [&](const uint4 raw[8]) __attribute__((always_inline)) {
    const uint32_t qpos = ROPE ? packed_pos(a, qlive ? qrow : a.rp.n_rot) : 0u;
    const float qm = a.qmul;
    const uint32_t sgn = a.qsign < 0.f ? 0x80008000u : 0u;
    const uint32_t keep = a.qsign == 0.f ? 0u : 0xffffffffu;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int c = 2 * s + hi;
      uint32_t wq[4] = {raw[s].x, raw[s].y, raw[s].z, raw[s].w};
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        if (ROPE) {  // rotated and scaled in fp32, rounded once
          if (!HALF) {  // (half-split rows were rotated in the staging area)
            const float x0 = bf16lo_to_f32(wq[p]), x1 = bf16hi_to_f32(wq[p]);
            const float2 cs = table_entry(tab, pair_idx(a, 4 * c + p), qpos);
            wq[p] = pack_bf16x2(fmaf(x0, cs.x, -x1 * cs.y) * qm, fmaf(x0, cs.y, x1 * cs.x) * qm);
          }
        } else {  // exact: sign only
          wq[p] = (wq[p] ^ sgn) & keep;
        }
      }
      qreg[s] = __builtin_bit_cast(bf16x8, make_uint4(wq[0], wq[1], wq[2], wq[3]));
    }
  };

  // ---- staging: wave w fills K blocks 2w, 2w + 1 (d-step w, both key blocks)
  // and V blocks 2w, 2w + 1 of every tile.  Byte offsets from the tile's
  // first row of what lane `lane` copies:
  const int kr0 = l32;                 // K rows kr0 and kr0 + 32 ...
  const int kc = 2 * wave + hi;        // ... 16-byte chunk kc
  const int kg0 = kr0 * rbytes + kc * 16;
  const int kg1 = kg0 + 32 * rbytes;
  int vg0, vg1;
  {
    const int vrow = 8 * hi + 4 * ((lane >> 4) & 1) + ((lane & 7) >> 1);
    const int vd = 16 * ((lane >> 3) & 1) + 8 * (lane & 1);
    const int b0 = 2 * wave, b1 = 2 * wave + 1;  // blocks (ks, mb) = (b >> 2, b & 3)
    vg0 = (vrow + 16 * (b0 >> 2)) * rbytes + 2 * (vd + 32 * (b0 & 3));
    vg1 = (vrow + 16 * (b1 >> 2)) * rbytes + 2 * (vd + 32 * (b1 & 3));
  }

  // rotary state of the fused path: the thread owns chunk kc of K rows kr0, kr0 + 32
  PairIdx kpi[4];
  uint32_t kpos[2] = {0u, 0u};
  if (ROPE_K) {
#pragma unroll
    for (int p = 0; p < 4; ++p) kpi[p] = pair_idx(a, 4 * kc + p);
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int n = kr0 + 32 * r;
      const int t = n / (a.rp.gh * a.rp.gw);
      const int rem = n - t * a.rp.gh * a.rp.gw;
      const int hh = rem / a.rp.gw;
      kpos[r] = ((uint32_t)t << 22) | ((uint32_t)hh << 11) | (uint32_t)(rem - hh * a.rp.gw);
    }
  }

  // Buffer resource of tile `tile`: its records end at the last valid key, so
  // rows at or beyond lv read as zero (and land in LDS as zero); tiles past
  // the end read all zeros and are never used.
  auto tile_rsrc = [&](const uint16_t* base, int tile) __attribute__((always_inline)) {
    const int rows = min(max(lv - tile * BN, 0), BN);
    const int nbytes = __builtin_amdgcn_readfirstlane(rows * rbytes);  // uniform
    return __builtin_amdgcn_make_buffer_rsrc((void*)(base + (size_t)tile * BN * tok), (short)0, nbytes, kBufferFlags);
  };

  // Direct global -> LDS copy of the wave's two operand blocks of a tile (16
  // bytes a lane, landing at the block base + 16 * lane).
  auto dma_tile = [&](const uint16_t* base, int tile, uint16_t* buf, int g0, int g1) __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t rs = tile_rsrc(base, tile);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr)(buf + (2 * wave) * BLK), 16, g0, 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr)(buf + (2 * wave + 1) * BLK), 16, g1, 0, 0, 0);
  };

  // fused path: the thread's two K chunks through registers
  auto load_k = [&](int tile, uint4 reg[2]) __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t rs = tile_rsrc(kbh, tile);
    const int g[2] = {kg0, kg1};
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(rs, g[r], 0, 0);
      reg[r] = make_uint4(x[0], x[1], x[2], x[3]);
    }
  };

  // Coefficients for the two K rows of the next tile to be staged; advances
  // the rows' packed coordinates by BN tokens.  Rows at or past the rotated
  // prefix take the identity position.
  auto fetch_coef = [&](int tile, float2 cs[2][4]) __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const uint32_t pos = tile * BN + kr0 + 32 * r < a.rp.n_rot ? kpos[r] : a.pos_sent;
#pragma unroll
      for (int p = 0; p < 4; ++p) cs[r][p] = table_entry(tab, kpi[p], pos);
      // mixed-radix step; past the grid the t field may wrap, but those rows use pos_sent
      uint32_t np = kpos[r] + a.pos_step;
      if ((np & 2047u) >= (uint32_t)a.rp.gw) np += (1u << 11) - (uint32_t)a.rp.gw;
      if (((np >> 11) & 2047u) >= (uint32_t)a.rp.gh) np += (1u << 22) - ((uint32_t)a.rp.gh << 11);
      kpos[r] = np;
    }
  };

  auto store_k = [&](uint16_t* buf, const uint4 reg[2], const float2 cs[2][4]) __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      uint4 kv = reg[r];
      kv.x = rotate_pair(kv.x, cs[r][0]);
      kv.y = rotate_pair(kv.y, cs[r][1]);
      kv.z = rotate_pair(kv.z, cs[r][2]);
      kv.w = rotate_pair(kv.w, cs[r][3]);
      *reinterpret_cast<uint4*>(buf + (2 * wave + r) * BLK + lane * 8) = kv;
    }
  };

  // per-lane LDS element offsets of the MFMA operands (operand order, above)
  const int koff = lane * 8;
  const int voff = lane * 4;

  // Rotated query (scaled into log2 units): the score accumulators start at
  // -cbase instead of zero, so that the products come out as s - cbase with
  // no vector work.  Unrotated query: they start at zero and p = exp2(s c2 -
  // mref) takes one FMA (cbase stays 0).
  float mref = -INFINITY;  // reference max (log2 units), identical in both lane halves
  float cbase = 0.f;       // the offset the score accumulators start from (mref once finite)
  f32x16 cneg = f32x16{};
  auto qk = [&](const uint16_t* kb, f32x16 s[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int st = 0; st < 8; ++st) {
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) {
        const bf16x8 kop = *reinterpret_cast<const bf16x8*>(kb + (2 * st + blk) * BLK + koff);
        s[blk] = mfma32(kop, qreg[st], st == 0 ? (ROPE ? cneg : f32x16{}) : s[blk]);
      }
    }
  };

  f32x16 oacc[4];
  float sum0 = INFINITY;   // start of the row sums: +inf until the first reset forces it
  float lsum = 0.f;        // this lane half's partial sum of p
  auto reset_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) oacc[mb] = f32x16{};
    mref = -INFINITY;
    cbase = 0.f;
    cneg = f32x16{};
    sum0 = INFINITY;
    lsum = 0.f;
  };
  const uint32_t ones = 0x3f803f80u;  // bf16 (1, 1)

  const float c2 = a.c2;
  // p = exp2(s) (rotated query: scores already relative to the reference) or
  // exp2(s c2 - mref) for the 32 keys of one key block as two bf16 MFMA
  // operands (16 keys each); returns tsum plus this lane's sum of p
  auto softmax_p = [&](const f32x16& s, bf16x8 pop[2], float tsum) __attribute__((always_inline)) {
    const float nm = -mref;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      uint32_t pw[4];
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const float p0 = __builtin_amdgcn_exp2f(ROPE ? s[8 * ks + e] : fmaf(s[8 * ks + e], c2, nm));
        const float p1 = __builtin_amdgcn_exp2f(ROPE ? s[8 * ks + e + 1] : fmaf(s[8 * ks + e + 1], c2, nm));
        pw[e >> 1] = pack_bf16x2(p0, p1);
        tsum = dot2(pw[e >> 1], ones, tsum);
      }
      pop[ks] = __builtin_bit_cast(bf16x8, make_uint4(pw[0], pw[1], pw[2], pw[3]));
    }
    return tsum;
  };

  // Probabilities of one key block.  The first block (its sum starts at
  // +inf) and a block whose row sum of p leaves [0, 2^64) reset the
  // reference to the running max, rescaling the output (which may already
  // hold the other block of the same tile) and the sum (see the header).
  // Score blocks already computed from the old offset are shifted to the new
  // one (shift_pending(delta)).
  auto softmax_blk = [&](f32x16& s, bf16x8 pop[2], auto&& shift_pending) __attribute__((always_inline)) {
    float tsum = softmax_p(s, pop, sum0);
    if (__builtin_amdgcn_ballot_w64(!(tsum < kSumLimit)) != 0) {
      sum0 = 0.f;
      float m = fmaxf(s[0], s[1]);
#pragma unroll
      for (int i = 2; i < 16; ++i) m = fmaxf(m, s[i]);
      const float mnew = fmaxf(mref, ROPE ? wave_half_max(m) + cbase : wave_half_max(m) * c2);
      const float alpha = __builtin_amdgcn_exp2f(mref - mnew);
      lsum *= alpha;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[mb][i] *= alpha;
      if (ROPE) {
        const float delta = mnew - cbase;
#pragma unroll
        for (int i = 0; i < 16; ++i) s[i] -= delta;
        shift_pending(delta);
        cbase = mnew;
#pragma unroll
        for (int i = 0; i < 16; ++i) cneg[i] = -mnew;
      }
      mref = mnew;
      tsum = softmax_p(s, pop, 0.f);
    }
    lsum += tsum;
  };

  // O^T += V^T P^T over the 32 keys of key block `blk`
  auto pv_blk = [&](const uint16_t* vb, const bf16x8 pop[2], int blk) __attribute__((always_inline)) {
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const int ks = 2 * blk + k2;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const i16x4 lo = lds_read_tr16(vb + (4 * ks + mb) * BLK + voff);
        const i16x4 hi4 = lds_read_tr16(vb + (4 * ks + mb) * BLK + BLK / 2 + voff);
        const bf16x8 vop = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi4, 0, 1, 2, 3, 4, 5, 6, 7));
        oacc[mb] = mfma32(vop, pop[k2], oacc[mb]);
      }
    }
  };

  // softmax and PV of one score tile, one key block at a time, so that the
  // second block's softmax overlaps the first block's PV products
  auto shift = [&](f32x16& x, float delta) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 16; ++i) x[i] -= delta;
  };
  // (snext: the scores of the next tile, already computed, or null)
  auto softmax_pv = [&](f32x16 s[2], const uint16_t* vb, f32x16* snext) __attribute__((always_inline)) {
    bf16x8 pop0[2], pop1[2];
    softmax_blk(s[0], pop0, [&](float delta) __attribute__((always_inline)) {
      shift(s[1], delta);
      if (snext) {
        shift(snext[0], delta);
        shift(snext[1], delta);
      }
    });
    pv_blk(vb, pop0, 0);
    softmax_blk(s[1], pop1, [&](float delta) __attribute__((always_inline)) {
      if (snext) {
        shift(snext[0], delta);
        shift(snext[1], delta);
      }
    });
    pv_blk(vb, pop1, 1);
  };

  // K_0, K_1 and V_0 of the current tile into K0, K1, V0
  auto first_copies = [&]() __attribute__((always_inline)) {
    if (ROPE_K) {
      uint4 k0[2], k1[2];
      float2 cs0[2][4], cs1[2][4];
      load_k(0, k0);
      load_k(1, k1);
      fetch_coef(0, cs0);
      fetch_coef(1, cs1);
      store_k(K0, k0, cs0);
      store_k(K1, k1, cs1);
    } else {
      dma_tile(kbh, 0, K0, kg0, kg1);
      dma_tile(kbh, 1, K1, kg0, kg1);
    }
    dma_tile(vbh, 0, V0, vg0, vg1);
  };

  f32x16 sa[2], sb[2];

  // Step j (parity P = j & 1): scores of tile j + 1, softmax and PV of tile j,
  // while K_{j+2} and V_{j+1} stream into the buffers that tiles j and j - 1
  // have freed.  The buffers are chosen at compile time.
  auto step = [&](auto parity, int j, f32x16 scur[2], f32x16 snext[2]) __attribute__((always_inline)) {
    constexpr int P = decltype(parity)::value;
    uint16_t* const kfree = P ? K1 : K0;  // held K_j
    uint16_t* const knext = P ? K0 : K1;  // holds K_{j+1}
    uint16_t* const vcur = P ? V1 : V0;   // holds V_j
    uint16_t* const vfree = P ? V0 : V1;  // held V_{j-1}
    uint4 kn[2];
    float2 cs[2][4];
    if (ROPE_K) {
      load_k(j + 2, kn);
      fetch_coef(j + 2, cs);
    } else {
      dma_tile(kbh, j + 2, kfree, kg0, kg1);
    }
    dma_tile(vbh, j + 1, vfree, vg0, vg1);
    qk(knext, snext);
    softmax_pv(scur, vcur, snext);
    if (ROPE_K) store_k(kfree, kn, cs);
    __builtin_amdgcn_s_waitcnt(0);  // this wave's copies have landed
    __syncthreads();
  };
  using even = std::integral_constant<int, 0>;
  using odd = std::integral_constant<int, 1>;

  // the tile whose first copies have landed (and been published): scores of
  // tile 0, the pipelined steps, and the last tile's softmax and PV
  auto run_tile = [&]() __attribute__((always_inline)) {
    qk(K0, sa);
    // step 0 refills K0 (with K_2): every wave must be done reading K_0 first
    __syncthreads();
    int j = 0;
    for (; j + 2 < ntiles; j += 2) {
      step(even(), j, sa, sb);
      step(odd(), j + 1, sb, sa);
    }
    f32x16* slast = sa;
    if (j + 1 < ntiles) {
      step(even(), j, sa, sb);
      ++j;
      slast = sb;
    }
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
      softmax_pv(s, (j & 1) ? V1 : V0, nullptr);
    }
  };

  // ---- output: O = O^T / l (zero when no key is valid), LSE = m + ln l,
  // through the staging area.  Buffer stores: rows past Lq address past the
  // records and are dropped, so every wave issues exactly kOutStores store
  // instructions.
  auto store_o = [&](int ob, int oh, int orow, bool olive, bool empty) __attribute__((always_inline)) {
    const float l = wave_half_sum(lsum);
    const float inv = empty ? 0.f : 1.0f / l;
    // the lane's row l32, d = 32 mb + 8 g + 4 hi .. + 3: half hi of chunk 4 mb + g
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        u32x2 pk;
        pk[0] = pack_bf16x2(oacc[mb][4 * g + 0] * inv, oacc[mb][4 * g + 1] * inv);
        pk[1] = pack_bf16x2(oacc[mb][4 * g + 2] * inv, oacc[mb][4 * g + 3] * inv);
        *reinterpret_cast<u32x2*>(stage + l32 * D + stage_slot(4 * mb + g, l32) * 8 + 4 * hi) = pk;
      }
    // whole rows out: slot lane & 15 of row 4 i + (lane >> 4) holds chunk stage_slot(lane & 15, row)
    const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(a.o + (size_t)ob * a.Lq * tok + (size_t)oh * D), (short)0, a.Lq * rbytes, kBufferFlags);
    const int row0 = orow - l32;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = 4 * i + (lane >> 4);
      const u32x4 v = *reinterpret_cast<const u32x4*>(stage + r * D + (lane & 15) * 8);
      const int grow = row0 + r;
      const int off = grow < a.Lq ? grow * rbytes + stage_slot(lane & 15, r) * 16 : 0x7ffffff0;
      __builtin_amdgcn_raw_buffer_store_b128(v, ro, off, 0, 0);
    }
    const __amdgpu_buffer_rsrc_t rl = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(a.lse ? a.lse + ((size_t)ob * a.H + oh) * a.Lq : a.lse), (short)0, a.lse ? a.Lq * 4 : 0,
        kBufferFlags);
    const float lse = empty ? -INFINITY : (mref + __log2f(l)) * 0.69314718055994531f;
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(lse), rl, olive && hi == 0 ? orow * 4 : 0x7ffffff0, 0, 0);
  };

  // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
  // contiguous range of positions so the query tiles of one (b, h) share
  // that XCD's L2 for the K/V stream.  The positions run over the eighths of
  // every batch in turn (eighth 0 of batch 0, of batch 1, ..., eighth 1 of
  // batch 0, ...), so that each XCD gets about an eighth of every batch:
  // batches of different valid lengths then load the XCDs evenly (with
  // batch after batch, the XCDs holding the longer batches finished last).
  // One batch: position = logical tile.
  int lid;
  {
    const int i = blockIdx.x, n = a.nwg;
    const int per = n >> 3, rem = n & 7, xcd = i & 7, kk = i >> 3;
    const int pos = xcd < rem ? xcd * (per + 1) + kk : rem * (per + 1) + (xcd - rem) * per + kk;
    const int N = a.nwg / a.B;  // tiles per batch: eighth c holds p + (c < r) of them
    const int p = N >> 3, r = N & 7;
    const int big = a.B * r * (p + 1);  // positions in the eighths of size p + 1
    const int c = pos < big ? pos / (a.B * (p + 1)) : r + (pos - big) / (a.B * p);
    const int sc = c < r ? p + 1 : p;
    const int cs = c * p + min(c, r);  // start of eighth c within a batch
    const int rm = pos - a.B * cs;
    lid = (rm / sc) * N + cs + rm % sc;
  }
  begin_tile(lid);
  reset_acc();
  if (lv == 0) {  // no valid key: O = 0, LSE = -inf
    store_o(b, h, qrow, qlive, true);
    return;
  }
  dma_q(lid);  // into the K/V buffers, which are free until the first copies
  if (ROPE) {
    for (int e = tid; e < a.tentries; e += NT) tab[e] = attn_table_entry(a, e);
    __syncthreads();
  }
  __builtin_amdgcn_s_waitcnt(0);  // this wave's query rows have landed
  {
    if (HALF) rotate_staged_half_split();
    uint4 raw[8];
    read_q(raw);
    make_q(raw);
  }
  __syncthreads();  // every wave has its queries out of the K/V buffers
  first_copies();
  __builtin_amdgcn_s_waitcnt(0);  // this wave's copies have landed in LDS
  __syncthreads();
  run_tile();
  __syncthreads();  // every wave is done with the last V tile before the output staging
  store_o(b, h, qrow, qlive, false);
}

}  // namespace

bool attn_rope_supported(const RopeParams& rp) {
  if (!rp.enabled) return true;
  // half-split pairs: queries only (the fused key rotation pairs interleaved channels)
  if (rp.pair_mode != 0 && !rp.keys_prerotated) return false;
  if (rp.gw > kAttnGridHWMax || rp.gh > kAttnGridHWMax || rp.gt > kAttnGridTMax) return false;
  const long entries = (long)(rp.gt + 1) * (rp.dt / 2) + (long)(rp.gh + 1) * (rp.dh / 2) + (long)(rp.gw + 1) * (rp.dw / 2);
  return entries <= kAttnTableMax;
}

// Compute units of the current device (queried once per device).
static int cu_count() {
  static int counts[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (counts[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    counts[dev] = n;
  }
  return counts[dev];
}

hipError_t launch_attn_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v, uint16_t* o,
                           float* lse, int B, int H, int Lq, int Lk, float scale,
                           const int32_t* kv_valid_len, const RopeParams& rp, hipStream_t stream) {
  AttnArgs a;
  a.q = q; a.k = k; a.v = v; a.o = o; a.lse = lse; a.kv_valid_len = kv_valid_len;
  a.B = B; a.H = H; a.Lq = Lq; a.Lk = Lk;
  a.nqt = (Lq + BM - 1) / BM;
  const long nwg = (long)a.nqt * B * H;
  a.nwg = (int)nwg;
  // rotated query: scores in log2 units straight from the products,
  // p = exp2(k . (scale log2(e) q) - m); unrotated query: p = exp2(c2 *
  // (qsign q).k - m), |scale| in the exponent and its sign in q
  a.qmul = scale * 1.4426950408889634f;
  a.c2 = scale == 0.f ? 1.f : fabsf(scale) * 1.4426950408889634f;
  a.qsign = scale > 0.f ? 1.f : (scale < 0.f ? -1.f : 0.f);
  a.rp = rp;
  a.tbase1 = a.tbase2 = a.tentries = 0;
  a.pos_step = a.pos_sent = 0;
  if (rp.enabled) {
    a.tbase1 = (rp.gt + 1) * (rp.dt / 2);
    a.tbase2 = a.tbase1 + (rp.gh + 1) * (rp.dh / 2);
    a.tentries = a.tbase2 + (rp.gw + 1) * (rp.dw / 2);
    const uint32_t sw = BN % rp.gw, sh = (BN / rp.gw) % rp.gh, st = BN / (rp.gw * rp.gh);
    a.pos_step = (st << 22) | (sh << 11) | sw;
    a.pos_sent = ((uint32_t)rp.gt << 22) | ((uint32_t)rp.gh << 11) | (uint32_t)rp.gw;
  }
  // short key sequences without rotation: one persistent workgroup per CU
  // (the per-workgroup scan over the batch lengths bounds B)
  const int cus = cu_count();
  if (!rp.enabled && Lk <= kAttnShortKeys && nwg > 4L * cus && B <= 4096)
    return launch_xattn_fwd(q, k, v, o, lse, B, H, Lq, Lk, scale, kv_valid_len, cus, stream);
  if (rp.enabled && !rp.keys_prerotated)
    return launch_kernel(attn_fwd_kernel<true, true>, (unsigned)nwg, (unsigned)NT, stream, a);
  if (rp.enabled && rp.pair_mode != 0)
    return launch_kernel(attn_fwd_kernel<true, false, true>, (unsigned)nwg, (unsigned)NT, stream, a);
  if (rp.enabled) return launch_kernel(attn_fwd_kernel<true, false>, (unsigned)nwg, (unsigned)NT, stream, a);
  return launch_kernel(attn_fwd_kernel<false, false>, (unsigned)nwg, (unsigned)NT, stream, a);
}

}  // namespace vidax
