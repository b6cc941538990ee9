// Flash-attention forward for short key sequences without rotation (text
// cross-attention: tens of thousands of video queries against a few hundred
// padded text keys), gfx950, head dim 128.
//
// With a few key tiles per query tile, the query loads and output stores
// (HBM) weigh as much as the products; the kernel is built so that they run
// beside the products instead of between them.
//   * One persistent workgroup per CU runs a contiguous run of "items"
//     (batch, head, 256-query tile), head by head so that the K/V of a head
//     stay in the XCD's L2; the runs are balanced by key-tile steps, not by
//     items, because batches differ in valid length.
//   * Three K and three V tile buffers (96 KB of LDS); step s of an item
//     reads buffer s mod 3.  Between the items of one (batch, head) the
//     buffers keep the last three tiles used: an item takes those first, in
//     buffer order, then its other tiles in increasing order, each copied
//     into the buffer that the step three before it has freed, two steps
//     before it is read.  An item of at most three tiles copies nothing and
//     meets no barrier before its end; an item of nt > 3 tiles copies nt - 3
//     of them, with one barrier per step.
//   * Memory roles: waves 0-3 move queries in (direct copies into a per-wave
//     LDS staging area) and outputs out; waves 4-7 copy the K/V tiles during
//     an item (the first tiles of a new head are copied by all eight).  A
//     wave's vector memory operations complete in issue order, so the copy
//     waits of waves 4-7 never include query/output traffic, which waves 0-3
//     issue at an item's start (the previous item's outputs out, the next
//     item's queries in) and wait for only when the next item's queries are
//     read, after the item's last scores.
// All eight waves compute, 32 queries each, with the dense kernel's
// matrix-core formulation and softmax (S^T = K Q^T, P taken from the
// accumulator, O^T += V^T P^T through the transposing LDS read, exp2 against
// a reference that resets only when a key block's row sum leaves [0, 2^64)).
// The first key block of an item takes its reference from its own maximum
// (the output is still zero) instead of computing its probabilities twice.
// Log-sum-exps leave straight from registers.
//
// LDS: K and V tiles, 3 x 16 KB each, in MFMA operand order (one 1 KB block
// per matrix instruction operand); query/output staging 8 x 8 KB: 160 KB.
#include "attn_tile.hpp"
#include "launch.hpp"

namespace vidax {
namespace {

using namespace tile;

constexpr int D = kHeadDim;
constexpr int BM = 256;  // queries per item
constexpr int BN = 64;   // keys per tile
constexpr int NW = 8;
constexpr int NT = NW * 64;
constexpr int TILE = BN * D;  // elements of one K or V tile
constexpr int BLK = 512;      // elements of one operand block
constexpr int AREA = 32 * D;  // elements of one wave's staging area
constexpr int kMemWaves = 4;
// Cache policy of the query loads and output stores: non-temporal.  Each
// query row is read once and each output row written once; as streaming
// accesses they do not displace the K/V tiles of the XCD's heads from the L2,
// which the K/V copies hit every step (measured: cross_text 0.60 -> 0.57 ms).
constexpr int kStreamPolicy = 2;

// x, as a value the compiler cannot see through: offsets computed from it are
// not hoisted out of the step loop (hoisted, every copy's uniform offsets live
// in scalar registers for the whole loop, and those are spilled).
__device__ __forceinline__ int opaque(int x) {
  asm volatile("" : "+s"(x));
  return x;
}

struct XArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  const int32_t* kv_valid_len;
  int B, H, Lq, Lk;
  int nqt;      // items (query tiles) per (b, h)
  float c2;     // |scale| * log2(e), or 1 when scale == 0
  float qsign;  // +1, -1 or 0 (scale == 0) applied to the query
};

// Item coordinates: (batch b, head h, 256-query tile qt).
struct Item {
  int qt, h, b;
};

__global__ __launch_bounds__(NT) void xattn_kernel(XArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t K0[TILE], K1[TILE], K2[TILE];
  __shared__ __attribute__((aligned(16))) uint16_t V0[TILE], V1[TILE], V2[TILE];
  __shared__ __attribute__((aligned(16))) uint16_t QO[NW * AREA];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool memw = wave < kMemWaves;
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  const int tok = a.H * D;
  const int rbytes = tok * 2;

  // kv_valid_len through the scalar cache (a constant-address-space load), so
  // that reading it never waits on the wave's outstanding vector memory
  const __attribute__((address_space(4))) int32_t* lens =
      (const __attribute__((address_space(4))) int32_t*)a.kv_valid_len;
  auto valid_len = [&](int b) __attribute__((always_inline)) {
    int l = a.Lk;
    if (lens) l = min(max(lens[b], 0), a.Lk);
    return __builtin_amdgcn_readfirstlane(l);
  };
  // key tiles of an item with lv valid keys (at least 1: an item without
  // valid keys runs one fully masked tile and ends with l = 0)
  auto tiles_of = [&](int lv) __attribute__((always_inline)) { return max(1, (lv + BN - 1) / BN); };
  auto steps_of = [&](int b) __attribute__((always_inline)) { return tiles_of(valid_len(b)); };

  // ---- this workgroup's run: the step stream is cut into G equal runs (at
  // item boundaries); XCD x owns a contiguous range of runs
  const int G = gridDim.x;  // a multiple of 8
  const int run = (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
  const long per_batch = (long)a.H * a.nqt;
  long total = 0;
  for (int b = 0; b < a.B; ++b) total += per_batch * steps_of(b);
  // first item whose first step is at or after step t, and that step
  auto item_at = [&](long t, long& first_step) __attribute__((always_inline)) {
    long cum = 0, base = 0;
    for (int b = 0; b < a.B; ++b) {
      const long nt = steps_of(b);
      const long steps = per_batch * nt;
      if (t < cum + steps) {
        const long i = t <= cum ? 0 : (t - cum + nt - 1) / nt;
        if (i < per_batch) {
          first_step = cum + i * nt;
          return base + i;
        }
      }
      cum += steps;
      base += per_batch;
    }
    first_step = cum;
    return base;
  };
  long s0, s1;
  const long lid0 = item_at(total * run / G, s0);
  const long lid1 = item_at(total * (run + 1) / G, s1);
  if (lid0 >= lid1) return;
  int steps_left = (int)(s1 - s0);

  auto next_item = [&](Item& it) __attribute__((always_inline)) {
    if (++it.qt == a.nqt) {
      it.qt = 0;
      if (++it.h == a.H) {
        it.h = 0;
        ++it.b;
      }
    }
  };

  // ---- queries in, outputs out (waves 0-3, each for staging areas wave and
  // wave + 4).  Buffer records end at the last query row, so rows past Lq read
  // as zero and their stores are dropped.  Copy i of an area brings rows
  // 4 i .. 4 i + 3: lane l the chunk that belongs in slot l & 15 of row
  // r = 4 i + (l >> 4), i.e. chunk stage_slot(l & 15, r) -- which depends on
  // i only through i & 3.
  uint16_t* const own = QO + wave * AREA;
  int qvo[4];  // byte offset within rows 4 i .. 4 i + 3 of what this lane moves, by i & 3
#pragma unroll
  for (int i = 0; i < 4; ++i) qvo[i] = (lane >> 4) * rbytes + stage_slot(lane & 15, 4 * i + (lane >> 4)) * 16;
  auto rows_rsrc = [&](const uint16_t* base, const Item& it) __attribute__((always_inline)) {
    const int row0 = it.qt * BM;
    return __builtin_amdgcn_make_buffer_rsrc(
        (void*)(base + ((size_t)it.b * a.Lq + row0) * tok + (size_t)it.h * D), (short)0,
        __builtin_amdgcn_readfirstlane(min(a.Lq - row0, BM) * rbytes), kBufferFlags);
  };
  auto load_queries = [&](const Item& it) __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t rq = rows_rsrc(a.q, it);
    const int rb = opaque(rbytes), w = opaque(wave);
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int area = w + kMemWaves * t;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rq, (lds_ptr)(QO + area * AREA + 4 * i * D), 16, qvo[i & 3],
                                                 (area * 32 + 4 * i) * rb, 0, kStreamPolicy);
    }
  };
  auto store_outputs = [&](const Item& it) __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t ro = rows_rsrc(a.o, it);
    const int rb = opaque(rbytes), w = opaque(wave);
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int area = w + kMemWaves * t;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const u32x4 val =
            *reinterpret_cast<const u32x4*>(QO + area * AREA + (4 * i + (lane >> 4)) * D + (lane & 15) * 8);
        __builtin_amdgcn_raw_buffer_store_b128(val, ro, qvo[i & 3], (area * 32 + 4 * i) * rb, kStreamPolicy);
      }
    }
  };
  auto store_lse = [&](const Item& it, float v) __attribute__((always_inline)) {
    const int row0 = it.qt * BM;
    const __amdgpu_buffer_rsrc_t rl = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(a.lse ? a.lse + ((size_t)it.b * a.H + it.h) * a.Lq + row0 : a.lse), (short)0,
        a.lse ? __builtin_amdgcn_readfirstlane(min(a.Lq - row0, BM) * 4) : 0, kBufferFlags);
    if (hi == 0) __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), rl, (wave * 32 + l32) * 4, 0, 0);
  };

  // ---- K/V tiles, in operand order: copy wave w fills operand blocks
  // 4 (w & 3) .. + 3 of a tile.
  //   K block 2 st + blk: lane l's 16 bytes = key row 32 blk + (l & 31),
  //     d = 16 st + 8 (l >> 5) .. + 7 (A operand of S^T = K Q^T, d-step st).
  //   V block 4 ks + mb, half r (512 bytes): lane l's 8 bytes = key row
  //     16 ks + 8 r + 4 (l >> 5) + ((l & 15) >> 2), d = 32 mb + 16 ((l >> 4) & 1)
  //     + 4 (l & 3) .. + 3 (what the transposing read of lane l fetches for the
  //     V^T operand of d block mb, keys 16 ks .. 16 ks + 15).
  // For copy wave w the K blocks 4 w + t have st = 2 w + (t >> 1), blk = t & 1,
  // and the V blocks ks = w, mb = t: a per-lane byte offset plus a uniform one.
  const int cw = wave & 3;
  const int kvo = l32 * rbytes + hi * 16;
  const int vvo = (8 * hi + 4 * ((lane >> 4) & 1) + ((lane & 7) >> 1)) * rbytes +
                  2 * (16 * ((lane >> 3) & 1) + 8 * (lane & 1));
  // buffer resource of key tile j of item `it` (lv valid keys): records end
  // at the last valid key, so rows at or past lv land in LDS as zero
  auto tile_rsrc = [&](const uint16_t* base, const Item& it, int lv, int j) __attribute__((always_inline)) {
    const int rows = min(max(lv - j * BN, 0), BN);
    return __builtin_amdgcn_make_buffer_rsrc(
        (void*)(base + ((size_t)it.b * a.Lk + (size_t)j * BN) * tok + (size_t)it.h * D), (short)0,
        __builtin_amdgcn_readfirstlane(rows * rbytes), kBufferFlags);
  };
  auto copy_k = [&](const Item& it, int lv, int j, uint16_t* buf) __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t rs = tile_rsrc(a.k, it, lv, j);
    const int rb = opaque(rbytes), w = opaque(cw);
#pragma unroll
    for (int t = 0; t < 4; ++t)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr)(buf + (4 * w + t) * BLK), 16, kvo,
                                               32 * (t & 1) * rb + (2 * (2 * w + (t >> 1))) * 16, 0, 0);
  };
  auto copy_v = [&](const Item& it, int lv, int j, uint16_t* buf) __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t rs = tile_rsrc(a.v, it, lv, j);
    const int rb = opaque(rbytes), w = opaque(cw);
#pragma unroll
    for (int t = 0; t < 4; ++t)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr)(buf + (4 * w + t) * BLK), 16, vvo,
                                               16 * w * rb + 64 * t, 0, 0);
  };
  // tiles 0 .. min(nt, 3) - 1 of a new (batch, head) into buffers 0 .. 2:
  // waves 0-3 copy the K tiles, waves 4-7 the V tiles
  auto load_head = [&](const Item& it, int lv, int nt) __attribute__((always_inline)) {
    if (memw) {
      copy_k(it, lv, 0, K0);
      if (nt > 1) copy_k(it, lv, 1, K1);
      if (nt > 2) copy_k(it, lv, 2, K2);
    } else {
      copy_v(it, lv, 0, V0);
      if (nt > 1) copy_v(it, lv, 1, V1);
      if (nt > 2) copy_v(it, lv, 2, V2);
    }
  };

  // ---- compute (every wave: queries l32 of its staging area, lane halves hi)
  bf16x8 qreg[8];  // d-chunks 2 s + hi of the lane's query, MFMA B operands
  auto read_q = [&]() __attribute__((always_inline)) {
    const uint32_t sgn = a.qsign < 0.f ? 0x80008000u : 0u;
    const uint32_t keep = a.qsign == 0.f ? 0u : 0xffffffffu;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      u32x4 raw = *reinterpret_cast<const u32x4*>(own + l32 * D + stage_slot(2 * s + hi, l32) * 8);
#pragma unroll
      for (int p = 0; p < 4; ++p) raw[p] = (raw[p] ^ sgn) & keep;
      qreg[s] = __builtin_bit_cast(bf16x8, raw);
    }
  };
  const int koff = lane * 8;  // per-lane element offsets of the operands (operand order)
  const int voff = lane * 4;
  auto qk = [&](const uint16_t* kb, f32x16 s[2]) __attribute__((always_inline)) {
    s[0] = f32x16{};
    s[1] = f32x16{};
#pragma unroll
    for (int st = 0; st < 8; ++st)
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) {
        const bf16x8 kop = *reinterpret_cast<const bf16x8*>(kb + (2 * st + blk) * BLK + koff);
        s[blk] = mfma32(kop, qreg[st], s[blk]);
      }
  };
  f32x16 oacc[4];
  float mref = -INFINITY;  // reference (log2 units), identical in both lane halves
  float lsum = 0.f;        // this lane half's partial sum of p
  auto reset_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) oacc[mb] = f32x16{};
    mref = -INFINITY;
    lsum = 0.f;
  };
  const float c2 = a.c2;
  // p = exp2(s c - mref) for the 32 keys of one key block as two bf16 MFMA
  // operands; returns this lane's sum of the rounded p
  auto softmax_p = [&](const f32x16& s, bf16x8 pop[2]) __attribute__((always_inline)) {
    const float nm = -mref;
    float tsum = 0.f;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      uint32_t pw[4];
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(s[8 * ks + e], c2, nm));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(s[8 * ks + e + 1], c2, nm));
        pw[e >> 1] = pack_bf16x2(p0, p1);
        tsum = dot2(pw[e >> 1], kOnesBf16x2, tsum);
      }
      pop[ks] = __builtin_bit_cast(bf16x8, make_uint4(pw[0], pw[1], pw[2], pw[3]));
    }
    return tsum;
  };
  auto block_max = [&](const f32x16& s) __attribute__((always_inline)) {
    float m = fmaxf(s[0], s[1]);
#pragma unroll
    for (int i = 2; i < 16; ++i) m = fmaxf(m, s[i]);
    return wave_half_max(m) * c2;
  };
  // Probabilities of one key block.  The first block of an item sets the
  // reference to its own maximum (0 when every key is masked: p = 0); a later
  // block whose row sum of p leaves [0, 2^64) resets the reference to the
  // running max, rescaling the output and the sum.
  auto softmax_blk = [&](const f32x16& s, bf16x8 pop[2], bool first) __attribute__((always_inline)) {
    if (first) {
      const float m = block_max(s);
      mref = m == -INFINITY ? 0.f : m;
    }
    float tsum = softmax_p(s, pop);
    if (__builtin_amdgcn_ballot_w64(!(tsum < kSumLimit)) != 0) {
      const float mnew = fmaxf(mref, block_max(s));
      const float alpha = __builtin_amdgcn_exp2f(mref - mnew);
      lsum *= alpha;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[mb][i] *= alpha;
      mref = mnew;
      tsum = softmax_p(s, pop);
    }
    lsum += tsum;
  };
  // O^T += V^T P^T over the 32 keys of key block blk
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
  // masks keys at or past `rem` (valid keys left in this tile)
  auto mask_tail = [&](f32x16 s[2], int rem) __attribute__((always_inline)) {
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (blk * 32 + 8 * (i >> 2) + 4 * hi + (i & 3) >= rem) s[blk][i] = -INFINITY;
  };
  // O = O^T / l (zero, with lse = -inf, when l = 0: no valid key) into the
  // wave's staging area (row l32, d = 32 mb + 8 g + 4 hi .. + 3: half hi of
  // chunk 4 mb + g); returns lse = m + ln l
  auto stage_outputs = [&]() __attribute__((always_inline)) -> float {
    const float l = wave_half_sum(lsum);
    const bool ok = l > 0.f;
    const float inv = ok ? 1.0f / l : 0.f;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        u32x2 pk;
        pk[0] = pack_bf16x2(oacc[mb][4 * g + 0] * inv, oacc[mb][4 * g + 1] * inv);
        pk[1] = pack_bf16x2(oacc[mb][4 * g + 2] * inv, oacc[mb][4 * g + 3] * inv);
        *reinterpret_cast<u32x2*>(own + l32 * D + stage_slot(4 * mb + g, l32) * 8 + 4 * hi) = pk;
      }
    return ok ? (mref + __log2f(l)) * 0.69314718055994531f : -INFINITY;
  };

  // ---- prologue: the first item's queries in registers, its head's first
  // tiles in LDS, the second item's queries on their way
  Item it;
  {
    const int qt = (int)(lid0 % a.nqt);
    const long bh = lid0 / a.nqt;
    it = Item{qt, (int)(bh % a.H), (int)(bh / a.H)};
  }
  int lv = valid_len(it.b), nt = tiles_of(lv);
  if (memw) load_queries(it);
  load_head(it, lv, nt);
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_s_barrier();
  read_q();
  __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
  __builtin_amdgcn_s_barrier();  // every wave has its queries out of the staging area
  Item nx = it;
  next_item(nx);
  bool more = steps_left > nt;
  if (memw && more) load_queries(nx);
  int res0 = 0, res1 = 1, res2 = 2;  // tile held by buffer 0, 1, 2 (uniform)

  while (true) {
    reset_acc();
    const int r0 = res0, r1 = res1, r2 = res2;  // the tiles this item starts with
    int cand = 0;                                 // next candidate of its other tiles
    // one step: s = step, B = its buffer (s mod 3)
    auto body = [&](auto bsel, int s) __attribute__((always_inline)) {
      constexpr int B = decltype(bsel)::value;
      uint16_t* const kb = B == 0 ? K0 : (B == 1 ? K1 : K2);
      uint16_t* const vb = B == 0 ? V0 : (B == 1 ? V1 : V2);
      int& res = B == 0 ? res0 : (B == 1 ? res1 : res2);
      const int t = res;
      const bool lastst = s + 1 == nt;
      f32x16 sc[2];
      qk(kb, sc);
      if (lastst && more) {
        // the item's last scores are formed: the next item's queries into
        // registers (they were loaded at this item's start)
        if (memw) __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_s_barrier();
        read_q();
      }
      if (t + 1 == nt && lv < nt * BN) mask_tail(sc, lv - t * BN);
      bf16x8 pop0[2], pop1[2];
      softmax_blk(sc[0], pop0, s == 0);
      pv_blk(vb, pop0, 0);
      softmax_blk(sc[1], pop1, false);
      pv_blk(vb, pop1, 1);
      if (nt > 3 && !lastst) {
        // the copy issued two steps ago has landed (every wave, after the
        // barrier); this step's buffer is free for the tile of step s + 3
        if (!memw && s >= 2) {
          if (s + 2 < nt) __builtin_amdgcn_s_waitcnt(wait_vm(8));
          else __builtin_amdgcn_s_waitcnt(0);
        }
        __builtin_amdgcn_s_barrier();
        if (s + 3 < nt) {
          while (cand == r0 || cand == r1 || cand == r2) ++cand;
          res = cand++;
          if (!memw) {
            copy_k(it, lv, res, kb);
            copy_v(it, lv, res, vb);
          }
        }
      }
    };
    using b0 = std::integral_constant<int, 0>;
    using b1 = std::integral_constant<int, 1>;
    using b2 = std::integral_constant<int, 2>;
    for (int s = 0; s < nt; s += 3) {
      body(b0(), s);
      if (s + 1 < nt) body(b1(), s + 1);
      if (s + 2 < nt) body(b2(), s + 2);
    }
    store_lse(it, stage_outputs());
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);  // staging writes done before the barrier
    __builtin_amdgcn_s_barrier();            // outputs staged; K/V of this item no longer read
    if (!more) break;
    const Item prev = it;
    steps_left -= nt;
    it = nx;
    next_item(nx);
    lv = valid_len(it.b);
    nt = tiles_of(lv);
    more = steps_left > nt;
    const bool new_head = it.b != prev.b || it.h != prev.h;  // uniform
    if (new_head) {
      load_head(it, lv, nt);
      res0 = 0;
      res1 = 1;
      res2 = 2;
    }
    if (memw) {
      // this item's outputs leave, the next item's queries come in
      store_outputs(prev);
      __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
      if (more) load_queries(nx);
    }
    if (new_head) {
      // the K/V copies (issued before the query/output traffic) have landed
      if (!memw) __builtin_amdgcn_s_waitcnt(0);
      else if (more) __builtin_amdgcn_s_waitcnt(wait_vm(32));
      else __builtin_amdgcn_s_waitcnt(wait_vm(16));
      __builtin_amdgcn_s_barrier();
    }
  }
  if (memw) store_outputs(it);
}

}  // namespace

hipError_t launch_xattn_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v, uint16_t* o, float* lse,
                            int B, int H, int Lq, int Lk, float scale, const int32_t* kv_valid_len, int cus,
                            hipStream_t stream) {
  XArgs a;
  a.q = q; a.k = k; a.v = v; a.o = o; a.lse = lse; a.kv_valid_len = kv_valid_len;
  a.B = B; a.H = H; a.Lq = Lq; a.Lk = Lk;
  a.nqt = (Lq + BM - 1) / BM;
  a.c2 = scale == 0.f ? 1.f : fabsf(scale) * 1.4426950408889634f;
  a.qsign = scale > 0.f ? 1.f : (scale < 0.f ? -1.f : 0.f);
  const unsigned g = (unsigned)(8 * ((cus + 7) / 8));
  return launch_kernel(xattn_kernel, g, (unsigned)NT, stream, a);
}

}  // namespace vidax
