// Standalone 3D rotary embedding, bf16 [B, L, H, 128] -> bf16 (HBM-bound),
// and its transpose (every pair rotated by minus its angle).
//
// Workgroups walk tokens with a grid stride.  A token's 16 channel chunks
// (16 B each) are handled by 16 consecutive lanes; a lane holds the four
// frequencies of its chunk, decodes its token's (t, h, w) once, forms the
// four (cos, sin) pairs, and applies them to the same chunk of every batch
// and head of that token (four heads' loads in flight at a time), so angle
// work is amortised over B * H rows and every global access is a 16-byte,
// row-contiguous load or store.  Interleaved pairs compute the angles in
// registers (no table, no barrier, so the first loads start at once);
// half-split pairs stage rows in LDS and read a (cos, sin) table built there.
#include "launch.hpp"

namespace vidax {
namespace {

constexpr int kThreads = 256;
constexpr int kTokensPerPass = kThreads / 16;

struct Rope3dArgs {
  const uint16_t* x;
  uint16_t* y;
  int B, L, H;
  RopeParams rp;
};

__device__ __forceinline__ int pos_of_axis(int axis, int t, int h, int w) {
  return axis == 0 ? t : (axis == 1 ? h : w);
}

// Interleaved pairs: all four pairs of a chunk are inside the chunk.
__global__ __launch_bounds__(kThreads) void rope3d_interleaved(Rope3dArgs a) {
  const RopeParams& rp = a.rp;
  const int c = threadIdx.x & 15;
  const size_t tok_stride = (size_t)a.H * kHeadDim;        // elements between tokens
  const size_t batch_stride = (size_t)a.L * tok_stride;    // elements between batches
  PairSlot slot[4];
  float omega[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    slot[p] = pair_slot(rp, 4 * c + p);
    const int base_a = slot[p].axis == 0 ? 0 : (slot[p].axis == 1 ? rp.base1 : rp.base2);
    const int j = slot[p].base - base_a, da = 2 * slot[p].stride;
    omega[p] = exp2f(-((float)(2 * j) / (float)da) * rp.log2_theta);
  }

  for (int n = blockIdx.x * kTokensPerPass + (threadIdx.x >> 4); n < a.L; n += gridDim.x * kTokensPerPass) {
    const bool rot = n < rp.n_rot;
    float cs[4], sn[4];
    if (rot) {
      int t = n / (rp.gh * rp.gw);
      int r = n - t * rp.gh * rp.gw;
      int h = r / rp.gw;
      int w = r - h * rp.gw;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        float sv, cv;
        sincosf((float)pos_of_axis(slot[p].axis, t, h, w) * omega[p], &sv, &cv);
        cs[p] = cv;
        sn[p] = rp.inverse ? -sv : sv;
      }
    }
    // one row: rotate (or copy) the 16-byte chunk v of row offset off
    auto put = [&](uint4 v, size_t off) {
      if (rot) {
        uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          float x0 = bf16lo_to_f32(wv[p]);
          float x1 = bf16hi_to_f32(wv[p]);
          float y0 = fmaf(x0, cs[p], -x1 * sn[p]);
          float y1 = fmaf(x0, sn[p], x1 * cs[p]);
          wv[p] = pack_bf16x2(y0, y1);
        }
        *reinterpret_cast<uint4*>(a.y + off) = make_uint4(wv[0], wv[1], wv[2], wv[3]);
      } else if (a.x != a.y) {
        *reinterpret_cast<uint4*>(a.y + off) = v;
      }
    };
    for (int b = 0; b < a.B; ++b) {
      const size_t row0 = b * batch_stride + (size_t)n * tok_stride + c * 8;
      int hh = 0;
      // four heads' loads in flight before the first use; a lane reads and
      // writes only its own chunks, so in-place calls stay race free
      for (; hh + 4 <= a.H; hh += 4) {
        uint4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const uint4*>(a.x + row0 + (size_t)(hh + u) * kHeadDim);
#pragma unroll
        for (int u = 0; u < 4; ++u) put(v[u], row0 + (size_t)(hh + u) * kHeadDim);
      }
      for (; hh < a.H; ++hh) {
        const size_t off = row0 + (size_t)hh * kHeadDim;
        put(*reinterpret_cast<const uint4*>(a.x + off), off);
      }
    }
  }
}

// Half-split pairs: a channel's partner sits d_a/2 channels away, usually in
// another lane's chunk, so each (token, batch, head) row is staged in LDS
// before any lane writes (this also keeps in-place calls race free).
__global__ __launch_bounds__(kThreads) void rope3d_half_split(Rope3dArgs a) {
  __shared__ float2 tab[kRopeTableMax];
  __shared__ uint16_t stage[kTokensPerPass][kHeadDim];
  const RopeParams& rp = a.rp;
  for (int e = threadIdx.x; e < rp.n_entries; e += kThreads) tab[e] = rope_table_entry(rp, e);
  __syncthreads();

  const int c = threadIdx.x & 15;
  const int slotrow = threadIdx.x >> 4;
  const size_t tok_stride = (size_t)a.H * kHeadDim;
  const size_t batch_stride = (size_t)a.L * tok_stride;
  const int offs[3] = {0, rp.dt, rp.dt + rp.dh};
  const int widths[3] = {rp.dt, rp.dh, rp.dw};
  const int bases[3] = {0, rp.base1, rp.base2};

  // Loop bound is uniform across the workgroup so the barriers are reached by all lanes.
  const int passes = (a.L + (int)gridDim.x * kTokensPerPass - 1) / ((int)gridDim.x * kTokensPerPass);
  for (int it = 0; it < passes; ++it) {
    const int n = (it * (int)gridDim.x + (int)blockIdx.x) * kTokensPerPass + slotrow;
    const bool live = n < a.L;
    const bool rot = live && n < rp.n_rot;
    int pos3[3] = {0, 0, 0};
    if (rot) {
      pos3[0] = n / (rp.gh * rp.gw);
      int r = n - pos3[0] * rp.gh * rp.gw;
      pos3[1] = r / rp.gw;
      pos3[2] = r - pos3[1] * rp.gw;
    }
    for (int b = 0; b < a.B; ++b) {
      for (int hh = 0; hh < a.H; ++hh) {
        const size_t off = b * batch_stride + (size_t)(live ? n : 0) * tok_stride + (size_t)hh * kHeadDim + c * 8;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (live) v = *reinterpret_cast<const uint4*>(a.x + off);
        *reinterpret_cast<uint4*>(&stage[slotrow][c * 8]) = v;
        __syncthreads();
        if (rot) {
          uint16_t outv[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int ch = c * 8 + e;
            int ax = ch < offs[1] ? 0 : (ch < offs[2] ? 1 : 2);
            const int half = widths[ax] >> 1;
            const int u = ch - offs[ax];
            const bool first = u < half;
            const int j = first ? u : u - half;
            float2 cs = tab[bases[ax] + pos3[ax] * half + j];
            if (rp.inverse) cs.y = -cs.y;
            const float x0 = __uint_as_float((uint32_t)stage[slotrow][first ? ch : ch - half] << 16);
            const float x1 = __uint_as_float((uint32_t)stage[slotrow][first ? ch + half : ch] << 16);
            const float y = first ? fmaf(x0, cs.x, -x1 * cs.y) : fmaf(x0, cs.y, x1 * cs.x);
            outv[e] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(y));
          }
          uint4 o;
          o.x = outv[0] | ((uint32_t)outv[1] << 16);
          o.y = outv[2] | ((uint32_t)outv[3] << 16);
          o.z = outv[4] | ((uint32_t)outv[5] << 16);
          o.w = outv[6] | ((uint32_t)outv[7] << 16);
          *reinterpret_cast<uint4*>(a.y + off) = o;
        } else if (live && a.x != a.y) {
          *reinterpret_cast<uint4*>(a.y + off) = v;
        }
        __syncthreads();
      }
    }
  }
}

}  // namespace

hipError_t launch_rope3d(const uint16_t* x, uint16_t* y, int B, int L, int H, const RopeParams& rp,
                         hipStream_t stream) {
  Rope3dArgs a{x, y, B, L, H, rp};
  int tokens_groups = (L + kTokensPerPass - 1) / kTokensPerPass;
  // 4 workgroups per CU (the half-split kernel builds its table once per workgroup)
  int grid = tokens_groups < 1024 ? tokens_groups : 1024;
  if (grid < 1) grid = 1;
  return rp.pair_mode == 0 ? launch_kernel(rope3d_interleaved, (unsigned)grid, (unsigned)kThreads, stream, a)
                           : launch_kernel(rope3d_half_split, (unsigned)grid, (unsigned)kThreads, stream, a);
}

}  // namespace vidax
