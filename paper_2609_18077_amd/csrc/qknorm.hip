// Query/key prologue, bf16 [B, L, H, 128] -> bf16 (HBM-bound): per-(token,
// head) RMS normalisation in fp32, a per-channel gain shared by all heads, the
// 3D rotation (interleaved or half-split pairs), rounding to bf16.
//
// Layout as in the standalone rotary kernel: the 16 channel chunks (16 B)
// of a (token, head) row go to 16 consecutive lanes; a lane holds the four
// frequencies of its chunk, decodes its token's (t, h, w) once, forms the four
// (cos, sin) pairs in registers and handles that chunk for every batch and
// head of the token, four heads' loads in flight at a time.  A row's sum of
// squares is combined across its 16 lanes with data-parallel lane moves
// (rotations within the 16-lane row, then permutations within quads), so
// each lane ends with the row total without touching LDS.  Every lane reads
// its chunk before any lane of the row writes, so y may alias x.  With
// half-split pairs a channel's partner (d_a / 2 further in its axis block)
// sits in another lane: the row's normalised fp32 values pass through a
// per-row LDS buffer of the 16 lanes (one wave's lanes, so no barrier), and
// each lane forms the angles of its 8 channels rather than of 4 pairs.
#include "launch.hpp"

namespace vidax {
namespace {

constexpr int kThreads = 256;
constexpr int kTokensPerPass = kThreads / 16;

struct QkNormArgs {
  const uint16_t* x;
  uint16_t* y;
  const float* gain;  // [128] or null (unit gain)
  float eps;
  int B, L, H;
  RopeParams rp;
};

// v summed over the 16 lanes of its row; every lane receives the sum.
__device__ __forceinline__ float row16_sum(float v) {
  // row_ror:8, row_ror:4, quad_perm [2,3,0,1], quad_perm [1,0,3,2]
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x124, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4e, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xb1, 0xf, 0xf, false));
  return v;
}

template <bool ROPE, bool HALF>
__global__ __launch_bounds__(kThreads) void qk_norm_kernel(QkNormArgs a) {
  const RopeParams& rp = a.rp;
  __shared__ float rowbuf[HALF ? kThreads * 8 : 1];  // half split: 128 channels of each lane group's row

  const int c = threadIdx.x & 15;  // chunk: channels 8c .. 8c + 7 = pairs 4c .. 4c + 3
  float g[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) g[e] = 1.f;
  if (a.gain) {
    const float4 g0 = *reinterpret_cast<const float4*>(a.gain + 8 * c);
    const float4 g1 = *reinterpret_cast<const float4*>(a.gain + 8 * c + 4);
    g[0] = g0.x; g[1] = g0.y; g[2] = g0.z; g[3] = g0.w;
    g[4] = g1.x; g[5] = g1.y; g[6] = g1.z; g[7] = g1.w;
  }
  PairSlot slot[4];
  float omega[4];  // frequency of each pair of the chunk
  // half split: per channel e of the chunk, its axis, frequency, whether it
  // is the first of its pair, and where its partner lies in the row buffer
  int hax[8], hpart[8];
  bool hfirst[8];
  float homega[8];
  if (HALF) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int ch = 8 * c + e;
      int o, hl;
      if (ch < rp.dt) { o = 0; hl = rp.dt >> 1; hax[e] = 0; }
      else if (ch < rp.dt + rp.dh) { o = rp.dt; hl = rp.dh >> 1; hax[e] = 1; }
      else { o = rp.dt + rp.dh; hl = rp.dw >> 1; hax[e] = 2; }
      hfirst[e] = ch - o < hl;
      const int j = hfirst[e] ? ch - o : ch - o - hl;
      hpart[e] = hfirst[e] ? ch + hl : ch - hl;
      homega[e] = exp2f(-((float)(2 * j) / (float)(2 * hl)) * rp.log2_theta);
    }
  } else if (ROPE) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      slot[p] = pair_slot(rp, 4 * c + p);
      const int base_a = slot[p].axis == 0 ? 0 : (slot[p].axis == 1 ? rp.base1 : rp.base2);
      const int j = slot[p].base - base_a, da = 2 * slot[p].stride;
      omega[p] = exp2f(-((float)(2 * j) / (float)da) * rp.log2_theta);
    }
  }
  const size_t tok_stride = (size_t)a.H * kHeadDim;      // elements between tokens
  const size_t batch_stride = (size_t)a.L * tok_stride;  // elements between batches
  const float inv_d = 1.0f / kHeadDim;

  for (int n = blockIdx.x * kTokensPerPass + (threadIdx.x >> 4); n < a.L; n += gridDim.x * kTokensPerPass) {
    const bool rot = ROPE && n < rp.n_rot;
    float cs[4] = {1.f, 1.f, 1.f, 1.f}, sn[4] = {0.f, 0.f, 0.f, 0.f};
    float hcs[8], hsn[8];  // half split: angle of each channel's pair
#pragma unroll
    for (int e = 0; e < 8; ++e) { hcs[e] = 1.f; hsn[e] = 0.f; }
    if (rot) {
      const int t = n / (rp.gh * rp.gw);
      const int r = n - t * rp.gh * rp.gw;
      const int h = r / rp.gw;
      const int w = r - h * rp.gw;
      if (HALF) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int pos = hax[e] == 0 ? t : (hax[e] == 1 ? h : w);
          sincosf((float)pos * homega[e], &hsn[e], &hcs[e]);
        }
      } else {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const int pos = slot[p].axis == 0 ? t : (slot[p].axis == 1 ? h : w);
          sincosf((float)pos * omega[p], &sn[p], &cs[p]);
        }
      }
    }
    float* const row = rowbuf + (HALF ? (threadIdx.x >> 4) * 128 : 0);
    // one row: normalise, scale, rotate and store the 16-byte chunk v
    auto put = [&](uint4 v, size_t off) {
        const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
        float xf[8];
        float ss = 0.f;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          xf[2 * p] = bf16lo_to_f32(wv[p]);
          xf[2 * p + 1] = bf16hi_to_f32(wv[p]);
          ss = fmaf(xf[2 * p], xf[2 * p], ss);
          ss = fmaf(xf[2 * p + 1], xf[2 * p + 1], ss);
        }
        const float r = rsqrtf(fmaf(row16_sum(ss), inv_d, a.eps));
        uint32_t o[4];
        if (HALF) {
          float yv[8], zv[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) yv[e] = xf[e] * r * g[e];
          if (rot) {
            // the row's normalised values through LDS: written and read by the
            // 16 lanes of this row (one wave, in order)
            *reinterpret_cast<float4*>(row + 8 * c) = make_float4(yv[0], yv[1], yv[2], yv[3]);
            *reinterpret_cast<float4*>(row + 8 * c + 4) = make_float4(yv[4], yv[5], yv[6], yv[7]);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float yp = row[hpart[e]];
              zv[e] = hfirst[e] ? fmaf(yv[e], hcs[e], -yp * hsn[e]) : fmaf(yp, hsn[e], yv[e] * hcs[e]);
            }
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) zv[e] = yv[e];
          }
#pragma unroll
          for (int p = 0; p < 4; ++p) o[p] = pack_bf16x2(zv[2 * p], zv[2 * p + 1]);
        } else {
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            const float y0 = xf[2 * p] * r * g[2 * p];
            const float y1 = xf[2 * p + 1] * r * g[2 * p + 1];
            o[p] = rot ? pack_bf16x2(fmaf(y0, cs[p], -y1 * sn[p]), fmaf(y0, sn[p], y1 * cs[p])) : pack_bf16x2(y0, y1);
          }
        }
        *reinterpret_cast<uint4*>(a.y + off) = make_uint4(o[0], o[1], o[2], o[3]);
    };
    for (int b = 0; b < a.B; ++b) {
      const size_t row0 = b * batch_stride + (size_t)n * tok_stride + c * 8;
      int hh = 0;
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

}  // namespace

hipError_t launch_qk_norm(const uint16_t* x, uint16_t* y, const float* gain, float eps, int B, int L, int H,
                          const RopeParams& rp, hipStream_t stream) {
  QkNormArgs a{x, y, gain, eps, B, L, H, rp};
  int groups = (L + kTokensPerPass - 1) / kTokensPerPass;
  int grid = groups < 1024 ? groups : 1024;  // 4 workgroups per CU
  if (grid < 1) grid = 1;
  if (!rp.enabled) return launch_kernel(qk_norm_kernel<false, false>, (unsigned)grid, (unsigned)kThreads, stream, a);
  return rp.pair_mode ? launch_kernel(qk_norm_kernel<true, true>, (unsigned)grid, (unsigned)kThreads, stream, a)
                      : launch_kernel(qk_norm_kernel<true, false>, (unsigned)grid, (unsigned)kThreads, stream, a);
}

}  // namespace vidax
