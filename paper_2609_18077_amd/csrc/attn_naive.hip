// Scalar fp32 attention forward: an independent, deliberately simple GPU
// implementation used to cross-check the matrix-core kernel at small sizes.
//
// One thread per query row keeps its rotated query and output accumulator in
// fp32 registers.  Keys and values are staged in LDS 32 at a time as fp32; the
// rotation of each staged key is evaluated directly with sincosf (no table).
// Softmax is the streaming form: running max, rescaled running sum.
#include "launch.hpp"

namespace vidax {
namespace {

constexpr int kQ = 64;     // queries per workgroup (one per thread)
constexpr int kKeys = 32;  // keys staged per step

struct NaiveArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  const int32_t* kv_valid_len;
  int B, H, Lq, Lk;
  float scale;
  RopeParams rp;
};

// Rotates channel pair `p` (0..63) of a row held in fp32 at `row` in place,
// for token n, evaluating the angle directly.
__device__ void rotate_pair_direct(const RopeParams& rp, float* row, int n, int p) {
  const int ht = rp.dt >> 1, hh = rp.dh >> 1;
  int axis, j, off, da;
  if (p < ht) { axis = 0; j = p; off = 0; da = rp.dt; }
  else if (p < ht + hh) { axis = 1; j = p - ht; off = rp.dt; da = rp.dh; }
  else { axis = 2; j = p - ht - hh; off = rp.dt + rp.dh; da = rp.dw; }
  int c0, c1;
  if (rp.pair_mode == 0) { c0 = off + 2 * j; c1 = c0 + 1; }
  else { c0 = off + j; c1 = off + j + (da >> 1); }
  const int t = n / (rp.gh * rp.gw);
  const int rem = n - t * rp.gh * rp.gw;
  const int h = rem / rp.gw;
  const int w = rem - h * rp.gw;
  const int pos = axis == 0 ? t : (axis == 1 ? h : w);
  const float omega = exp2f(-((float)(2 * j) / (float)da) * rp.log2_theta);
  float s, c;
  sincosf((float)pos * omega, &s, &c);
  const float x0 = row[c0], x1 = row[c1];
  row[c0] = fmaf(x0, c, -x1 * s);
  row[c1] = fmaf(x0, s, x1 * c);
}

__global__ __launch_bounds__(kQ) void attn_naive_kernel(NaiveArgs a) {
  __shared__ float ks[kKeys][kHeadDim];
  __shared__ float vs[kKeys][kHeadDim];
  const int nqb = (a.Lq + kQ - 1) / kQ;
  const int qb = blockIdx.x % nqb;
  const int bh = blockIdx.x / nqb;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int i = qb * kQ + threadIdx.x;
  const bool live = i < a.Lq;
  const size_t tok = (size_t)a.H * kHeadDim;

  int lv = a.Lk;
  if (a.kv_valid_len) lv = min(max(a.kv_valid_len[b], 0), a.Lk);

  float qr[kHeadDim];
  float acc[kHeadDim];
  {
    const uint16_t* qp = a.q + ((size_t)b * a.Lq + (live ? i : 0)) * tok + (size_t)h * kHeadDim;
#pragma unroll
    for (int c = 0; c < kHeadDim; ++c) {
      qr[c] = live ? __uint_as_float((uint32_t)qp[c] << 16) : 0.f;
      acc[c] = 0.f;
    }
    if (a.rp.enabled && live && i < a.rp.n_rot) {
      for (int p = 0; p < kHeadDim / 2; ++p) rotate_pair_direct(a.rp, qr, i, p);
    }
  }
  float m = -INFINITY, l = 0.f;

  for (int k0 = 0; k0 < lv; k0 += kKeys) {
    __syncthreads();
    // stage kKeys keys/values: thread t fills channel pairs of rows
    for (int e = threadIdx.x; e < kKeys * kHeadDim; e += kQ) {
      const int r = e / kHeadDim, c = e % kHeadDim;
      const int n = k0 + r;
      float kv = 0.f, vv = 0.f;
      if (n < lv) {
        const size_t off = ((size_t)b * a.Lk + n) * tok + (size_t)h * kHeadDim + c;
        kv = __uint_as_float((uint32_t)a.k[off] << 16);
        vv = __uint_as_float((uint32_t)a.v[off] << 16);
      }
      ks[r][c] = kv;
      vs[r][c] = vv;
    }
    __syncthreads();
    if (a.rp.enabled) {
      for (int e = threadIdx.x; e < kKeys * (kHeadDim / 2); e += kQ) {
        const int r = e / (kHeadDim / 2), p = e % (kHeadDim / 2);
        const int n = k0 + r;
        if (n < lv && n < a.rp.n_rot && !a.rp.keys_prerotated) rotate_pair_direct(a.rp, ks[r], n, p);
      }
      __syncthreads();
    }
    const int nk = min(kKeys, lv - k0);
    for (int r = 0; r < nk; ++r) {
      float s = 0.f;
#pragma unroll
      for (int c = 0; c < kHeadDim; ++c) s = fmaf(qr[c], ks[r][c], s);
      s *= a.scale;
      const float mn = fmaxf(m, s);
      const float alpha = expf(m - mn);
      const float p = expf(s - mn);
      l = l * alpha + p;
#pragma unroll
      for (int c = 0; c < kHeadDim; ++c) acc[c] = fmaf(p, vs[r][c], acc[c] * alpha);
      m = mn;
    }
  }

  if (!live) return;
  uint16_t* op = a.o + ((size_t)b * a.Lq + i) * tok + (size_t)h * kHeadDim;
  const float inv = lv > 0 ? 1.f / l : 0.f;
#pragma unroll
  for (int c = 0; c < kHeadDim; ++c) op[c] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(acc[c] * inv));
  if (a.lse) a.lse[((size_t)b * a.H + h) * a.Lq + i] = lv > 0 ? m + logf(l) : -INFINITY;
}

}  // namespace

hipError_t launch_attn_naive(const uint16_t* q, const uint16_t* k, const uint16_t* v, uint16_t* o,
                             float* lse, int B, int H, int Lq, int Lk, float scale,
                             const int32_t* kv_valid_len, const RopeParams& rp, hipStream_t stream) {
  NaiveArgs a{q, k, v, o, lse, kv_valid_len, B, H, Lq, Lk, scale, rp};
  const long nqb = (Lq + kQ - 1) / kQ;
  const long grid = nqb * B * H;
  return launch_kernel(attn_naive_kernel, (unsigned)grid, (unsigned)kQ, stream, a);
}

}  // namespace vidax
