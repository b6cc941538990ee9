// C ABI of libvidax: argument validation and dispatch to the gfx950 kernels.
//
// Every check runs before any HIP call, so a rejected call has no side effect
// (and can be exercised on a machine without a GPU).
#include <math.h>
#include <stdint.h>

#include "../../include/vidax.h"
#include "launch.hpp"

static_assert(VIDAX_NOALLOC_MAX_ROWS == vidax::kNoAllocRows, "allocation-free scratch size");

namespace {

using vidax::RopeParams;

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

// [p, p + bytes) and [q, q + bytes_q) overlap?
bool overlaps(const void* p, uint64_t bytes, const void* q, uint64_t bytes_q) {
  if (bytes == 0 || bytes_q == 0) return false;
  const uintptr_t a0 = (uintptr_t)p, a1 = a0 + bytes;
  const uintptr_t b0 = (uintptr_t)q, b1 = b0 + bytes_q;
  return a0 < b1 && b0 < a1;
}

// Elements of a [B, L, H, d] tensor, or -1 if it does not fit in int64 byte offsets.
int64_t numel4(int64_t B, int64_t L, int64_t H, int64_t d) {
  const int64_t lim = INT64_C(1) << 60;
  int64_t n = 1;
  for (int64_t x : {B, L, H, d}) {
    if (x != 0 && n > lim / x) return -1;
    n *= x;
  }
  return n;
}

// Validates a rotary descriptor against the token counts it will see and
// converts it.  `max_tokens`: rotated tokens must not exceed it.
vidax_status make_rope(const vidax_rope3d_desc* r, int64_t max_tokens, int32_t d, RopeParams* out) {
  if (r->grid_t < 1 || r->grid_h < 1 || r->grid_w < 1) return VIDAX_ERR_INVALID_ARG;
  if (r->dim_t < 0 || r->dim_h < 0 || r->dim_w < 0) return VIDAX_ERR_INVALID_ARG;
  if ((r->dim_t | r->dim_h | r->dim_w) & 1) return VIDAX_ERR_INVALID_ARG;
  if ((int64_t)r->dim_t + r->dim_h + r->dim_w != d) return VIDAX_ERR_INVALID_ARG;
  if (!(r->theta > 0.0f) || !isfinite(r->theta)) return VIDAX_ERR_INVALID_ARG;
  if (r->pair_mode != 0 && r->pair_mode != 1) return VIDAX_ERR_INVALID_ARG;
  if (r->keys_prerotated != 0 && r->keys_prerotated != 1) return VIDAX_ERR_INVALID_ARG;
  const int64_t n_rot = (int64_t)r->grid_t * r->grid_h * r->grid_w;
  if (n_rot > max_tokens) return VIDAX_ERR_INVALID_ARG;
  const int64_t entries = (int64_t)r->grid_t * (r->dim_t / 2) + (int64_t)r->grid_h * (r->dim_h / 2) +
                          (int64_t)r->grid_w * (r->dim_w / 2);
  if (entries > vidax::kRopeTableMax) return VIDAX_ERR_UNSUPPORTED;
  out->enabled = 1;
  out->gt = r->grid_t;
  out->gh = r->grid_h;
  out->gw = r->grid_w;
  out->dt = r->dim_t;
  out->dh = r->dim_h;
  out->dw = r->dim_w;
  out->pair_mode = r->pair_mode;
  out->keys_prerotated = r->keys_prerotated;
  out->inverse = 0;
  out->n_rot = (int)n_rot;
  out->base1 = r->grid_t * (r->dim_t / 2);
  out->base2 = out->base1 + r->grid_h * (r->dim_h / 2);
  out->n_entries = (int)entries;
  out->log2_theta = log2f(r->theta);
  return VIDAX_OK;
}

RopeParams no_rope() {
  RopeParams p{};
  p.enabled = 0;
  p.gt = p.gh = p.gw = 1;
  return p;
}

enum class AttnImpl { kMatrixCore, kNaive };

vidax_status attn_common(AttnImpl impl, const void* q, const void* k, const void* v, void* o, float* lse,
                         int32_t B, int32_t H, int32_t Lq, int32_t Lk, int32_t d, float scale,
                         const int32_t* kv_valid_len, const vidax_rope3d_desc* rope, hipStream_t stream) {
  if (B < 0 || H < 0 || Lq < 0 || Lk < 0 || d < 0) return VIDAX_ERR_INVALID_ARG;
  const int64_t nq = numel4(B, Lq, H, d), nk = numel4(B, Lk, H, d);
  if (nq < 0 || nk < 0) return VIDAX_ERR_INVALID_ARG;
  // a pointer may be NULL only when its tensor has no elements
  if ((nq > 0 && (!q || !o)) || (nk > 0 && (!k || !v))) return VIDAX_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16)) return VIDAX_ERR_INVALID_ARG;
  if (lse && !aligned(lse, 4)) return VIDAX_ERR_INVALID_ARG;
  if (kv_valid_len && !aligned(kv_valid_len, 4)) return VIDAX_ERR_INVALID_ARG;
  if (!isfinite(scale)) return VIDAX_ERR_INVALID_ARG;
  if (d != vidax::kHeadDim) return VIDAX_ERR_UNSUPPORTED;
  const uint64_t qbytes = (uint64_t)nq * 2, kbytes = (uint64_t)nk * 2;
  if (overlaps(o, qbytes, q, qbytes) || overlaps(o, qbytes, k, kbytes) || overlaps(o, qbytes, v, kbytes))
    return VIDAX_ERR_INVALID_ARG;
  // outputs (o, lse) must not overlap each other or any input (kv_valid_len included)
  const uint64_t lbytes = lse ? (uint64_t)B * H * Lq * 4 : 0, vbytes = kv_valid_len ? (uint64_t)B * 4 : 0;
  if (overlaps(lse, lbytes, o, qbytes) || overlaps(lse, lbytes, q, qbytes) || overlaps(lse, lbytes, k, kbytes) ||
      overlaps(lse, lbytes, v, kbytes) || overlaps(kv_valid_len, vbytes, o, qbytes) ||
      overlaps(kv_valid_len, vbytes, lse, lbytes))
    return VIDAX_ERR_INVALID_ARG;
  RopeParams rp = no_rope();
  if (rope) {
    const vidax_status st = make_rope(rope, Lq < Lk ? Lq : Lk, d, &rp);
    if (st != VIDAX_OK) return st;
    if (impl == AttnImpl::kMatrixCore && !vidax::attn_rope_supported(rp)) return VIDAX_ERR_UNSUPPORTED;
  }
  // the kernels address one batch of q, o (and of k, v within a tile) with
  // 32-bit buffer offsets: one batch of a tensor must stay below 2 GiB
  if ((int64_t)(Lq > Lk ? Lq : Lk) * H * d * 2 > INT32_MAX - 4096) return VIDAX_ERR_UNSUPPORTED;
  // one workgroup per 256 (matrix core) or 64 (naive) query rows of each (b, h)
  const int64_t rows = impl == AttnImpl::kMatrixCore ? 256 : 64;
  const int64_t grid = ((int64_t)Lq + rows - 1) / rows * B * H;
  if (grid > INT32_MAX) return VIDAX_ERR_UNSUPPORTED;
  if (B == 0 || H == 0 || Lq == 0) return VIDAX_OK;

  hipError_t e;
  if (impl == AttnImpl::kMatrixCore)
    e = vidax::launch_attn_fwd((const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)v, (uint16_t*)o, lse, B, H,
                               Lq, Lk, scale, kv_valid_len, rp, stream);
  else
    e = vidax::launch_attn_naive((const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)v, (uint16_t*)o, lse, B,
                                 H, Lq, Lk, scale, kv_valid_len, rp, stream);
  return e == hipSuccess ? VIDAX_OK : VIDAX_ERR_LAUNCH;
}

vidax_status rope3d_common(bool inverse, const void* x, void* y, int32_t B, int32_t L, int32_t H, int32_t d,
                          const vidax_rope3d_desc* rope, hipStream_t stream) {
  if (B < 0 || L < 0 || H < 0 || d < 0) return VIDAX_ERR_INVALID_ARG;
  if (!rope) return VIDAX_ERR_INVALID_ARG;
  const int64_t n = numel4(B, L, H, d);
  if (n < 0) return VIDAX_ERR_INVALID_ARG;
  if (n > 0 && (!x || !y)) return VIDAX_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(y, 16)) return VIDAX_ERR_INVALID_ARG;
  if (d != vidax::kHeadDim) return VIDAX_ERR_UNSUPPORTED;
  if (x != y && overlaps(x, (uint64_t)n * 2, y, (uint64_t)n * 2)) return VIDAX_ERR_INVALID_ARG;
  vidax_rope3d_desc r = *rope;
  r.keys_prerotated = 0;  // attention-only field
  RopeParams rp;
  const vidax_status st = make_rope(&r, L, d, &rp);
  if (st != VIDAX_OK) return st;
  rp.inverse = inverse ? 1 : 0;
  if (B == 0 || L == 0 || H == 0) return VIDAX_OK;
  const hipError_t e = vidax::launch_rope3d((const uint16_t*)x, (uint16_t*)y, B, L, H, rp, stream);
  return e == hipSuccess ? VIDAX_OK : VIDAX_ERR_LAUNCH;
}

// The backward's checks; `noalloc`: D goes to the library's fixed device
// array (the workspace must be NULL, of 0 values) instead of the caller's.
vidax_status bwd_common(bool noalloc, const void* q, const void* k, const void* v, const void* o, const void* dout,
                        const float* lse, void* dq, void* dk, void* dv, float* ws, size_t ws_floats, int32_t B,
                        int32_t H, int32_t Lq, int32_t Lk, int32_t d, float scale, const int32_t* kv_valid_len,
                        hipStream_t stream) {
  if (B < 0 || H < 0 || Lq < 0 || Lk < 0 || d < 0) return VIDAX_ERR_INVALID_ARG;
  const int64_t nq = numel4(B, Lq, H, d), nk = numel4(B, Lk, H, d);
  if (nq < 0 || nk < 0) return VIDAX_ERR_INVALID_ARG;
  const int64_t nrow = (int64_t)B * H * Lq;  // lse, D
  if ((nq > 0 && (!q || !o || !dout || !dq)) || (nk > 0 && (!k || !v || !dk || !dv)) ||
      (nrow > 0 && (!lse || (!noalloc && !ws))))
    return VIDAX_ERR_INVALID_ARG;
  if (noalloc && (ws || ws_floats)) return VIDAX_ERR_INVALID_ARG;
  if (!noalloc && (uint64_t)ws_floats < (uint64_t)nrow) return VIDAX_ERR_INVALID_ARG;
  if (ws_floats > ((uint64_t)1 << 60)) return VIDAX_ERR_INVALID_ARG;
  if (!ws) ws_floats = 0;
  for (const void* p : {q, k, v, o, dout, (const void*)dq, (const void*)dk, (const void*)dv})
    if (!aligned(p, 16)) return VIDAX_ERR_INVALID_ARG;
  if (!aligned(lse, 16) || !aligned(ws, 16)) return VIDAX_ERR_INVALID_ARG;
  if (kv_valid_len && !aligned(kv_valid_len, 4)) return VIDAX_ERR_INVALID_ARG;
  if (!isfinite(scale)) return VIDAX_ERR_INVALID_ARG;
  if (d != vidax::kHeadDim) return VIDAX_ERR_UNSUPPORTED;
  const uint64_t qb = (uint64_t)nq * 2, kb = (uint64_t)nk * 2, rb = (uint64_t)nrow * 4;
  const uint64_t vb = kv_valid_len ? (uint64_t)B * 4 : 0;
  // outputs (dq, dk, dv, the workspace) must not overlap each other or any input
  const void* outs[4] = {dq, dk, dv, ws};
  const uint64_t osz[4] = {qb, kb, kb, (uint64_t)ws_floats * 4};
  const void* ins[7] = {q, k, v, o, dout, lse, kv_valid_len};
  const uint64_t isz[7] = {qb, kb, kb, qb, qb, rb, vb};
  for (int i = 0; i < 4; ++i) {
    for (int j = 0; j < 7; ++j)
      if (overlaps(outs[i], osz[i], ins[j], isz[j])) return VIDAX_ERR_INVALID_ARG;
    for (int j = i + 1; j < 4; ++j)
      if (overlaps(outs[i], osz[i], outs[j], osz[j])) return VIDAX_ERR_INVALID_ARG;
  }
  // grids: dq up to ceil(Lq / 128) B H, key side up to 16 ceil(Lk / 128) B H
  const int64_t grid_q = ((int64_t)Lq + 127) / 128 * B * H, grid_k = ((int64_t)Lk + 127) / 128 * 16 * B * H;
  if (grid_q > INT32_MAX || grid_k > INT32_MAX) return VIDAX_ERR_UNSUPPORTED;
  // buffer offsets are 32-bit and relative to a 64-row tile
  if ((int64_t)64 * H * d * 2 > INT32_MAX - 4096) return VIDAX_ERR_UNSUPPORTED;
  if (noalloc && nrow > vidax::kNoAllocRows) return VIDAX_ERR_TOO_LARGE;
  if (B == 0 || H == 0 || (Lq == 0 && Lk == 0)) return VIDAX_OK;
  const hipError_t e =
      noalloc ? vidax::launch_attn_bwd_noalloc((const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)v,
                                               (const uint16_t*)o, (const uint16_t*)dout, lse, (uint16_t*)dq,
                                               (uint16_t*)dk, (uint16_t*)dv, B, H, Lq, Lk, scale, kv_valid_len, stream)
              : vidax::launch_attn_bwd((const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)v, (const uint16_t*)o,
                                       (const uint16_t*)dout, lse, ws, ws_floats, (uint16_t*)dq, (uint16_t*)dk,
                                       (uint16_t*)dv, B, H, Lq, Lk, scale, kv_valid_len, stream);
  return e == hipSuccess ? VIDAX_OK : VIDAX_ERR_LAUNCH;
}

}  // namespace

extern "C" {

vidax_status vidax_attn_bwd(const void* q, const void* k, const void* v, const void* o, const void* dout,
                            const float* lse, void* dq, void* dk, void* dv, float* workspace,
                            size_t workspace_floats, int32_t B, int32_t H, int32_t Lq, int32_t Lk, int32_t d,
                            float scale, const int32_t* kv_valid_len, hipStream_t stream) {
  return bwd_common(false, q, k, v, o, dout, lse, dq, dk, dv, workspace, workspace_floats, B, H, Lq, Lk, d, scale,
                    kv_valid_len, stream);
}

size_t vidax_attn_bwd_workspace_floats(int32_t B, int32_t H, int32_t Lq, int32_t Lk, int32_t d) {
  if (B < 0 || H < 0 || Lq < 0 || Lk < 0 || d != vidax::kHeadDim) return 0;
  if (numel4(B, Lq, H, d) < 0 || numel4(B, Lk, H, d) < 0) return 0;
  return vidax::attn_bwd_split(B, H, Lq, Lk, vidax::device_cu_count()).floats;
}

vidax_status vidax_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o, const void* dout,
                                    const float* lse, void* dq, void* dk, void* dv, int32_t B, int32_t H,
                                    int32_t Lq, int32_t Lk, int32_t d, float scale, const int32_t* kv_valid_len,
                                    hipStream_t stream) {
  return bwd_common(true, q, k, v, o, dout, lse, dq, dk, dv, nullptr, 0, B, H, Lq, Lk, d, scale, kv_valid_len,
                    stream);
}

vidax_status vidax_qk_norm_rope(const void* x, void* y, const float* gain, float eps, int32_t B, int32_t L, int32_t H,
                                int32_t d, const vidax_rope3d_desc* rope, hipStream_t stream) {
  if (B < 0 || L < 0 || H < 0 || d < 0) return VIDAX_ERR_INVALID_ARG;
  const int64_t n = numel4(B, L, H, d);
  if (n < 0) return VIDAX_ERR_INVALID_ARG;
  if (n > 0 && (!x || !y)) return VIDAX_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(y, 16) || !aligned(gain, 16)) return VIDAX_ERR_INVALID_ARG;
  if (!(eps >= 0.0f) || !isfinite(eps)) return VIDAX_ERR_INVALID_ARG;
  if (d != vidax::kHeadDim) return VIDAX_ERR_UNSUPPORTED;
  if (x != y && overlaps(x, (uint64_t)n * 2, y, (uint64_t)n * 2)) return VIDAX_ERR_INVALID_ARG;
  if (gain && overlaps(gain, (uint64_t)d * 4, y, (uint64_t)n * 2)) return VIDAX_ERR_INVALID_ARG;
  RopeParams rp = no_rope();
  if (rope) {
    vidax_rope3d_desc r = *rope;
    r.keys_prerotated = 0;  // attention-only field
    const vidax_status st = make_rope(&r, L, d, &rp);
    if (st != VIDAX_OK) return st;
  }
  if (B == 0 || L == 0 || H == 0) return VIDAX_OK;
  const hipError_t e = vidax::launch_qk_norm((const uint16_t*)x, (uint16_t*)y, gain, eps, B, L, H, rp, stream);
  return e == hipSuccess ? VIDAX_OK : VIDAX_ERR_LAUNCH;
}

vidax_status vidax_rope3d(const void* x, void* y, int32_t B, int32_t L, int32_t H, int32_t d,
                          const vidax_rope3d_desc* rope, hipStream_t stream) {
  return rope3d_common(false, x, y, B, L, H, d, rope, stream);
}

vidax_status vidax_rope3d_transpose(const void* x, void* y, int32_t B, int32_t L, int32_t H, int32_t d,
                                    const vidax_rope3d_desc* rope, hipStream_t stream) {
  return rope3d_common(true, x, y, B, L, H, d, rope, stream);
}

vidax_status vidax_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int32_t B, int32_t H,
                            int32_t Lq, int32_t Lk, int32_t d, float scale, const int32_t* kv_valid_len,
                            const vidax_rope3d_desc* rope, hipStream_t stream) {
  return attn_common(AttnImpl::kMatrixCore, q, k, v, o, lse, B, H, Lq, Lk, d, scale, kv_valid_len, rope, stream);
}

vidax_status vidax_attn_fwd_naive(const void* q, const void* k, const void* v, void* o, float* lse, int32_t B,
                                  int32_t H, int32_t Lq, int32_t Lk, int32_t d, float scale,
                                  const int32_t* kv_valid_len, const vidax_rope3d_desc* rope, hipStream_t stream) {
  return attn_common(AttnImpl::kNaive, q, k, v, o, lse, B, H, Lq, Lk, d, scale, kv_valid_len, rope, stream);
}

vidax_status vidax_na3d_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int32_t B, int32_t H,
                            int32_t grid_t, int32_t grid_h, int32_t grid_w, int32_t d, int32_t win_t, int32_t win_h,
                            int32_t win_w, int32_t border, float scale, hipStream_t stream) {
  if (B < 0 || H < 0 || grid_t < 0 || grid_h < 0 || grid_w < 0 || d < 0) return VIDAX_ERR_INVALID_ARG;
  for (int32_t w : {win_t, win_h, win_w})
    if (w < 1 || (w & 1) == 0) return VIDAX_ERR_INVALID_ARG;
  if (border != 0 && border != 1) return VIDAX_ERR_INVALID_ARG;
  if (!isfinite(scale)) return VIDAX_ERR_INVALID_ARG;
  const int64_t L = (int64_t)grid_t * grid_h * grid_w;
  const int64_t n = numel4(B, L, H, d);
  if (n < 0) return VIDAX_ERR_INVALID_ARG;
  if (n > 0 && (!q || !k || !v || !o)) return VIDAX_ERR_INVALID_ARG;
  for (const void* p : {q, k, v, (const void*)o})
    if (!aligned(p, 16)) return VIDAX_ERR_INVALID_ARG;
  if (!aligned(lse, 4)) return VIDAX_ERR_INVALID_ARG;
  if (d != vidax::kHeadDim) return VIDAX_ERR_UNSUPPORTED;
  if (win_w > 11) return VIDAX_ERR_UNSUPPORTED;  // a wave's key runs are 16 positions along w
  if (n == 0) return VIDAX_OK;
  const uint64_t xb = (uint64_t)n * 2, lb = lse ? (uint64_t)B * H * L * 4 : 0;
  // outputs must not overlap each other or an input
  for (const void* in : {q, k, v})
    if (overlaps(o, xb, in, xb) || overlaps(lse, lb, in, xb)) return VIDAX_ERR_INVALID_ARG;
  if (overlaps(o, xb, lse, lb)) return VIDAX_ERR_INVALID_ARG;
  // 32-bit buffer offsets within one batch (plus a staged row past its end);
  // launch size
  if ((L + 32) * H * 256 > INT32_MAX) return VIDAX_ERR_UNSUPPORTED;
  const int64_t nwg = (int64_t)B * H * ((grid_t + 1) / 2) * ((grid_h + 3) / 4) * ((grid_w + 15) / 16);
  if (nwg > INT32_MAX) return VIDAX_ERR_UNSUPPORTED;
  const hipError_t e =
      vidax::launch_na3d_fwd((const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)v, (uint16_t*)o, lse, B, H,
                             grid_t, grid_h, grid_w, win_t, win_h, win_w, border, scale, stream);
  return e == hipSuccess ? VIDAX_OK : VIDAX_ERR_LAUNCH;
}

vidax_status vidax_qkv_proj(const void* x, const void* w, const float* bias, const float* gain_q,
                            const float* gain_k, float eps, void* q, void* k, void* v, int32_t B, int32_t L,
                            int32_t H, int32_t d, int32_t C, const vidax_rope3d_desc* rope, hipStream_t stream) {
  if (B < 0 || L < 0 || H < 0 || d < 0 || C < 0) return VIDAX_ERR_INVALID_ARG;
  const int64_t M = (int64_t)B * L;
  const int64_t nx = numel4(M, C, 1, 1), nw = numel4(3, H, d, C), no = numel4(M, H, d, 1);
  if (nx < 0 || nw < 0 || no < 0) return VIDAX_ERR_INVALID_ARG;
  if (!(eps >= 0.0f) || !isfinite(eps)) return VIDAX_ERR_INVALID_ARG;
  if (no > 0 && (!q || !k || !v || (C > 0 && (!x || !w)))) return VIDAX_ERR_INVALID_ARG;
  for (const void* p : {x, w, (const void*)bias, (const void*)gain_q, (const void*)gain_k, (const void*)q,
                        (const void*)k, (const void*)v})
    if (!aligned(p, 16)) return VIDAX_ERR_INVALID_ARG;
  if (d != vidax::kHeadDim) return VIDAX_ERR_UNSUPPORTED;
  if (C % 64 != 0 || (C == 0 && no > 0)) return VIDAX_ERR_UNSUPPORTED;  // stages of 64 input channels
  RopeParams rp = no_rope();
  if (rope) {
    vidax_rope3d_desc r = *rope;
    r.keys_prerotated = 0;  // attention-only field
    const vidax_status st = make_rope(&r, L, d, &rp);
    if (st != VIDAX_OK) return st;
  }
  if (no == 0) return VIDAX_OK;
  const uint64_t ob = (uint64_t)no * 2;
  const void* outs[3] = {q, k, v};
  const void* ins[5] = {x, w, bias, gain_q, gain_k};
  const uint64_t isz[5] = {(uint64_t)nx * 2, (uint64_t)nw * 2, bias ? (uint64_t)3 * H * d * 4 : 0,
                           gain_q ? (uint64_t)d * 4 : 0, gain_k ? (uint64_t)d * 4 : 0};
  for (int i = 0; i < 3; ++i) {
    for (int j = 0; j < 5; ++j)
      if (overlaps(outs[i], ob, ins[j], isz[j])) return VIDAX_ERR_INVALID_ARG;
    for (int j = i + 1; j < 3; ++j)
      if (overlaps(outs[i], ob, outs[j], ob)) return VIDAX_ERR_INVALID_ARG;
  }
  // 32-bit buffer offsets within a 256-row tile; launch size
  if ((int64_t)256 * C * 2 > INT32_MAX) return VIDAX_ERR_UNSUPPORTED;
  const int64_t nwg = ((int64_t)3 * H * d + 255) / 256 * ((M + 255) / 256);
  if (nwg > INT32_MAX || M > INT32_MAX) return VIDAX_ERR_UNSUPPORTED;
  const hipError_t e = vidax::launch_qkv_proj((const uint16_t*)x, (const uint16_t*)w, bias, gain_q, gain_k, eps,
                                              (uint16_t*)q, (uint16_t*)k, (uint16_t*)v, B, L, H, C, rp, stream);
  return e == hipSuccess ? VIDAX_OK : VIDAX_ERR_LAUNCH;
}

const char* vidax_status_string(int32_t status) {
  switch (status) {
    case VIDAX_OK: return "ok";
    case VIDAX_ERR_INVALID_ARG: return "invalid argument";
    case VIDAX_ERR_UNSUPPORTED: return "unsupported configuration";
    case VIDAX_ERR_LAUNCH: return "kernel launch failed";
    case VIDAX_ERR_TOO_LARGE: return "request exceeds the fixed device scratch of an allocation-free entry point";
  }
  return "unknown status";
}

int32_t vidax_abi_version(void) { return VIDAX_ABI_VERSION; }

}  // extern "C"
