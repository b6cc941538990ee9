// Launchers of the gfx950 kernels (not part of the C ABI), implemented in the
// .hip files and called by the C ABI layer after validation.  Kept apart
// from the kernels' shared definitions so that a new entry point changes no
// file a kernel is built from.
#pragma once

#include "common.hpp"

// All pointers are device pointers; sizes already validated.
namespace vidax {

// Enqueues kernel(arg) on `stream` and returns the status of this launch
// alone (an error left behind by an earlier, unrelated HIP call is not
// reported as this launch's failure, as hipGetLastError would).
template <typename A>
inline hipError_t launch_kernel(void (*kernel)(A), unsigned grid, unsigned block, hipStream_t stream, A arg) {
  void* args[] = {&arg};
  return hipLaunchKernel(reinterpret_cast<const void*>(kernel), dim3(grid), dim3(block), args, 0, stream);
}

hipError_t launch_rope3d(const uint16_t* x, uint16_t* y, int B, int L, int H, const RopeParams& rp,
                         hipStream_t stream);
// Compute units of the current device (queried once per device).
int device_cu_count();

// Query-stream split of the backward's key-side kernel.  Its workgroups
// own 128 keys of one (b, h) and stream every query in 64-row tiles; when
// there are fewer of them than twice the compute units, the query tiles are
// cut into qsplit runs of qper tiles (at least 8 tiles a run, at most 16
// runs) so that about four workgroups per compute unit exist.  The fp32
// partial dK and dV of the runs follow D in the workspace, from a 256-byte
// aligned offset; `floats` is the workspace size this needs (B * H * Lq when
// qsplit is 1).
struct BwdSplit {
  int qsplit, qper;
  size_t part_offset, floats;
};

inline BwdSplit attn_bwd_split(int B, int H, int Lq, int Lk, int cus) {
  constexpr int kRows = 64, kOwn = 128;
  BwdSplit r;
  const size_t rows = (size_t)B * H * Lq;
  const int qtiles = (Lq + kRows - 1) / kRows;
  const long nkv = (long)((Lk + kOwn - 1) / kOwn) * B * H;
  r.qsplit = 1;
  if (nkv > 0 && nkv < 2L * cus) {
    long want = (4L * cus + nkv - 1) / nkv;
    const long cap = qtiles / 8;
    if (want > cap) want = cap;
    if (want > 16) want = 16;
    if (want > 1) r.qsplit = (int)want;
  }
  r.qper = (qtiles + r.qsplit - 1) / r.qsplit;
  r.part_offset = (rows + 63) / 64 * 64;
  r.floats = r.qsplit > 1 ? r.part_offset + 2 * (size_t)r.qsplit * B * Lk * H * kHeadDim : rows;
  return r;
}
// ws: D in its first B * H * Lq values; the split needs ws_floats >=
// attn_bwd_workspace_floats(...), fewer run unsplit.
hipError_t launch_attn_bwd(const uint16_t* q, const uint16_t* k, const uint16_t* v, const uint16_t* o,
                           const uint16_t* dout, const float* lse, float* ws, size_t ws_floats, uint16_t* dq,
                           uint16_t* dk, uint16_t* dv, int B, int H, int Lq, int Lk, float scale,
                           const int32_t* kv_valid_len, hipStream_t stream);
// The backward with D in the library's fixed device array (allocation-free
// entry point); B * H * Lq must not exceed kNoAllocRows.
constexpr long kNoAllocRows = 4194304;
hipError_t launch_attn_bwd_noalloc(const uint16_t* q, const uint16_t* k, const uint16_t* v, const uint16_t* o,
                                   const uint16_t* dout, const float* lse, uint16_t* dq, uint16_t* dk, uint16_t* dv,
                                   int B, int H, int Lq, int Lk, float scale, const int32_t* kv_valid_len,
                                   hipStream_t stream);
hipError_t launch_qk_norm(const uint16_t* x, uint16_t* y, const float* gain, float eps, int B, int L, int H,
                          const RopeParams& rp, hipStream_t stream);
hipError_t launch_attn_naive(const uint16_t* q, const uint16_t* k, const uint16_t* v, uint16_t* o,
                             float* lse, int B, int H, int Lq, int Lk, float scale,
                             const int32_t* kv_valid_len, const RopeParams& rp, hipStream_t stream);
bool attn_rope_supported(const RopeParams& rp);
hipError_t launch_na3d_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v, uint16_t* o, float* lse, int B,
                           int H, int T, int Hp, int Wp, int kt, int kh, int kw, int shift, float scale,
                           hipStream_t stream);
hipError_t launch_attn_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v, uint16_t* o,
                           float* lse, int B, int H, int Lq, int Lk, float scale,
                           const int32_t* kv_valid_len, const RopeParams& rp, hipStream_t stream);
// Short unrotated key sequences (text cross-attention): one persistent
// workgroup per CU (`cus` compute units).
hipError_t launch_xattn_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v, uint16_t* o, float* lse,
                            int B, int H, int Lq, int Lk, float scale, const int32_t* kv_valid_len, int cus,
                            hipStream_t stream);
hipError_t launch_qkv_proj(const uint16_t* x, const uint16_t* w, const float* bias, const float* gain_q,
                           const float* gain_k, float eps, uint16_t* q, uint16_t* k, uint16_t* v, int B, int L, int H,
                           int C, const RopeParams& rp, hipStream_t stream);
}  // namespace vidax
