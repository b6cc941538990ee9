/*
 * vidax.h -- C ABI of the MI355X (gfx950) video-attention hot path.
 *
 * Two operations of a video diffusion transformer's attention block, over
 * patchified multi-frame latent volumes (paper Section 2, "3D RoPE, 3D VAEs,
 * and flash attention"; Section 4 and the full benchmark table give the
 * workloads: tens of thousands of video tokens per sequence):
 *
 *   vidax_rope3d    3D rotary position embedding of query/key tokens over
 *                   their (time, height, width) latent coordinates.
 *   vidax_attn_fwd  non-causal softmax(scale * Q K^T) V, flash-attention style
 *                   (the score matrix is never materialised), with the 3D
 *                   rotation optionally fused into the Q/K loads and a
 *                   per-batch valid-key prefix that replaces a dense mask
 *                   (Appendix, porting-bug table, "Sharding, Parallelism &
 *                   Custom Kernels": skip invalid key blocks instead of
 *                   building a (B, H, Sq, Sk) mask).  The same entry point
 *                   serves self-attention (Lq == Lk), text cross-attention
 *                   (Lk = text length, no rotation) and joint video+text
 *                   attention (rotation on the video prefix only).
 *
 * Conventions shared by every entry point
 *   Layout    dense B x L x H x d ("BSHD"): element (b, n, h, c) sits at
 *             ((b * L + n) * H + h) * d + c, bfloat16 storage.  Offsets are
 *             64-bit inside the library.
 *   Ownership the caller allocates and owns every buffer (device memory).  The
 *             library never allocates, frees or synchronises, and keeps no
 *             state between calls -- except vidax_attn_bwd_noalloc, which
 *             works in a fixed device array of the library (one per GPU,
 *             held until the process ends) instead of a caller workspace.  Work is enqueued on `stream`
 *             (a hipStream_t; NULL = the legacy default stream).
 *   Alignment q, k, v, o, x, y must be 16-byte aligned; lse and kv_valid_len
 *             4-byte aligned.  A tensor pointer may be NULL only when that
 *             tensor has no elements.
 *   Errors    arguments are validated synchronously; on any error nothing is
 *             launched and a non-zero vidax_status is returned.  No C++
 *             exception crosses this boundary.  Faults inside a kernel surface
 *             at the caller's next synchronisation of `stream`.
 */
#ifndef VIDAX_H
#define VIDAX_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define VIDAX_ABI_VERSION 8

typedef enum vidax_status {
  VIDAX_OK = 0,
  VIDAX_ERR_INVALID_ARG = 1,  /* null/misaligned pointer, negative size, bad descriptor */
  VIDAX_ERR_UNSUPPORTED = 2,  /* valid request outside what the kernels implement (e.g. d != 128) */
  VIDAX_ERR_LAUNCH = 3,       /* the HIP runtime rejected the launch */
  VIDAX_ERR_TOO_LARGE = 4     /* the request exceeds a fixed device scratch size (allocation-free entry points) */
} vidax_status;

/*
 * 3D rotary embedding descriptor (paper Section 2: each family keeps its own
 * convention, so the convention is data, not code).
 *
 *   Tokens n < grid_t * grid_h * grid_w are video tokens in patchify order,
 *   n = (t * grid_h + h) * grid_w + w; later tokens (e.g. appended text) are
 *   left unrotated.  The head dim is split into consecutive channel blocks of
 *   widths dim_t, dim_h, dim_w (each even, >= 0, summing to d) for the t, h
 *   and w coordinates.  In the block of axis a (offset o_a, width d_a), pair
 *   j in [0, d_a/2) turns by phi = pos_a * theta^(-2j/d_a):
 *     (x0, x1) -> (x0 cos phi - x1 sin phi, x0 sin phi + x1 cos phi),
 *   with pair_mode 0 pairing channels (o_a+2j, o_a+2j+1) (interleaved) and
 *   pair_mode 1 pairing (o_a+j, o_a+j+d_a/2) (half split).
 *   Angles and the rotation are evaluated in fp32; results are rounded to
 *   bfloat16 (nearest even).
 */
typedef struct vidax_rope3d_desc {
  int32_t grid_t, grid_h, grid_w;
  int32_t dim_t, dim_h, dim_w;
  float theta;              /* > 0, finite; e.g. 10000 */
  int32_t pair_mode;        /* 0 interleaved, 1 half split */
  int32_t keys_prerotated;  /* attention only: 1 = k was already rotated (for
                               instance by vidax_rope3d), rotate q only; 0 = rotate
                               both inside the kernel.  vidax_rope3d ignores it. */
} vidax_rope3d_desc;

/*
 * y = rope3d(x).  x, y: bf16 [B, L, H, d] (device).  x == y (in place) is
 * allowed; other overlap is not.  Requires d == 128 (VIDAX_ERR_UNSUPPORTED
 * otherwise), 1 <= grid_t*grid_h*grid_w <= L, B, L, H >= 0 (zero-sized calls
 * are no-ops).  `rope` is a host pointer and must not be NULL.
 */
vidax_status vidax_rope3d(const void* x, void* y, int32_t B, int32_t L, int32_t H, int32_t d,
                          const vidax_rope3d_desc* rope, hipStream_t stream);

/*
 * y = R^T x: the transpose of vidax_rope3d (every pair rotated by minus its
 * angle), which carries a gradient with respect to rotated queries/keys back
 * to the unrotated ones (the rotation is orthogonal).  Same arguments and
 * requirements as vidax_rope3d.
 */
vidax_status vidax_rope3d_transpose(const void* x, void* y, int32_t B, int32_t L, int32_t H, int32_t d,
                                    const vidax_rope3d_desc* rope, hipStream_t stream);

/*
 * Query/key prologue of the served 3D-RoPE models (Section 3, "Supported
 * Models"; the paper gives no formula, the standard RMS normalisation is
 * used):  for every (batch, token, head) row x of d channels
 *
 *   y[c] = rope3d( x[c] / sqrt(mean_c'(x[c']^2) + eps) * gain[c] )
 *
 * computed in fp32 from the bf16 input and rounded to bf16 once.
 *   x, y : bf16 [B, L, H, d] (device); x == y (in place) is allowed, other
 *          overlap is not.
 *   gain : fp32 [d] on the device, shared by all heads, 16-byte aligned; or
 *          NULL for unit gain.
 *   eps  : >= 0 and finite (e.g. 1e-6); an all-zero row with eps = 0 gives NaN.
 *   rope : host pointer to a descriptor (as vidax_rope3d, either pair_mode;
 *          keys_prerotated is ignored), or NULL for normalisation and gain
 *          only.
 * Requires d == 128 (VIDAX_ERR_UNSUPPORTED otherwise); B, L, H >= 0
 * (zero-sized calls are no-ops).  HBM-bound: one read and one write of x.
 */
vidax_status vidax_qk_norm_rope(const void* x, void* y, const float* gain, float eps, int32_t B, int32_t L,
                                int32_t H, int32_t d, const vidax_rope3d_desc* rope, hipStream_t stream);

/*
 * o = softmax(scale * rope(q) rope(k)^T + mask) v, per batch b and head h.
 *
 *   q, o : bf16 [B, Lq, H, d] (device);  k, v : bf16 [B, Lk, H, d] (device).
 *   lse  : fp32 [B, H, Lq] natural-log sum-exp of the scaled scores of every
 *          query row (device), or NULL to skip it.
 *   scale: multiplies q.k (e.g. 1/sqrt(d) in fp32).
 *   kv_valid_len: int32 [B] on the device, or NULL (= Lk for every batch).
 *          Lv_b = clamp(kv_valid_len[b], 0, Lk): every query of batch b sees
 *          keys [0, Lv_b) only.  Rows with Lv_b = 0 produce o = 0, lse = -inf.
 *   rope : host pointer to a descriptor, or NULL for no rotation.  When given,
 *          query token n and key token n are rotated as in vidax_rope3d
 *          (fused into the loads; rotated values are rounded to bf16 before
 *          the matrix products).  With keys_prerotated = 1 only the queries
 *          are rotated in the kernel and k must hold keys already rotated
 *          with the same descriptor (vidax_rope3d): every query tile of a
 *          head re-rotates every key tile in the fused form, so one
 *          vidax_rope3d pass over k is cheaper at long sequence lengths.
 *          Half-split pairs (pair_mode 1) require keys_prerotated = 1 (the
 *          fused key rotation pairs interleaved channels).  Requires grid_t,
 *          grid_h, grid_w <= 1023, a rotary table of at most 4096 entries
 *          (VIDAX_ERR_UNSUPPORTED otherwise) and grid_t*grid_h*grid_w <=
 *          min(Lq, Lk).
 *   All Lq rows are computed; there is no causal mask.  Matrix products run
 *   on bf16 inputs with fp32 accumulation; the softmax is fp32.
 *   Requires d == 128; o must not alias q, k or v.  B, H, Lq, Lk >= 0.
 *   One batch of a tensor, max(Lq, Lk) * H * d * 2 bytes, must stay below
 *   2 GiB - 4 KiB (the kernels use 32-bit buffer offsets within a batch):
 *   VIDAX_ERR_UNSUPPORTED beyond; vidax_attn_fwd_naive has the same limit.
 */
vidax_status vidax_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse,
                            int32_t B, int32_t H, int32_t Lq, int32_t Lk, int32_t d, float scale,
                            const int32_t* kv_valid_len, const vidax_rope3d_desc* rope,
                            hipStream_t stream);

/*
 * Gradient of vidax_attn_fwd without rotation (for post-training, named as the
 * next direction in Section 5, "Conclusions & Future Work"): for every batch
 * b and head h, with keys j < Lv_b and P = exp(scale q k^T - lse),
 *
 *   dv = P^T dout,  ds = P * (dout v^T - D),  D_i = <dout_i, o_i>,
 *   dq = scale ds k,  dk = scale ds^T q;   keys j >= Lv_b get dk = dv = 0,
 *   a batch with Lv_b = 0 gets dq = 0.
 *
 *   q, o, dout, dq : bf16 [B, Lq, H, d];  k, v, dk, dv : bf16 [B, Lk, H, d]
 *   lse   : fp32 [B, H, Lq], the natural-log sum-exp vidax_attn_fwd returned
 *           with the same q, k, v, scale and kv_valid_len (o is its output).
 *   workspace : fp32 device workspace owned by the caller, workspace_floats
 *           values, at least B * H * Lq (VIDAX_ERR_INVALID_ARG below); its
 *           first B * H * Lq values hold D on return (layout [B, H, Lq]).
 *           With at least vidax_attn_bwd_workspace_floats(B, H, Lq, Lk, d)
 *           values the key-side kernels may cut the query stream into runs
 *           handled by separate workgroups, their partial dK and dV summed
 *           in fp32 in the rest of the workspace (faster when
 *           B * H * ceil(Lk / 128) is small against the compute units, e.g.
 *           text cross-attention); with fewer they run unsplit.  Both give
 *           the same gradients up to the order of the fp32 sums.
 *   scale, kv_valid_len: as for vidax_attn_fwd.
 * q and k are the vectors the scores were formed from: when the forward
 * rotated them, pass the rotated ones (vidax_rope3d) and take dq, dk back
 * through vidax_rope3d_transpose.  All device pointers 16-byte aligned (lse,
 * workspace too); outputs and the workspace must not overlap each other or
 * any input.  Products
 * run on bf16 inputs (P and ds rounded to bf16) with fp32 accumulation.
 * Requires d == 128 (VIDAX_ERR_UNSUPPORTED otherwise); B, H, Lq, Lk >= 0.
 * Buffer offsets are 32-bit and relative to a 64-row tile: 64 * H * d * 2
 * bytes must stay below 2 GiB - 4 KiB (VIDAX_ERR_UNSUPPORTED beyond).
 */
vidax_status vidax_attn_bwd(const void* q, const void* k, const void* v, const void* o, const void* dout,
                            const float* lse, void* dq, void* dk, void* dv, float* workspace,
                            size_t workspace_floats, int32_t B, int32_t H, int32_t Lq, int32_t Lk, int32_t d,
                            float scale, const int32_t* kv_valid_len, hipStream_t stream);

/*
 * fp32 values of vidax_attn_bwd's workspace with which it splits the query
 * stream of its key-side kernels on the current device (the split depends on
 * the device's compute-unit count); B * H * Lq when it would not split; 0 for
 * invalid arguments (a negative size, d != 128, a product that overflows).
 * Makes no device call besides querying the current device's attributes.
 */
size_t vidax_attn_bwd_workspace_floats(int32_t B, int32_t H, int32_t Lq, int32_t Lk, int32_t d);

/*
 * Allocation-free variant of vidax_attn_bwd, for callers that cannot allocate
 * device memory or pass a workspace (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc).  Same arguments, meaning,
 * layouts, results and errors as vidax_attn_bwd without a workspace (it runs
 * unsplit, so its gradients equal those of vidax_attn_bwd given a workspace
 * of exactly B * H * Lq values): D lives in a
 * fixed device array of the library (VIDAX_NOALLOC_MAX_ROWS fp32 values,
 * 16 MiB, one copy per GPU, looked up once per device on the first call with
 * that device current and held until the process ends).  The call itself
 * allocates nothing.
 *   B * H * Lq > VIDAX_NOALLOC_MAX_ROWS -> VIDAX_ERR_TOO_LARGE (nothing launched);
 *   the device array cannot be located -> VIDAX_ERR_LAUNCH.
 * Every call on one GPU shares that GPU's array: calls that overlap in time on
 * one GPU (different streams, or different host threads without ordering)
 * race and give undefined results; calls ordered on one stream are safe.
 * The array is fully rewritten by each call before it is read (nothing needs
 * to start at zero).
 */
#define VIDAX_NOALLOC_MAX_ROWS 4194304
vidax_status vidax_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o, const void* dout,
                                    const float* lse, void* dq, void* dk, void* dv, int32_t B, int32_t H,
                                    int32_t Lq, int32_t Lk, int32_t d, float scale, const int32_t* kv_valid_len,
                                    hipStream_t stream);

/*
 * 3D neighbourhood (windowed) attention, the attention of the LTX-2.5 VAE
 * decoder (Section 2, "3D RoPE, 3D VAEs, and flash attention"; porting-bug
 * table, "Memory, Tiling & Execution Graphs"): on a token grid of
 * grid_t x grid_h x grid_w (L = grid_t * grid_h * grid_w tokens, patchify
 * order n = (t * grid_h + h) * grid_w + w), query (t, h, w) attends to the
 * keys (t', h', w') of its window, per axis an inclusive range of odd size
 * win around the query's coordinate c on an axis of N positions:
 *   border 0 (clip):  [max(0, c - r), min(N - 1, c + r)], r = (win - 1) / 2;
 *   border 1 (shift): the window keeps win positions, moved inward at the
 *                     border: start clamp(c - r, 0, N - win) (whole axis if
 *                     N <= win).
 *   o_i = softmax_j(scale <q_i, k_j>) v_j over the window, lse_i its
 *   natural-log sum-exp.
 *
 *   q, k, v, o : bf16 [B, L, H, d] device pointers, 16-byte aligned
 *   lse        : fp32 [B, H, L] device pointer (4-byte aligned) or NULL
 *   win_t, win_h, win_w: odd >= 1 (VIDAX_ERR_INVALID_ARG otherwise);
 *                win_w <= 11 (VIDAX_ERR_UNSUPPORTED beyond)
 *   scale: finite.  Requires d == 128 (VIDAX_ERR_UNSUPPORTED otherwise).
 * o and lse must not overlap each other or q, k, v.  Scores
 * are fp32 sums of bf16 products; the probabilities are rounded to bf16
 * before the product with v, as in vidax_attn_fwd.
 */
vidax_status vidax_na3d_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int32_t B, int32_t H,
                            int32_t grid_t, int32_t grid_h, int32_t grid_w, int32_t d, int32_t win_t, int32_t win_h,
                            int32_t win_w, int32_t border, float scale, hipStream_t stream);

/*
 * Q/K/V projection with the query/key prologue in its epilogue: the step that
 * produces an attention call's inputs in the served video DiTs (Section 3,
 * "Supported Models"; rotation as in Section 2).  With M = B * L tokens,
 *
 *   y = x W^T (+ bias)           x: bf16 [M, C], W: bf16 [3 H d, C] (rows =
 *                                output channels: q heads, k heads, v heads),
 *                                bias: fp32 [3 H d] or NULL
 *   q = rope(rms_norm(y_q) * gain_q),  k = rope(rms_norm(y_k) * gain_k),  v = y_v
 *
 * where rms_norm acts on each (token, head) over its d channels with eps, as
 * in vidax_qk_norm_rope; gains fp32 [d] (shared by the heads) or NULL (unit);
 * rope as vidax_rope3d (token n of each sequence of L, either pair_mode), or
 * NULL for none.  q, k, v: bf16 [B, L, H, d] outputs, rounded once.
 * fp32 accumulation.  All pointers 16-byte aligned; outputs must not overlap
 * each other or an input.  Requires d == 128 and C a multiple of 64
 * (VIDAX_ERR_UNSUPPORTED otherwise); eps >= 0 finite.
 */
vidax_status vidax_qkv_proj(const void* x, const void* w, const float* bias, const float* gain_q,
                            const float* gain_k, float eps, void* q, void* k, void* v, int32_t B, int32_t L,
                            int32_t H, int32_t d, int32_t C, const vidax_rope3d_desc* rope, hipStream_t stream);

/*
 * Same contract as vidax_attn_fwd, computed by a plain scalar fp32 kernel (one
 * thread per query row, rotation evaluated on the fly, no matrix cores).  It
 * exists as an independent second GPU implementation for cross-checks at
 * small sizes; it also accepts pair_mode 1.  Slow: O(Lq * Lk * d) per head
 * with no reuse.
 */
vidax_status vidax_attn_fwd_naive(const void* q, const void* k, const void* v, void* o, float* lse,
                                  int32_t B, int32_t H, int32_t Lq, int32_t Lk, int32_t d, float scale,
                                  const int32_t* kv_valid_len, const vidax_rope3d_desc* rope,
                                  hipStream_t stream);

/* Static string describing a status code (never NULL; any int32_t value is
 * accepted, codes that are not a vidax_status give "unknown status"). */
const char* vidax_status_string(int32_t status);

/* VIDAX_ABI_VERSION of the loaded library. */
int32_t vidax_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* VIDAX_H */
