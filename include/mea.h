/*
 * mea.h - memory-efficient exact attention on MI355X (gfx950), C ABI.
 *
 * Computes dense softmax attention exactly (Rabe & Staats, "Self-attention
 * Does Not Need O(n^2) Memory", arXiv 2112.05682):
 *   Section 1: s_ij = dot(q_i, k_j), w_ij = softmax_j(s_ij),
 *              o_i = sum_j w_ij v_j;
 *   Section 4: q is scaled before the dot product (by 1/sqrt(d) there; here
 *              an explicit `scale`, so s_ij = scale * dot(q_i, k_j)).
 * The keys are consumed tile by tile with the lazy softmax of Section 2
 * (Eq. 1) made stable by the running maximum of Section 3: a running row
 * max m, a rescaled running numerator sum_j e^{s_j - m} v_j and a running
 * denominator sum_j e^{s_j - m}, divided once at the end.  The score matrix
 * is never written to memory.  The backward recomputes each tile's scores
 * (the checkpointing of Section 5.2) from the saved per-row log-sum-exp.
 *
 * Conventions shared by every entry point:
 *   - Layout: q, dq are [B, H, n_q, d]; k, dk are [B, H, n_k, d]; v, dv are
 *     [B, H, n_k, d_v] and o, do [B, H, n_q, d_v] (d_v = d unless
 *     mea_problem.d_v says otherwise); by default contiguous row-major with the feature index
 *     innermost, or with the batch, head and row strides given per tensor in
 *     mea_problem.strides (features always contiguous), which covers the
 *     paper's [n, heads, d] layout and views into a packed QKV projection;
 *     lse is always contiguous [B, H, n_q] float32.
 *   - Pointers: q, k, v, o, o_lo, do, dq, dk, dv, lse and workspace are
 *     DEVICE pointers, 16-byte aligned.  The mea_problem pointer is a HOST pointer.
 *   - Ownership: the caller allocates every buffer, including the workspace.
 *     The library allocates no device memory, keeps no mutable global state
 *     and never synchronises: work is enqueued on `stream` (0 = the null
 *     stream) and completes asynchronously.  Calls are re-entrant.
 *   - Outputs are overwritten, never accumulated into.
 *   - Masking (`causal` = 1): key j is visible to query i iff j <= i,
 *     aligned at the top-left (key 0 is always visible, so no row is empty,
 *     also when n_q != n_k).  The paper defines no mask; this is the reading
 *     the library adopts.
 *   - Key padding (`kv_len` != NULL): batch b sees only its keys
 *     j < kv_len[b] (clamped to [0, n_k]), on top of the causal mask; the
 *     keys from there to n_k are never weighted (their dk and dv rows are
 *     written as zeros).  A query row with no visible key (kv_len[b] <= 0)
 *     gets o = 0, lse = -inf and zero gradients.
 *   - Errors: arguments are validated before anything is launched; on a
 *     validation error nothing is enqueued and the status says why.  A
 *     launch failure reported by the HIP runtime returns MEA_ERR_HIP.  Errors
 *     during kernel execution surface at the caller's next synchronisation.
 *   - Supported: d and d_v in {64, 128}; dtype f32, f16 or bf16 (q, k, v and the
 *     gradients share it; o and do share it too unless out_f32 asks for
 *     float32; lse, the workspace and all accumulation are float32).
 *     Sizes: batch, heads, n_q, n_k >= 1; every element count must fit in
 *     int64 and n_q, n_k <= 2^31 - 1.
 */
#ifndef MEA_H_
#define MEA_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MEA_OK = 0,
  MEA_ERR_INVALID_ARG = 1, /* null/misaligned pointer, size < 1, bad scale */
  MEA_ERR_UNSUPPORTED = 2, /* d or dtype outside the supported set */
  MEA_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required */
  MEA_ERR_HIP = 4,         /* the HIP runtime rejected a launch */
  MEA_ERR_SCRATCH = 5      /* problem needs more than the static scratch of
                              mea_attention_bwd_noalloc holds */
} mea_status;

typedef enum { MEA_F32 = 0, MEA_F16 = 1, MEA_BF16 = 2 } mea_dtype;

/* Element strides of one [B, H, n, d] tensor: element (b, h, i, f) is at
 * b * batch + h * head + i * row + f.  Every stride is a multiple of 16 bytes
 * (8 elements for 16-bit types, 4 for float32) and row is in [d, 2^24); batch
 * and head may be 0 for inputs (one head's keys shared by several query
 * heads), not for outputs.  The library does not check that the rows of an
 * output are disjoint beyond that. */
typedef struct {
  int64_t batch, head, row;
} mea_tensor_strides;

/* Strides of every tensor of a call (the backward's tensors unused by a call
 * are ignored, and the forward reads only q, k, v, o). */
typedef struct {
  mea_tensor_strides q, k, v, o, d_o, dq, dk, dv;
} mea_strides;

/* Problem description (host memory, read during the call only). */
typedef struct {
  int64_t batch;  /* B >= 1 */
  int64_t heads;  /* H >= 1 */
  int64_t n_q;    /* queries per (b, h) >= 1 */
  int64_t n_k;    /* keys = values per (b, h) >= 1 */
  int64_t d;      /* head dimension of q, k and v: 64 or 128 */
  int32_t dtype;   /* mea_dtype of q, k, v, dq, dk, dv (and of o, do unless out_f32) */
  int32_t causal;  /* 0 = no mask, 1 = top-left causal mask (see above) */
  float scale;     /* score scale, finite and > 0; 1/sqrt(d) in the paper */
  int32_t out_f32; /* 0: o and do in `dtype`; 1: o and do in float32 (the
                      paper's experiments use 16-bit inputs with a float32
                      output, Section 5.1); ignored when dtype is MEA_F32 */
  const mea_strides* strides; /* HOST pointer or NULL (every tensor contiguous
                                 [B, H, n, d]); read during the call only */
  const int32_t* kv_len;      /* DEVICE pointer to int32 [B] (4-byte aligned):
                                 valid keys per batch (key padding, see above),
                                 read by the kernels; NULL = all n_k keys */
  int64_t d_v;                /* head dimension of v, o, do and dv: 0 (= d),
                                 64 or 128; q, k, dq and dk have d features */
} mea_problem;

/* Bytes of device workspace mea_attention_fwd needs for `p` (written to
 * *bytes).  Zero unless the keys are split over several workgroups per query
 * tile (long key sequences with few query tiles), in which case it holds the
 * per-split partial numerators (float32 [S, B, H, n_q, d]) and running
 * max / denominator (float32 [S, B, H, n_q] each) that the combine step of
 * Section 4 rescales and adds.  Returns MEA_OK or a validation error. */
mea_status mea_attention_fwd_workspace_size(const mea_problem* p, size_t* bytes);

/* Bytes of device workspace mea_attention_bwd needs for `p`: per padded row
 * (B*H*ceil(n_q/64)*64 rows) the values -lse/scale and -D_i with
 * D_i = sum_t dO_it O_it (Section 5.2's recompute needs only these and the
 * inputs), O(n) like the lse: 16 bytes per row (each value as three bf16
 * parts) where the backward runs its two-group kernels -- 16-bit inputs and
 * outputs at d = d_v = 64, except causal problems of up to 2048 queries and
 * unmasked ones of up to 512 -- else two float32 values.  For
 * 16-bit inputs with float32 o and dO (out_f32) it also holds dO rounded to
 * the input dtype (B*H*n_q*d_v 16-bit values, O(n d) like dO itself), so that
 * the kernels of 16-bit outputs run; the rounding is the one those problems'
 * kernels would otherwise apply while staging dO, so the results are the
 * same, and the per-row values then take the 16-bit-output layout. */
mea_status mea_attention_bwd_workspace_size(const mea_problem* p, size_t* bytes);

/* Forward (Sections 2-4): o = softmax(scale * q k^T) v, computed tile by
 * tile with the running max / numerator / denominator; writes o (in dtype, or
 * float32 with out_f32) and,
 * if lse != NULL, lse_i = max_j s_ij + ln sum_j e^{s_ij - max_j s_ij} in
 * natural-log units (float32), which the backward needs.
 * o_lo (DEVICE pointer or NULL; must be NULL when o is float32): for a 16-bit
 * o, the rounding residual of o in the same dtype, o_lo = round(o_f32 - o)
 * with o_f32 the float32 quotient before rounding, contiguous
 * [B, H, n_q, d_v] whatever o's strides.  o + o_lo carries about 16
 * significant bits, and the backward forms D_i = do_i . (o_i + o_lo_i) from
 * it: D enters dS_ij = w_ij (do_i . v_j - D_i), which is a small difference
 * of two O(1) numbers wherever the softmax saturates (large logits, the
 * numerical-stability setting of Section 3), so o's own 2^-9 rounding would
 * dominate the true dS there.  Caller-owned, O(n d) like o.
 * `workspace` may be NULL only when the required size is 0. */
mea_status mea_attention_fwd(const mea_problem* p, const void* q, const void* k,
                             const void* v, void* o, float* lse, void* o_lo,
                             void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Backward (Section 5.2, recompute instead of storing the n_q x n_k matrix):
 * given the forward's o and lse and the upstream gradient do (both in the
 * output dtype), writes
 *   dv_j = sum_i w_ij do_i,
 *   dk_j = scale sum_i w_ij (do_i . v_j - D_i) q_i,
 *   dq_i = scale sum_j w_ij (do_i . v_j - D_i) k_j,
 * with D_i = do_i . o_i and w_ij = exp(s_ij - lse_i) recomputed per tile.
 * o_lo is the forward's residual of a 16-bit o (see mea_attention_fwd), or
 * NULL: then D_i uses the rounded o alone, which is accurate to the 16-bit
 * tolerance for ordinary inputs but not where the softmax saturates (with
 * logits of order 1e3, gradients can be off by more than 2e-2 of their
 * largest element).  It must be NULL when o is float32.
 * All inputs must come from one mea_attention_fwd call on the same problem.
 * dq may be NULL to skip dQ; dk and dv may be NULL together to skip dK and dV
 * (at least one of the two groups must be requested). */
mea_status mea_attention_bwd(const mea_problem* p, const void* q, const void* k,
                             const void* v, const void* o, const void* o_lo,
                             const void* d_o, const float* lse, void* dq, void* dk,
                             void* dv, void* workspace, size_t workspace_bytes,
                             hipStream_t stream);

/* Bytes of the static device scratch of mea_attention_bwd_noalloc: 16 MiB
 * for the per-row values plus 256 bytes of alignment slack, one copy per GPU
 * the library runs on, held until the process ends. */
#define MEA_NOALLOC_SCRATCH_BYTES (((size_t)16 << 20) + 256)

/* mea_attention_bwd without the workspace arguments, for callers that cannot
 * allocate device memory: code being captured into a HIP graph, tight
 * serving loops, harnesses that forbid allocation.  The per-row values (the
 * workspace of mea_attention_bwd without its 16-bit copy of a float32 dO:
 * those problems run the kernels that round dO while staging it) live in a
 * file-scope device array of MEA_NOALLOC_SCRATCH_BYTES per GPU instead; the
 * call itself
 * allocates nothing (no hipMalloc, no library allocation).  Problems whose
 * workspace exceeds that size return MEA_ERR_SCRATCH before anything is
 * enqueued: B * H * ceil(n_q / 64) * 64 padded query rows must not exceed
 * 2^20 where the backward keeps 16 bytes per row (16-bit inputs and outputs
 * at d = d_v = 64, except causal problems of up to 2048 queries and
 * unmasked ones of up to 512), or 2^21
 * otherwise (8 bytes per row).  The first call on a device
 * looks up that device's copy of the array; `stream` must belong to the
 * current device (0 = its null stream), else MEA_ERR_INVALID_ARG.
 * Every call on one GPU shares its array, and the backward fully writes the
 * part it reads before reading it (nothing needs to start at zero): calls
 * that overlap on one GPU (different streams, or threads) race and must be
 * serialised by the caller.  Results are identical to mea_attention_bwd's
 * (the same arithmetic in the same order). */
mea_status mea_attention_bwd_noalloc(const mea_problem* p, const void* q, const void* k,
                                     const void* v, const void* o, const void* o_lo,
                                     const void* d_o, const float* lse, void* dq, void* dk,
                                     void* dv, hipStream_t stream);

/* Static description of a status code (never NULL). */
const char* mea_status_string(mea_status s);

#ifdef __cplusplus
}
#endif

#endif /* MEA_H_ */
