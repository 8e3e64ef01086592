/*
 * infcl.h -- C ABI of the tiled symmetric InfoNCE (CLIP) loss on AMD Instinct
 * MI355X (gfx950).
 *
 * The loss follows "Breaking the Memory Barrier: Near Infinite Batch Size
 * Scaling for Contrastive Loss" (Inf-CL):
 *   - Sec. 2.2, Eq. 1: image->text InfoNCE over x_ij = s * <I_i, T_j>; the
 *     text->image half is its symmetric twin and the loss is their mean:
 *        L = (1/2b) * ( sum_i (r_i - x_ii) + sum_j (c_j - x_jj) ),
 *        r_i = log sum_j e^{x_ij},  c_j = log sum_i e^{x_ij};
 *   - Sec. 3.1, Eq. 2-5: the b x b similarity matrix is never stored; it is
 *     streamed tile by tile and only the log-sum-exp vectors are kept;
 *   - Sec. 3.1, Eq. 6-8 and the appendix's backward algorithms: the backward
 *     pass recomputes each tile from the saved log-sum-exp values and
 *     accumulates dI, dT (and, here, ds) without storing the softmax.
 *
 * Conventions shared by every entry point
 *   - img, txt: device pointers, row-major [b, d], contiguous, 16-byte
 *     aligned; element type given by `dtype` (INFCL_BF16, INFCL_F32 or
 *     INFCL_F16).  With 16-bit inputs the products run on the matching
 *     16-bit MFMA with fp32 accumulation, and the backward rounds its
 *     gradient weights (the softmax terms) to the input type, round to
 *     nearest even, before the second product; with f32 everything is fp32.
 *     They are used exactly as given (no normalisation inside the loss).
 *   - scale: device pointer to one float, the logit scale s (1/temperature).
 *   - All float vectors are device pointers, 16-byte aligned.
 *   - stream: a hipStream_t (NULL = the default stream).  Work is enqueued
 *     asynchronously; the call never synchronises the host and never
 *     allocates: the caller owns every buffer, including the workspace, and
 *     must keep them alive until the stream reaches this work.
 *   - Errors: arguments are validated on the host before anything is
 *     enqueued; an invalid call returns a status and launches nothing.  A
 *     launch failure is reported as INFCL_ERR_HIP.  Non-finite input values
 *     are outside the contract (they propagate).
 *   - Supported shapes: 1 <= b <= 2^30; d a multiple of 8 with d <= 1024
 *     for bf16 and f16, a multiple of 4 with d <= 512 for f32 (rows of
 *     whole 16-byte units; INFCL_ERR_UNSUPPORTED otherwise).  The kernels
 *     are built for multiples of 128 (16-bit) and 64 (f32); at any other
 *     width the calls copy img and txt into the workspace with zero features
 *     appended up to the next such multiple and write the gradients through
 *     padded buffers there.  Zero features change no dot product: every
 *     output is exactly that of the unpadded inputs.
 *   - Results are bitwise reproducible for a given (b, d, dtype): no atomics,
 *     all reductions run in a fixed order.
 *   - The calls may be captured into a HIP graph: they enqueue kernels only
 *     (no allocation, no memset or copy nodes, no host synchronisation), and
 *     replays give the bits of the eager calls.
 */
#ifndef INFCL_H
#define INFCL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  INFCL_OK = 0,
  INFCL_ERR_INVALID = 1,     /* NULL/misaligned pointer, b < 1, d < 1, bad dtype */
  INFCL_ERR_UNSUPPORTED = 2, /* valid but not implemented shape (see above)      */
  INFCL_ERR_WORKSPACE = 3,   /* workspace smaller than infcl_workspace_size()    */
  INFCL_ERR_HIP = 4          /* a kernel launch failed                           */
} infcl_status;

/* Input element types.  INFCL_F16 (IEEE half) is the type of mixed-precision
 * (AMP) training, under which the paper trains (Sec. 4.1). */
typedef enum { INFCL_BF16 = 0, INFCL_F32 = 1, INFCL_F16 = 2 } infcl_dtype;

/* Bytes of device workspace that infcl_fwd / infcl_bwd need for (b, d, dtype).
 * The same workspace size serves both calls.  It is linear in b: a few
 * vectors of b floats, plus, when d is not a multiple of 128 (16-bit) or 64
 * (f32), the padded copies of img and txt and the padded gradients
 * (2 b d' fp32 elements, d' the padded width).  Returns INFCL_ERR_INVALID for
 * a NULL `bytes` or b < 1, d < 1 or an unknown dtype. */
infcl_status infcl_workspace_size(int64_t b, int64_t d, int dtype, size_t* bytes);

/* Forward pass (Eq. 1-2 with the tiling of Eq. 3-5 / the in-GPU forward
 * algorithm): streams tiles of S = s * img * txt^T and keeps online row and
 * column log-sum-exp statistics; S is never written to memory.
 * Outputs (device):
 *   loss    [1] float   L
 *   loss64  [1] double  L in fp64 (may be NULL); L can be far below the float
 *                       range's normal numbers when s is large (e.g. 1e-43)
 *   lse_r   [b] float   r_i = log sum_j e^{x_ij}
 *   lse_c   [b] float   c_j = log sum_i e^{x_ij}
 *   aux     [3b] float  aux[0:b]   = r_i - x_ii   (per-sample row term, >= 0)
 *                       aux[b:2b]  = c_j - x_jj   (per-sample column term)
 *                       aux[2b:3b] = <img_i, txt_i> (unscaled diagonal)
 * lse_r, lse_c and aux are what infcl_bwd needs from the forward pass. */
infcl_status infcl_fwd(const void* img, const void* txt, int64_t b, int64_t d, int dtype,
                       const float* scale, float* loss, double* loss64, float* lse_r, float* lse_c,
                       float* aux, void* workspace, size_t ws_bytes, void* stream);

/* Backward pass (Eq. 6-8 completed for both halves, the text side and the
 * scale; the appendix's in-GPU backward algorithm with recomputed tiles):
 *   dimg  [b, d] grad_dtype  dloss * dL/dimg
 *   dtxt  [b, d] grad_dtype  dloss * dL/dtxt
 *   dscale [1] float         dloss * dL/ds (derivative w.r.t. s itself)
 * grad_dtype: INFCL_F32, or for 16-bit inputs also their own type (bf16
 * gradients of bf16 inputs, f16 of f16): the gradients accumulate in fp32 and
 * are rounded once, to nearest even, when stored.  Another known type returns
 * INFCL_ERR_UNSUPPORTED, an unknown one INFCL_ERR_INVALID.  dloss is a device
 * pointer to one float (NULL means 1).  lse_r, lse_c and aux must come from
 * infcl_fwd on the same inputs.  Two sweeps run: one owns rows of img and
 * accumulates dimg in registers, the other owns rows of txt; the softmax is
 * never written to memory. */
infcl_status infcl_bwd(const void* img, const void* txt, int64_t b, int64_t d, int dtype,
                       const float* scale, const float* lse_r, const float* lse_c, const float* aux,
                       const float* dloss, void* dimg, void* dtxt, int grad_dtype, float* dscale,
                       void* workspace, size_t ws_bytes, void* stream);

/* ---- One GPU's share of a batch sharded over n GPUs (Sec. 3.2, cross-GPU
 * tiling, Alg. 1 and Alg. 3).  GPU g owns samples [r0, r0 + bs): its rows of
 * S (image side) and its columns (text side).  Instead of the paper's ring,
 * which moves text blocks between GPUs step by step, every GPU holds all of
 * img and txt (an all-gather of 2 b d elements per GPU), computes its rows
 * against all b columns, and one exchange of column pairs completes the
 * column statistics:
 *   1. infcl_fwd_shard on every GPU: row statistics of own rows (kept in the
 *      workspace) and one pair per column over own rows, for all b columns;
 *   2. all-to-all: GPU g receives, from each of the n GPUs, the pairs of its
 *      own columns [r0, r0 + bs);
 *   3. infcl_fwd_shard_finish on every GPU: own lse_r, lse_c, aux and its
 *      share of the loss (loss = sum of the shares: an all-reduce);
 *   4. all-gather of lse_r, lse_c and aux (4 b bytes each);
 *   5. infcl_bwd_shard on every GPU: dimg and dtxt of own samples, and its
 *      share of dscale (dscale = sum of the shares).
 * The kernels are those of infcl_fwd / infcl_bwd on a rectangle of bs own
 * rows by b columns.  r0 must be a multiple of 32 and 1 <= bs <= b - r0
 * (INFCL_ERR_INVALID otherwise).  The workspace is that of
 * infcl_workspace_size(b, d, dtype); infcl_fwd_shard_finish must get the same
 * workspace as the infcl_fwd_shard call of its shard, untouched in between.
 * With one shard (r0 = 0, bs = b) the three calls compute what infcl_fwd
 * and infcl_bwd compute. */

/* Step 1.  colpair [2b] float (device, 16-byte aligned): colpair[j] = R_j and
 * colpair[b + j] = l_j, the base-2 log-sum-exp pair (log2 l_j + R_j) of
 * column j over own rows i != j.  The forward's ordinary outputs are not
 * produced here. */
infcl_status infcl_fwd_shard(const void* img, const void* txt, int64_t b, int64_t d, int dtype,
                             int64_t r0, int64_t bs, const float* scale, float* colpair,
                             void* workspace, size_t ws_bytes, void* stream);

/* Step 3.  colpairs [nparts][2 bs] float (device): for each of the nparts
 * shards, the R values then the l values of this shard's columns
 * [r0, r0 + bs) from that shard's colpair.  Outputs for own samples
 * (device): lse_r [bs], lse_c [bs], aux [3 bs] (laid out as infcl_fwd's aux
 * with bs in place of b) and loss_part [1] double, this shard's share
 * (sum over own samples of (r_i - x_ii) + (c_i - x_ii)) / (2b). */
infcl_status infcl_fwd_shard_finish(int64_t b, int64_t d, int dtype, int64_t r0, int64_t bs,
                                    int64_t nparts, const float* colpairs, const float* scale,
                                    float* lse_r, float* lse_c, float* aux, double* loss_part,
                                    void* workspace, size_t ws_bytes, void* stream);

/* Step 5.  lse_r, lse_c [b] and aux [3b] cover all b samples (the all-gather
 * of every shard's finish outputs, in sample order).  Outputs (device):
 * dimg, dtxt [bs, d] of grad_dtype (as in infcl_bwd), the gradients of own
 * samples, and dscale_part [1] double, this shard's share of dloss * dL/ds. */
infcl_status infcl_bwd_shard(const void* img, const void* txt, int64_t b, int64_t d, int dtype,
                             int64_t r0, int64_t bs, const float* scale, const float* lse_r,
                             const float* lse_c, const float* aux, const float* dloss,
                             void* dimg, void* dtxt, int grad_dtype, double* dscale_part,
                             void* workspace, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): infcl_fwd
 * without the workspace arguments.  The workspace is a fixed 32 MiB array in
 * the library's device code, one per device, held until the process ends; its
 * address is looked up (hipGetSymbolAddress) on the first call on each device.
 * No allocation of any kind happens.  The outputs and their meaning are those
 * of infcl_fwd, bit for bit.  Returns INFCL_ERR_WORKSPACE when
 * infcl_workspace_size(b, d, dtype) exceeds 32 MiB (about b = 99,000 for
 * 16-bit inputs, b = 43,000 for f32), INFCL_ERR_HIP if the scratch address
 * cannot be obtained.  Every call on one device shares that device's scratch:
 * calls that overlap in time on one device (two streams, two host threads)
 * race and give wrong results; calls in one stream order are safe. */
infcl_status infcl_fwd_noalloc(const void* img, const void* txt, int64_t b, int64_t d, int dtype,
                               const float* scale, float* loss, double* loss64, float* lse_r, float* lse_c,
                               float* aux, void* stream);

/* Static, NUL-terminated description of a status code. */
const char* infcl_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* INFCL_H */
