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
 *   - Supported shapes: 1 <= b <= 2^30; d a multiple of 128 with d <= 1024
 *     for bf16 and f16, a multiple of 64 with d <= 512 for f32
 *     (INFCL_ERR_UNSUPPORTED otherwise).
 *   - Results are bitwise reproducible for a given (b, d, dtype): no atomics,
 *     all reductions run in a fixed order.
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
 * The same workspace size serves both calls.  Returns INFCL_ERR_INVALID for a
 * NULL `bytes` or b < 1, d < 1 or an unknown dtype. */
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
 *   dimg  [b, d] float   dloss * dL/dimg
 *   dtxt  [b, d] float   dloss * dL/dtxt
 *   dscale [1] float     dloss * dL/ds (derivative w.r.t. s itself)
 * dloss is a device pointer to one float (NULL means 1).  lse_r, lse_c and aux
 * must come from infcl_fwd on the same inputs.  Two sweeps run: one owns rows
 * of img and accumulates dimg in registers, the other owns rows of txt; the
 * softmax is never written to memory. */
infcl_status infcl_bwd(const void* img, const void* txt, int64_t b, int64_t d, int dtype,
                       const float* scale, const float* lse_r, const float* lse_c, const float* aux,
                       const float* dloss, float* dimg, float* dtxt, float* dscale,
                       void* workspace, size_t ws_bytes, void* stream);

/* Static, NUL-terminated description of a status code. */
const char* infcl_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* INFCL_H */
