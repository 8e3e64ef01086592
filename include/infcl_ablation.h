/*
 * infcl_ablation.h -- the single-launch backward of the appendix's in-GPU
 * backward algorithm, for the ablation against infcl_bwd (not part of the
 * loss's API).
 *
 * The appendix's backward computes each similarity tile and its softmax
 * weights once, keeps the image gradient of a row block on chip, and updates
 * the text-gradient tile in memory for every tile: with row blocks in parallel
 * that is an atomic add per element and tile.  infcl_ablation_bwd_single does
 * exactly that in one sweep (64 image rows per workgroup, start tiles
 * staggered over the workgroups, hardware fp32 atomics into dtxt), where
 * infcl_bwd instead runs the sweep twice (image rows owned, then text rows
 * owned), recomputing the similarity tile and writing each gradient once.
 *
 * Arguments, layouts and outputs are those of infcl_bwd (include/infcl.h):
 * img, txt [b, d] bf16; scale; lse_r, lse_c, aux from infcl_fwd; dloss (NULL
 * means 1); outputs dimg, dtxt [b, d] float and dscale.  dtxt is zeroed by the
 * call before the sweep.  workspace: device, 256-byte aligned, at least
 * infcl_workspace_size(b, d, INFCL_BF16) bytes.  Work is enqueued on stream;
 * nothing is allocated.  The atomic additions make dtxt (and only dtxt)
 * differ from run to run in the last bits.
 * Returns 0; 1 for an invalid argument (NULL or misaligned pointer, b < 1,
 * d < 1); 2 for an unsupported shape (dtype other than bf16, d other than 256
 * or 512, b > 2^30); 3 for a workspace too small; 4 for a launch failure.
 */
#ifndef INFCL_ABLATION_H
#define INFCL_ABLATION_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

int infcl_ablation_bwd_single(const void* img, const void* txt, int64_t b, int64_t d, int dtype,
                              const float* scale, const float* lse_r, const float* lse_c, const float* aux,
                              const float* dloss, float* dimg, float* dtxt, float* dscale, void* workspace,
                              size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* INFCL_ABLATION_H */
