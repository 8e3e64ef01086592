/*
 * infcl_ablation.h -- measurement entry point of the single-launch backward
 * ablation (not part of the loss).
 *
 * The appendix's in-GPU backward algorithm updates the text gradient in HBM
 * for every tile: read dT^j, add the row block's contribution, write it back.
 * With row blocks in parallel that is an atomic add per element and tile.
 * infcl_ablation_dt_atomics issues that traffic alone: ceil(b / bm)
 * workgroups (one per row block of bm rows) each add a 32 x d block of 1.0
 * into every 32-row tile of dT with hardware fp32 atomics, in sweep order.
 * Its time bounds the single-launch backward from below; the two-launch
 * backward of infcl_bwd recomputes each similarity tile instead.
 *
 *   dT      device pointer, [b, d] float, 16-byte aligned; every element is
 *           increased by ceil(b / bm) (exact in fp32 for any b up to 2^30
 *           with bm >= 64)
 *   stream  hipStream_t (NULL = default); asynchronous, allocates nothing
 * Returns 0, 1 for an invalid argument (NULL or misaligned dT, b < 1,
 * d < 1, bm < 1, b > 2^30, d > 65536), 4 for a launch failure.
 */
#ifndef INFCL_ABLATION_H
#define INFCL_ABLATION_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

int infcl_ablation_dt_atomics(float* dT, int64_t b, int64_t d, int64_t bm, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* INFCL_ABLATION_H */
