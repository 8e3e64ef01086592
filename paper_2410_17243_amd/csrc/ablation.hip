// Ablation of the single-launch backward (gfx950): the text-gradient update
// traffic of the appendix's in-GPU backward algorithm, measured on its own.
//
// That algorithm keeps dI of a row block on chip and, for every column tile
// j, reads dT^j from HBM, adds the row block's contribution and writes it
// back.  With the row blocks running in parallel (one workgroup each, as on
// any GPU), the update has to be an atomic add.  This kernel issues exactly
// that traffic, with no arithmetic around it: workgroup w (row block w, bm
// rows) sweeps the column tiles in order and adds a 32 x d block of ones into
// dT^j with hardware fp32 atomics.  Its time is a lower bound on the
// single-launch backward, to set against the two-launch design, which
// recomputes the similarity tile once more instead of moving any gradient
// through memory during the sweep.
//
// Every element of dT receives ceil(b / bm) additions of 1.0, an exact
// integer in fp32, so the result is checkable bit for bit.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "infcl_ablation.h"

namespace infcl {

constexpr int kAblBN = 32;  // column tile rows, as in the sweeps

__global__ void __launch_bounds__(256) abl_dt_atomic(float* dT, int64_t b, int64_t d) {
  const int64_t ntile = (b + kAblBN - 1) / kAblBN;
  const int64_t blk = (int64_t)kAblBN * d;
  for (int64_t jt = 0; jt < ntile; ++jt) {
    const int64_t j0 = jt * kAblBN;
    const int64_t lim = (b - j0 < kAblBN ? b - j0 : kAblBN) * d;
    float* base = dT + j0 * d;
    for (int64_t e = threadIdx.x; e < blk; e += 256)
      if (e < lim) unsafeAtomicAdd(base + e, 1.0f);
  }
}

}  // namespace infcl

extern "C" int infcl_ablation_dt_atomics(float* dT, int64_t b, int64_t d, int64_t bm, void* stream) {
  if (dT == nullptr || ((uintptr_t)dT % 16) != 0 || b < 1 || d < 1 || bm < 1 || b > ((int64_t)1 << 30) ||
      d > 65536)
    return 1;
  const int64_t nwg = (b + bm - 1) / bm;
  if (nwg > ((int64_t)1 << 31) - 1) return 1;
  hipLaunchKernelGGL(infcl::abl_dt_atomic, dim3((unsigned)nwg), dim3(256), 0, (hipStream_t)stream, dT, b, d);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}
