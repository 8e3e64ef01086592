// Shared declarations of the backward sweeps (gfx950).
#pragma once

#include "sweep.hpp"

namespace infcl {

struct BwdParams {
  const void* own;    // [b, d] rows whose gradient this launch produces
  const void* swept;  // [b, d] the other modality
  int64_t b, d;
  const float* scale;
  const float* lse_own;     // [b]  natural-log log-sum-exp of the own side
  const float* lse2_swept;  // [b]  log-sum-exp of the swept side times log2(e)
  const float* ell_own;     // [b]  r_i - x_ii of the own side
  const float* ell_swept;   // [b]
  const float* udiag;       // [b]  <img_i, txt_i>
  const float* dloss;       // device scalar or nullptr (= 1)
  int64_t own_off, own_end;  // own rows [own_off, own_end) (a shard; 0 and b for the whole batch)
  void* dOwn;               // [own_end - own_off, d], by own row - own_off: fp32, or with gdt = 1 the
                            // input's 16-bit type
  double* ds_part;          // [gridDim.x]
  const float* g16;         // fp16 inputs: (alpha, 1/alpha), the power of two G' is scaled by
  int gdt;                  // gradient type, which chooses the kernel instantiation: 0 fp32, 1 16-bit
};

constexpr int kBwdBN = kSweepBN;  // swept rows per tile

// Gradient element type of a sweep: fp32, or with G16 the 16-bit input type
// (fp16 with F16, else bf16), rounded to nearest even from the fp32 gradient
// when stored.  The fp32 value is materialised first: the compiler would
// otherwise fuse the final scaling into an fp16 conversion (a mixed-precision
// multiply that rounds the exact product once), whose result differs from a
// cast of the fp32 gradient by one unit where that lands on a tie.
template <bool G16, bool F16>
struct GradOut {
  using type = float;
  static __device__ __forceinline__ float cvt(float v) { return v; }
};
template <bool F16>
struct GradOut<true, F16> {
  using type = __bf16;
  static __device__ __forceinline__ __bf16 cvt(float v) {
    asm volatile("" : "+v"(v));
    return to16<F16>(v);
  }
};

}  // namespace infcl
