// Shared device helpers for the tiled contrastive-loss kernels (gfx950 only).
//
// Conventions used by both sweeps
//   - Matrix products run on the 32x32x16 bf16 or fp16 MFMA (fp32 accumulate)
//     or the 32x32x2 fp32 MFMA.  Fragments of both 16-bit types are carried
//     in bf16x8 registers; only the MFMA opcode and the conversions differ.  For a 32x32 output block, lane L holds column
//     n = L % 32 and rows m = 8*(r/4) + 4*(L/32) + r%4 for accumulator r = 0..15.
//     Operand fragments: lane L holds row L % 32 and the 8 consecutive
//     contraction slots 8*(L/32) .. 8*(L/32)+7 of a 16-wide contraction step.
//   - Log-sum-exp statistics are kept in base 2: y = s*log2(e)*<a, b>, a
//     running pair (R, l) stands for log2(l) + R, and exp2 maps to v_exp_f32.
//   - Tiles are staged in LDS in 16-byte chunks with an XOR swizzle of the chunk
//     index so that both the row-fragment reads and the transposing reads of
//     the backward pass are bank-conflict free.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace infcl {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

#define INFCL_LDS __attribute__((address_space(3)))
#define INFCL_GLOBAL __attribute__((address_space(1)))

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// A per-tile partial sum above this bound, or a non-finite one, sends a tile
// through the exact (max-rescaled) path.  With at most 2^22 terms per sum the
// accumulated value stays below 2^86, far from float overflow.
constexpr float kLazyBound = 18446744073709551616.0f;  // 2^64

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ f32x16 mfma_bf16(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// 16-bit MFMA on fragments held as bf16x8: bf16 operands, or fp16 (F16).
template <bool F16>
__device__ __forceinline__ f32x16 mfma16(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  if constexpr (F16)
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                  0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// float -> 16-bit element, round to nearest even (bf16, or the bits of fp16)
template <bool F16>
__device__ __forceinline__ __bf16 to16(float x) {
  if constexpr (F16)
    return __builtin_bit_cast(__bf16, (_Float16)x);
  else
    return (__bf16)x;
}
// 16-bit element (bf16, or fp16 bits) -> float, exact
template <bool F16>
__device__ __forceinline__ float from16(__bf16 x) {
  if constexpr (F16)
    return (float)__builtin_bit_cast(_Float16, x);
  else
    return (float)x;
}
__device__ __forceinline__ f32x16 mfma_f32(float a, float b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// Asynchronous 16-byte global -> LDS copy.  Lane L writes LDS bytes
// [lds_base + 16 L, lds_base + 16 L + 16); lds_base must be wave-uniform.
__device__ __forceinline__ void dma16(const void* gsrc, INFCL_LDS void* lds_base) {
  __builtin_amdgcn_global_load_lds((const INFCL_GLOBAL void*)gsrc, lds_base, 16, 0, 0);
}
__device__ __forceinline__ void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// Wait until at most n (0..63) vector-memory operations of this wave are in
// flight.  Operations complete in issue order, so this waits for all but the n
// most recently issued ones.
__device__ __forceinline__ void wait_dma_allow(int n) {
  switch (n) {
#define INFCL_VM_CASE(k) \
  case k: asm volatile("s_waitcnt vmcnt(" #k ")" ::: "memory"); break;
    INFCL_VM_CASE(0) INFCL_VM_CASE(1) INFCL_VM_CASE(2) INFCL_VM_CASE(3) INFCL_VM_CASE(4) INFCL_VM_CASE(5)
    INFCL_VM_CASE(6) INFCL_VM_CASE(7) INFCL_VM_CASE(8) INFCL_VM_CASE(9) INFCL_VM_CASE(10) INFCL_VM_CASE(11)
    INFCL_VM_CASE(12) INFCL_VM_CASE(13) INFCL_VM_CASE(14) INFCL_VM_CASE(15) INFCL_VM_CASE(16) INFCL_VM_CASE(17)
    INFCL_VM_CASE(18) INFCL_VM_CASE(19) INFCL_VM_CASE(20) INFCL_VM_CASE(21) INFCL_VM_CASE(22) INFCL_VM_CASE(23)
    INFCL_VM_CASE(24) INFCL_VM_CASE(25) INFCL_VM_CASE(26) INFCL_VM_CASE(27) INFCL_VM_CASE(28) INFCL_VM_CASE(29)
    INFCL_VM_CASE(30) INFCL_VM_CASE(31) INFCL_VM_CASE(32) INFCL_VM_CASE(33) INFCL_VM_CASE(34) INFCL_VM_CASE(35)
    INFCL_VM_CASE(36) INFCL_VM_CASE(37) INFCL_VM_CASE(38) INFCL_VM_CASE(39) INFCL_VM_CASE(40) INFCL_VM_CASE(41)
    INFCL_VM_CASE(42) INFCL_VM_CASE(43) INFCL_VM_CASE(44) INFCL_VM_CASE(45) INFCL_VM_CASE(46) INFCL_VM_CASE(47)
#undef INFCL_VM_CASE
    default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
  }
}

// Raw buffer resource over [base, base + nbytes): loads past the end return 0.
// Rebased per tile so that 32-bit per-lane offsets address inputs of any size.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t nbytes) {
  const int64_t n = nbytes < 0 ? 0 : (nbytes > 0xFFFFFFF0ll ? 0xFFFFFFF0ll : nbytes);
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, (int)(uint32_t)n, 0x00020000);
}
// 16-byte buffer -> LDS copy; lane L writes LDS bytes [lds_base + 16 L, +16).
__device__ __forceinline__ void dma16b(__amdgpu_buffer_rsrc_t rs, INFCL_LDS void* lds_base, uint32_t voff,
                                       uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, lds_base, 16, voff, soff, 0, 0);
}

// The same copy issued from inline assembly, with a raw descriptor (see
// rsrc_words).  The compiler does not see this as a write to LDS, so it never
// stalls later LDS reads on it: the caller waits for completion explicitly
// (wait_dma / wait_dma_allow) before the written buffer is read.  m0 holds
// the wave-uniform LDS base.  The compiler's hazard checks do not look inside
// inline assembly, and it may restore an operand right before it (an SGPR of
// the descriptor with v_readlane, the offset with v_accvgpr_read): the five
// wait states cover a VALU-written SGPR read by a vector memory instruction,
// which is the longest of those requirements (and the one of m0).
__device__ __forceinline__ u32x4 rsrc_words(const void* base, int64_t nbytes) {
  const int64_t n = nbytes < 0 ? 0 : (nbytes > 0xFFFFFFF0ll ? 0xFFFFFFF0ll : nbytes);
  const uint64_t a = (uint64_t)base;
  u32x4 r;
  r[0] = (uint32_t)a;
  r[1] = (uint32_t)(a >> 32) & 0xFFFFu;  // stride 0
  r[2] = (uint32_t)n;                    // num_records (bytes)
  r[3] = 0x00020000u;
  return r;
}
__device__ __forceinline__ void dma16_asm(const u32x4& rs, const INFCL_LDS void* lds_base, uint32_t voff) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds_base);
  asm volatile("s_nop 4\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voff), "s"(rs), "{m0}"(m0v));
}
// ... with a wave-uniform byte offset soff added to every lane's offset.
__device__ __forceinline__ void dma16_asm(const u32x4& rs, const INFCL_LDS void* lds_base, uint32_t voff,
                                          uint32_t soff) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds_base);
  const uint32_t so = __builtin_amdgcn_readfirstlane(soff);
  asm volatile("s_nop 4\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds" ::"v"(voff), "s"(rs), "s"(so), "{m0}"(m0v));
}

// The same with one wait state only (m0 written by a scalar instruction just
// before), for bursts whose other operands are set up well ahead; the build's
// wait-state check verifies every use.
__device__ __forceinline__ void dma16_asm_w1(const u32x4& rs, const INFCL_LDS void* lds_base, uint32_t voff) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds_base);
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voff), "s"(rs), "{m0}"(m0v));
}
__device__ __forceinline__ void dma16_asm_w1(const u32x4& rs, const INFCL_LDS void* lds_base, uint32_t voff,
                                             uint32_t soff) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds_base);
  const uint32_t so = __builtin_amdgcn_readfirstlane(soff);
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds" ::"v"(voff), "s"(rs), "s"(so), "{m0}"(m0v));
}

// Merge of two base-2 log-sum-exp pairs (R, l) -> (max R, rescaled sum).
__device__ __forceinline__ void lse2_merge(float& R, float& l, float R2, float l2) {
  float M = fmaxf(R, R2);
  if (M == -__builtin_inff()) return;  // both empty
  l = l * exp2_hw(R - M) + l2 * exp2_hw(R2 - M);
  R = M;
}

__device__ __forceinline__ bool lazy_ok(float t) { return t <= kLazyBound; }  // false for NaN/inf

// Cross-lane helpers (full 64-lane wave).
__device__ __forceinline__ float shfl_xor(float v, int mask) {
  int l = __lane_id();
  return __int_as_float(__builtin_amdgcn_ds_bpermute((l ^ mask) << 2, __float_as_int(v)));
}
__device__ __forceinline__ float shfl_idx(float v, int src) {
  return __int_as_float(__builtin_amdgcn_ds_bpermute(src << 2, __float_as_int(v)));
}
__device__ __forceinline__ bool wave_any(bool p) { return __builtin_amdgcn_ballot_w64(p) != 0; }

}  // namespace infcl
