// Swept-tile machinery shared by the forward and backward sweeps (gfx950).
//
// A sweep keeps 32 rows per wave of one side ("own") in registers and streams
// 32-row tiles of the other side ("swept") through LDS.  The tiles sit in LDS
// segment-blocked: features are cut into segments of 256 bytes (16 chunks of
// 16 bytes); segment c >> 4 of all 32 rows is one contiguous 8 KiB block, rows
// 256 bytes apart, so chunk c of row r lives at
//   kSeg (c >> 4) + kSegRow r + 16 ((c & 15) ^ sweep_g(r)).
// The layout makes the row-fragment reads (first product) and the transposing
// reads (second product of the backward) bank-conflict free, and every DMA
// lane offset a per-wave constant (see sweep_dma_lane_off).
#pragma once

#include "common.hpp"

namespace infcl {

constexpr int kSweepBN = 32;  // swept rows per tile
constexpr int kSegRow = 256;
constexpr int kSeg = kSweepBN * kSegRow;

// Chunk swizzle: 16 rows reading one logical chunk, and the 4 rows x 4 chunks
// of a transposing read, are both spread over all 64 banks.
// The index helpers below are host-callable too: a CPU test enumerates every
// lane, wave and step with them and checks the layout's bounds and coverage.
__host__ __device__ __forceinline__ int sweep_g(int r) { return 4 * (r & 3) + ((r >> 2) & 3); }
// Row permutation of the first product: MFMA row m loads swept row perm(m)
// (bits 2 and 3 swapped), so that accumulator register 8s+t of lane half h
// holds swept row 16s + 8h + t of the tile.
__host__ __device__ __forceinline__ int sweep_perm(int m) { return (m & 0x13) | ((m & 4) << 1) | ((m & 8) >> 1); }

// DMA of a swept tile: instruction k = wave + 4 kk fills LDS bytes
// [1024 k, 1024 k + 1024): segment k >> 3, rows 4 (k & 7) .. +3; lane L fills
// row 4 (k & 7) + (L >> 4), physical chunk L & 15, i.e. logical chunk
// (L & 15) ^ sweep_g(row).  Since sweep_g(row) = 4 (L >> 4) + (k & 3) and
// k & 3 = wave, the per-lane part of every source offset is one constant
// (lane_off) and the rest is wave-uniform (kk_off).  rowg = bytes per row.
__host__ __device__ __forceinline__ uint32_t sweep_dma_lane_off(int lo, int wave, int rowg) {
  return (uint32_t)((lo >> 4) * rowg + 16 * ((lo & 15) ^ (4 * (lo >> 4)) ^ wave));
}
__host__ __device__ __forceinline__ uint32_t sweep_dma_kk_off(int kk, int wave, int rowg) {
  const int k = wave + 4 * kk;
  return (uint32_t)(4 * (k & 7) * rowg + 256 * (k >> 3));
}

// Chunk c (0..15) of row r within its segment: the part of the layout's
// address below the segment base.
__host__ __device__ __forceinline__ int sweep_seg_off(int r, int c) { return r * kSegRow + 16 * (c ^ sweep_g(r)); }
// Chunk c of row r within the tile (any c).
__host__ __device__ __forceinline__ int sweep_chunk_off(int r, int c) {
  return kSeg * (c >> 4) + sweep_seg_off(r, c & 15);
}

// Transposing read of the backward's second product (ds_read_b64_tr_b16):
// offset of the 8 bytes that lane `lane` reads for row group tt (0 or 1) of
// 32-feature block fb, contraction rows 0..15 (add 16 kSegRow for rows
// 16..31).  Lane L reads features 4 (L & 3) .. +3 of the block's 16-feature
// half (L >> 4) & 1 in row 8 (L >> 5) + 4 tt + ((L & 15) >> 2): 4 rows x 4
// features per 16-lane group.  The chunk order inside a row group spreads
// each half-wave's 32 reads over all 64 banks.
__host__ __device__ __forceinline__ int sweep_tr_off(int lane, int tt, int fb) {
  const int g4 = lane >> 4, l16 = lane & 15;
  const int e = l16 >> 2, qq = l16 & 3, nb16 = g4 & 1, hh = g4 >> 1;
  const int lb = 2 * nb16 + (qq >> 1);
  const int fo = (qq & 1) * 8;
  return (8 * hh + 4 * tt + e) * kSegRow + kSeg * (fb >> 2) + 16 * (4 * ((fb & 3) ^ e) + (lb ^ ((tt + 2 * hh) & 3))) +
         fo;
}

// G' block of the backward: 64 bytes per own row (32 swept columns, 16-bit),
// its four 16-byte chunks XOR-swizzled by (row >> 2) & 3.
__host__ __device__ __forceinline__ int gp_chunk_off(int row, int c) { return row * 64 + 16 * (c ^ ((row >> 2) & 3)); }

// 16-bit 32x32x16 MFMA (bf16, or fp16 with F16) accumulating in VGPRs (the
// compiler would place an accumulation chain in AGPRs, which the backward
// needs for its gradients).  Volatile, so that the chain keeps its order with
// interleaved DMA instructions.  Hazards inside inline assembly are not
// checked by the compiler: with PAD, two wait states precede each MFMA (a
// VALU write of a source operand, e.g. an operand the compiler restores with
// v_accvgpr_read, must be two wait states old), and the last MFMA of a chain
// is followed by the wait states a VALU read of its result needs, inside the
// same statement so that nothing reads the accumulator earlier.
#define INFCL_MFMA16_VGPR(PRE, OP)                                                                              \
  if (first && last)                                                                                           \
    asm volatile(PRE OP " %0, %1, %2, 0\n\ts_nop 7\n\ts_nop 7\n\ts_nop 3" : "=&v"(acc) : "v"(a), "v"(b));   \
  else if (first)                                                                                              \
    asm volatile(PRE OP " %0, %1, %2, 0" : "=&v"(acc) : "v"(a), "v"(b));                                        \
  else if (last)                                                                                               \
    asm volatile(PRE OP " %0, %1, %2, %0\n\ts_nop 7\n\ts_nop 7\n\ts_nop 3" : "+v"(acc) : "v"(a), "v"(b));  \
  else                                                                                                         \
    asm volatile(PRE OP " %0, %1, %2, %0" : "+v"(acc) : "v"(a), "v"(b));

// PAD = false drops the two leading wait states, for call sites whose source
// operands are never written by a VALU instruction just before (LDS loads and
// registers set up before the sweep); the build's wait-state scan checks
// every site of either form.
template <bool F16, bool PAD = true>
__device__ __forceinline__ void mfma16_vgpr(f32x16& acc, const bf16x8& a, const bf16x8& b, bool first, bool last) {
  if constexpr (F16) {
    if constexpr (PAD) {
      INFCL_MFMA16_VGPR("s_nop 1\n\t", "v_mfma_f32_32x32x16_f16")
    } else {
      INFCL_MFMA16_VGPR("", "v_mfma_f32_32x32x16_f16")
    }
  } else {
    if constexpr (PAD) {
      INFCL_MFMA16_VGPR("s_nop 1\n\t", "v_mfma_f32_32x32x16_bf16")
    } else {
      INFCL_MFMA16_VGPR("", "v_mfma_f32_32x32x16_bf16")
    }
  }
}
#undef INFCL_MFMA16_VGPR

}  // namespace infcl
