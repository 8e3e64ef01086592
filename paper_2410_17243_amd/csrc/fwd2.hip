// Forward sweep of the tiled symmetric InfoNCE loss with resident own rows
// (16-bit inputs: bf16 or fp16, d a multiple of 128 up to 1024, gfx950).
//
// What is computed (Sec. 3.1, Eq. 2-5; the in-GPU forward of Sec. 3.2,
// Alg. 2): the off-diagonal log-sum-exp of every row i and every column j of
// S = s * img * txt^T, without storing S.
//
// Work decomposition.  Workgroup (q, g) of a P_r x P_c grid owns row blocks
// q, q + P_r, ... of 32 NW image rows (32 rows per wave, held in registers as
// the MFMA operand for the whole block, as Alg. 2 keeps its row tile on chip)
// and sweeps the text tiles of column group g (32 rows each, streamed through
// LDS by DMA in the swept-tile layout).  Each tile is one 32 x 32 block of S^T
// per wave.  Only text tiles move: 32 KiB of DMA per tile and workgroup for
// 8.4 MFLOP at d = 512 with 8 waves.  g = blockIdx mod P_c, so with P_c = 8 the
// workgroups of a column group share one XCD and its L2.
//  - d <= 512: NW = 8 waves, one workgroup per CU (d/4 VGPRs of own rows).
//  - d > 512: the own rows take d/4 registers of the wave's 512, so NW = 4
//    (one wave per SIMD) and the own-row operand lives in AGPRs, which the
//    MFMA reads directly; this leaves the VGPRs to the tile ring and the
//    statistics.
//
// Statistics.  Log-sum-exp values are kept in base 2 as running pairs (R, l)
// meaning log2(l) + R; the empty sum is l = 0 with any finite R.  New values y
// are added lazily as exp2(y - R) against a reference R that starts at the
// diagonal value y_ii = s log2(e) <img_i, txt_i> of the row or column
// (computed before the sweep; the diagonal itself is excluded from the sums).
// A tile's addition is accepted while the partial sum stays at most 2^64 and
// the running sum at least 2^-64 (so that no entry that matters underflows);
// otherwise the tile is redone exactly: the old pair is normalised to
// (R + log2 l, 1) and merged with the tile's max-rescaled sum.
//  - Rows: every lane accumulates its own row over the 16 entries it holds;
//    the two lane halves merge at the end of the row block into the group's
//    slot rowR/rowL[g].
//  - Columns: every column of a tile gets one partial pair per wave (a sum
//    over its 32 rows, reduced across lanes) against the running pair
//    colR/colL[q][j] of the workgroup; a wave whose partial fails the bounds
//    takes its own column maxima as references instead.  The four wave pairs
//    meet in LDS, and lanes 0..7 of each wave merge them into the running
//    pairs of 8 columns during the next tile's GEMM1.
//  The running column pairs of a tile come into LDS with the tile's DMA, so
//  the sweep makes no other loads, and (as in the backward sweep) the DMA is
//  issued from inline assembly, so the compiler never waits for it before
//  unrelated LDS reads.
#include <utility>

#include "sweep.hpp"


namespace infcl {

// f(std::integral_constant<int, 0>), ..., f(std::integral_constant<int, N-1>):
// a loop unrolled by construction, with a compile-time index in each body.
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

struct Fwd2Params {
  const __bf16* img;  // own rows i, [b, d] (bf16, or fp16 bits)
  const __bf16* txt;  // swept rows j, [b, d]
  int64_t b;
  const float* scale;
  const float* ref2;  // [b]  s log2(e) <img_i, txt_i>
  float* rowR;        // [Pc][rstride]  indexed by own row - r0
  float* rowL;
  int r0, rend;     // own rows [r0, rend) (a shard of the batch; 0 and b for the whole batch)
  int64_t rstride;  // rend - r0
  float* colR;  // [Pr][b]
  float* colL;
  int Pr, Pc;
  int nRB;  // row blocks of 32 NW own rows
  int nCT;  // column tiles of 32
};

// waves per workgroup: 8 (one workgroup per CU, a text tile loaded once per
// CU) or 4 (two workgroups per CU)
#ifndef INFCL_FWD2_WAVES
#define INFCL_FWD2_WAVES 8
#endif
constexpr int kF2NW = INFCL_FWD2_WAVES;
// Waves per workgroup at width d: above 512 the own rows' operand (d/4
// registers) leaves room for one wave per SIMD only, so 4 waves (128 own
// rows) and one workgroup per CU.
__host__ __device__ constexpr int fwd2_waves(int64_t d) { return d > 512 ? 4 : kF2NW; }
constexpr float kTinyBound = 5.421010862427522e-20f;  // 2^-64
// mfma16_vgpr with the B operand (the own rows) held in AGPRs, for d > 512;
// the same wait states around the MFMA.
#define INFCL_MFMA16_AB(PRE, OP)                                                                                \
  if (first && last)                                                                                           \
    asm volatile(PRE OP " %0, %1, %2, 0\n\ts_nop 7\n\ts_nop 7\n\ts_nop 3" : "=&v"(acc) : "v"(a), "a"(b));   \
  else if (first)                                                                                              \
    asm volatile(PRE OP " %0, %1, %2, 0" : "=&v"(acc) : "v"(a), "a"(b));                                        \
  else if (last)                                                                                               \
    asm volatile(PRE OP " %0, %1, %2, %0\n\ts_nop 7\n\ts_nop 7\n\ts_nop 3" : "+v"(acc) : "v"(a), "a"(b));  \
  else                                                                                                         \
    asm volatile(PRE OP " %0, %1, %2, %0" : "+v"(acc) : "v"(a), "a"(b));
template <bool F16, bool PAD = true>
__device__ __forceinline__ void mfma16_vgpr_ab(f32x16& acc, const bf16x8& a, const bf16x8& b, bool first, bool last) {
  if constexpr (F16) {
    if constexpr (PAD) {
      INFCL_MFMA16_AB("s_nop 1\n\t", "v_mfma_f32_32x32x16_f16")
    } else {
      INFCL_MFMA16_AB("", "v_mfma_f32_32x32x16_f16")
    }
  } else {
    if constexpr (PAD) {
      INFCL_MFMA16_AB("s_nop 1\n\t", "v_mfma_f32_32x32x16_bf16")
    } else {
      INFCL_MFMA16_AB("", "v_mfma_f32_32x32x16_bf16")
    }
  }
}
#undef INFCL_MFMA16_AB
// Widest spread (log2 units) between the wave reference and a row or column
// reference for which the factorised column pass keeps every entry that
// matters: a lost term is below 2^-(126 - kWide) of its column reference.
constexpr float kWide = 30.f;

// <img_i, txt_i> in fp32 and its base-2 scaled value; 8 lanes per row.
template <bool F16>
__global__ void __launch_bounds__(256) fwd2_diag(const __bf16* img, const __bf16* txt, int64_t b, int64_t d,
                                                 const float* scale, float* udiag, float* ref2) {
  const int64_t i = (int64_t)blockIdx.x * 32 + (threadIdx.x >> 3);
  const int l8 = threadIdx.x & 7;
  float acc = 0.f;
  if (i < b) {
    const bf16x8* a = (const bf16x8*)(img + i * d);
    const bf16x8* t = (const bf16x8*)(txt + i * d);
    for (int64_t c = l8; c < d / 8; c += 8) {
      const bf16x8 x = a[c], y = t[c];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc = __builtin_fmaf(from16<F16>(x[e]), from16<F16>(y[e]), acc);
    }
  }
  acc += shfl_xor(acc, 1);
  acc += shfl_xor(acc, 2);
  acc += shfl_xor(acc, 4);
  if (i < b && l8 == 0) {
    udiag[i] = acc;
    ref2[i] = acc * (scale[0] * kLog2e);
  }
}

template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
// Lane of a 32-lane half that ends with value index i in rs16_sum.
__device__ __forceinline__ int rs16_index(int lane) {
  return 8 * ((lane >> 4) & 1) + 4 * ((lane >> 3) & 1) + 2 * ((lane >> 2) & 1) + ((lane >> 1) & 1);
}
// Reduce-scatter (sum, or max when kMax) over the 32 lanes of each wave half
// for 16 values, without LDS traffic: on exit lane l holds the total of value
// index rs16_index(l) (lanes l and l ^ 1 alike).  Lanes l and l ^ 16 pair up
// through permlane16_swap, then l ^ 8 (row rotate by 8), l ^ 7 (half-row
// mirror), l ^ 3 and l ^ 1 (quad permutes) through DPP.
template <bool kMax>
__device__ __forceinline__ float rs16_op(float a, float b) {
  return kMax ? fmaxf(a, b) : a + b;
}
template <bool kMax>
__device__ __forceinline__ float rs16(float (&v)[16], int lane) {
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    // even rows keep v[t] and receive the odd rows' v[t]; odd rows keep v[t+8]
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v[t]), __float_as_uint(v[t + 8]), false, false);
    v[t] = rs16_op<kMax>(__uint_as_float(r[0]), __uint_as_float(r[1]));
  }
  const bool b3 = (lane & 8) != 0, b2 = (lane & 4) != 0, b1 = (lane & 2) != 0;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const float send = b3 ? v[t] : v[t + 4], keep = b3 ? v[t + 4] : v[t];
    v[t] = rs16_op<kMax>(keep, dpp_f<0x128>(send));  // row_ror:8
  }
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const float send = b2 ? v[t] : v[t + 2], keep = b2 ? v[t + 2] : v[t];
    v[t] = rs16_op<kMax>(keep, dpp_f<0x141>(send));  // row_half_mirror
  }
  {
    const float send = b1 ? v[0] : v[1], keep = b1 ? v[1] : v[0];
    v[0] = rs16_op<kMax>(keep, dpp_f<0x1B>(send));  // quad_perm [3,2,1,0]
  }
  return rs16_op<kMax>(v[0], dpp_f<0xB1>(v[0]));  // quad_perm [1,0,3,2]
}

// The pair (R, l) as one reference: R + log2 l, or -inf when empty.
__device__ __forceinline__ float pair_level(float R, float l) {
  return l > 0.f ? R + __builtin_amdgcn_logf(l) : -__builtin_inff();
}

template <int D, bool F16>
__global__ void __launch_bounds__(64 * fwd2_waves(D), D > 512 ? 1 : 2) fwd_sweep2(Fwd2Params p) {
  constexpr int NW = fwd2_waves(D);
  constexpr int BM = 32 * NW;  // own rows per row block
  constexpr int KS = D / 16;
  constexpr int ROWG = D * 2;
  constexpr int TILEB = kSweepBN * ROWG;
  constexpr int NIW = TILEB / 1024 / NW;  // 1 KiB DMA instructions per wave and tile
#ifndef INFCL_F2_PRE
#define INFCL_F2_PRE 4
#endif
#ifndef INFCL_F2_PRE_WIDE
#define INFCL_F2_PRE_WIDE 6
#endif
  constexpr int kPreD = D > 512 ? INFCL_F2_PRE_WIDE : INFCL_F2_PRE;
  constexpr int kPre = KS < kPreD ? KS : kPreD;
  static_assert(D % 64 == 0 && D <= 1024 && NIW >= 1 && KS % NIW == 0, "tile DMA layout");
  static_assert((D > 512 ? 1 : 2) * (2 * TILEB + 4 * 1024 + 5 * 512) <= 160 * 1024, "workgroups per CU");
  __shared__ __attribute__((aligned(1024))) char tA_[TILEB];
  __shared__ __attribute__((aligned(1024))) char tB_[TILEB];
  // running pairs of the tile's 32 columns: R at [0, 256), l at [256, 512);
  // the DMA writes 8 copies of each 32-float row
  __shared__ __attribute__((aligned(1024))) float sA_[512];
  __shared__ __attribute__((aligned(1024))) float sB_[512];
  // per tile parity, column and wave: the wave's partial pair (reference, sum)
  __shared__ __attribute__((aligned(16))) float cxR_[2][32][NW];
  __shared__ __attribute__((aligned(16))) float cxS_[2][32][NW];
  __shared__ __attribute__((aligned(16))) float cw_[NW][32];  // per wave: column maxima (bounds-failure path)
  INFCL_LDS char* const tA = (INFCL_LDS char*)tA_;
  INFCL_LDS char* const tB = (INFCL_LDS char*)tB_;
  INFCL_LDS float* const sA = (INFCL_LDS float*)sA_;
  INFCL_LDS float* const sB = (INFCL_LDS float*)sB_;

  const int lane = __lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31, h = lane >> 5;
  // tile DMA: instruction k = wq + 4 kk of the swept-tile layout, kk in [kk0, kk0 + NIW)
  const int wq = wave & 3, kk0 = (wave >> 2) * NIW;
  // the running column pairs of a tile are loaded by one wave (8 waves) or,
  // branch-free, by every wave (4 waves)
  const bool slot_wave = NW == 4 || wave == 0;
  const int b = (int)p.b;  // at most 2^30
  const int g = blockIdx.x % p.Pc;
  const int q = blockIdx.x / p.Pc;
  const int ct_lo = (int)(((uint32_t)g * (uint32_t)p.nCT) / (uint32_t)p.Pc);
  const int ct_hi = (int)(((uint32_t)(g + 1) * (uint32_t)p.nCT) / (uint32_t)p.Pc);
  if (ct_hi <= ct_lo || q >= p.nRB) return;  // uniform over the workgroup
  const float k2 = p.scale[0] * kLog2e;
  const float ninf = -__builtin_inff();
  float* const cR = p.colR + (int64_t)q * b;
  float* const cL = p.colL + (int64_t)q * b;

  // Per-lane address parts, computed once (rebuilding them per tile costs
  // VALU cycles between the tile's phases): the DMA source offset of this
  // lane, the column-pair slot offset, and GEMM1's swept fragment offsets
  // (tile base + kSeg (n >> 3) + offA[n & 7]).
  const uint32_t dma_lo = sweep_dma_lane_off(lane, wq, ROWG);
  // d > 512 (registers to spare): the full source offset of each of the
  // wave's DMA instructions, computed once, so that no VALU instruction
  // writes a DMA operand inside the sweep and the DMA needs one wait state
  uint32_t dvo[D > 512 ? NIW : 1];
#pragma unroll
  for (int k = 0; k < (D > 512 ? NIW : 1); ++k) dvo[k] = dma_lo + sweep_dma_kk_off(kk0 + k, wq, ROWG);
  const uint32_t slot_lo = 16u * (uint32_t)(lane & 7);
  int offA[8];
  {
    const int rA = sweep_perm(l32);
#pragma unroll
    for (int k = 0; k < 8; ++k) offA[k] = sweep_seg_off(rA, 2 * k + h);
  }
  // swept row (tile-relative) of accumulator entry r of this lane
  auto jrow = [&](int r) { return 16 * (r >> 3) + 8 * h + (r & 7); };
  auto tile_rsrc = [&](int jt) {
    const int j0 = (jt < 0 ? 0 : jt) * kSweepBN;
    return rsrc_words((const char*)p.txt + (int64_t)j0 * ROWG, jt < 0 ? 0 : (int64_t)(b - j0) * ROWG);
  };
  // running column pairs of tile jt into slot: on a workgroup's first row
  // block the reference is the diagonal value and the sum empty (a resource
  // of zero bytes loads zeros)
  auto issue_slot = [&](int jt, bool first_rb, INFCL_LDS float* slot) {
    const int j0 = (jt < 0 ? 0 : jt) * kSweepBN;
    const int64_t nb = jt < 0 ? 0 : (int64_t)(b - j0) * 4;
    dma16_asm(rsrc_words(first_rb ? p.ref2 + j0 : cR + j0, nb), slot, slot_lo);
    dma16_asm(rsrc_words(cL + j0, first_rb ? 0 : nb), slot + 256, slot_lo);
  };

  for (int rb = q; rb < p.nRB; rb += p.Pr) {
    const bool first_rb = rb == q;
    const int own0 = p.r0 + rb * BM + 32 * wave;  // r0 is a multiple of 32: own blocks stay tile-aligned
    const int iown = own0 + l32;
    const bool own_ok = iown < p.rend;
    const int irow = own_ok ? iown : p.rend - 1;
    const bool wave_rows_ok = own0 + 32 <= p.rend;
    const bool wave_any_row = own0 < p.rend;

    bf16x8 ownf[KS];
    {
      const __bf16* src = p.img + (int64_t)irow * D + 8 * h;
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2) ownf[s2] = *(const bf16x8*)(src + 16 * s2);
    }
    float rowR = p.ref2[irow], rowL = 0.f;  // this lane's pair for its row over its half of the columns
    // wave reference c = max of the wave's row references, alpha = exp2(R_i - c)
    float cw = 0.f, alpha = 0.f;
    bool rows_wide = false;
    auto refresh = [&]() {
      float m = own_ok ? rowR : ninf;
#pragma unroll
      for (int k = 1; k < 64; k <<= 1) m = fmaxf(m, shfl_xor(m, k));
      cw = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(m == ninf ? 0.f : m)));
      alpha = own_ok ? exp2_hw(rowR - cw) : 0.f;
      rows_wide = wave_any(own_ok && rowR < cw - kWide);
    };
    refresh();

    {
      const u32x4 rs = tile_rsrc(ct_lo);
#pragma unroll
      for (int k = 0; k < NIW; ++k)
        dma16_asm(rs, tA + 1024 * (wq + 4 * (kk0 + k)), dma_lo + sweep_dma_kk_off(kk0 + k, wq, ROWG));
      if (slot_wave) issue_slot(ct_lo, first_rb, sA);
    }
    wait_dma();
    __syncthreads();

    // one tile: GEMM1 of the tile in cur (issuing the DMA of tile jt+1 into
    // nxt between its MFMAs), row statistics, column partials, exchange, merge
    // merge of a tile's column pairs, deferred into the next tile: lanes 0..7
    // of wave w own columns 8w .. 8w+7 of the tile
    int pjg = -1;              // global column of the pending merge (-1: none)
    float pRold = 0.f, pLold = 0.f;
    const int jc = 8 * wq + (lane & 7);
    const bool merger = lane < 8 && wave < 4;
    // the NW wave pairs of column jc of a tile (parity par)
    auto pairs = [&](int par, float (&rw)[NW], float (&sw)[NW]) {
#pragma unroll
      for (int w4 = 0; w4 < NW; w4 += 4) {
        const f32x4 r4 = *(const INFCL_LDS f32x4*)&cxR_[par][jc][w4];
        const f32x4 s4 = *(const INFCL_LDS f32x4*)&cxS_[par][jc][w4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          rw[w4 + c] = r4[c];
          sw[w4 + c] = s4[c];
        }
      }
    };
    auto merge = [&](const float (&rw)[NW], const float (&sw)[NW]) {
      if (merger && pjg >= 0 && pjg < b) {
        float R, L;
        bool same = true;
#pragma unroll
        for (int w = 0; w < NW; ++w) same = same & (rw[w] == pRold);
        if (same) {
          float t = 0.f;
#pragma unroll
          for (int w = 0; w < NW; ++w) t += sw[w];
          R = pRold;
          L = pLold + t;
        } else {
          // some wave used its own reference: merge the pairs by level
          float lv[NW + 1];
          lv[0] = pair_level(pRold, pLold);
#pragma unroll
          for (int w = 0; w < NW; ++w) lv[w + 1] = pair_level(rw[w], sw[w]);
          float M = lv[0];
#pragma unroll
          for (int k = 1; k <= NW; ++k) M = fmaxf(M, lv[k]);
          if (M == ninf) {
            R = pRold;
            L = 0.f;
          } else {
            L = 0.f;
#pragma unroll
            for (int k = 0; k <= NW; ++k) L += exp2_hw(lv[k] - M);
            R = M;
          }
        }
        cR[pjg] = R;
        cL[pjg] = L;
      }
    };

    // GEMM1 of the tile in cur (S^T block of the wave's rows), with the DMA
    // of tile jn into nxt (its column pairs into snxt) issued between the MFMAs
    auto gemm1 = [&](const INFCL_LDS char* cur, int jn, INFCL_LDS char* nxt, INFCL_LDS float* snxt) {
      f32x16 sacc;
      const u32x4 drs = tile_rsrc(jn);
      bf16x8 ring[kPre];
#pragma unroll
      for (int i = 0; i < kPre; ++i) ring[i] = *(const INFCL_LDS bf16x8*)(cur + offA[i & 7] + kSeg * (i >> 3));
      __builtin_amdgcn_sched_group_barrier(0x100, kPre, 0);
      // (MFMAs without leading padding: their sources are LDS loads and the
      // own rows loaded before the sweep, which the build's scan confirms)
      static_for<KS>([&](auto s2c) {
        constexpr int s2 = decltype(s2c)::value;
        if constexpr (D > 512)  // own rows in AGPRs
          mfma16_vgpr_ab<F16, false>(sacc, ring[s2 % kPre], ownf[s2], s2 == 0, s2 == KS - 1);
        else
          mfma16_vgpr<F16, false>(sacc, ring[s2 % kPre], ownf[s2], s2 == 0, s2 == KS - 1);
        constexpr int SPI = KS / NIW;  // steps per DMA instruction
        if ((s2 + 1) % SPI == 0) {
          const int kk = kk0 + (s2 + 1) / SPI - 1;
          if constexpr (D > 512)
            dma16_asm_w1(drs, nxt + 1024 * (wq + 4 * kk), dvo[(s2 + 1) / SPI - 1]);
          else
            dma16_asm(drs, nxt + 1024 * (wq + 4 * kk), dma_lo + sweep_dma_kk_off(kk, wq, ROWG));
        }
        if (slot_wave && s2 == (KS > 1 ? 1 : 0)) issue_slot(jn, first_rb, snxt);
        if constexpr (s2 + kPre < KS) {
          constexpr int n = s2 + kPre;
          ring[s2 % kPre] = *(const INFCL_LDS bf16x8*)(cur + offA[n & 7] + kSeg * (n >> 3));
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
      });
      return sacc;
    };

    // Statistics of tile jt from its S^T block: row update, this wave's column
    // partial pairs into LDS (parity par)
    auto stats = [&](int jt, const f32x16& sacc, const INFCL_LDS float* scur, int par, float Rmine, float Lmine) {
      const int j0 = jt * kSweepBN;
      const int jl = jrow(rs16_index(lane));  // the column whose partial this lane ends with
      // entries off the problem or on the diagonal take no part (uniform test)
      const bool special = (j0 == own0) || (j0 + kSweepBN > b) || !wave_rows_ok;
      // (bitwise operators: no short-circuit branches)
      auto keep = [&](int r) {
        const int j = j0 + jrow(r);
        return (bool)(own_ok & (j < b) & (j != iown));
      };
      // scaled entry r, -inf when it takes no part.  Used only on the rare
      // paths below; the opaque copy keeps the compiler from hoisting these
      // 16 products (and the masks) out of those paths into the common one.
      auto yv = [&](int r) {
        float x = sacc[r];
        asm volatile("" : "+v"(x));
        return (!special | keep(r)) ? x * k2 : ninf;
      };
      // ---- row: lazy against its reference, exact when a bound fails
      float e[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) e[r] = exp2_hw(__builtin_fmaf(sacc[r], k2, -rowR));
      if (special) {
#pragma unroll
        for (int r = 0; r < 16; ++r) e[r] = keep(r) ? e[r] : 0.f;
      }
      bool rchg = false;
      {
        float t = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) t += e[r];
        const float nl = rowL + t;
        if (lazy_ok(t) && nl >= kTinyBound) {
          rowL = nl;
        } else {
          float m = ninf;
#pragma unroll
          for (int r = 0; r < 16; ++r) m = fmaxf(m, yv(r));
          const float lev = pair_level(rowR, rowL);
          const float Rn = fmaxf(lev, m);
          if (Rn != ninf) {
            float s = rowL > 0.f ? exp2_hw(lev - Rn) : 0.f;
#pragma unroll
            for (int r = 0; r < 16; ++r) s += exp2_hw(yv(r) - Rn);
            rowR = Rn;
            rowL = s;
            rchg = true;
          }
        }
      }
      // ---- columns: this wave's partial per column against the column's
      // running reference.  Factorised: exp2(y - R_j) = e * alpha *
      // exp2(c - R_j) with e = exp2(y - R_i) from the row pass, so one
      // exponential per entry; when references lie far apart (wide), the
      // entries are exponentiated against R_j directly.
      float v[16];
      float part;
      if (!wave_any(rows_wide || Rmine < cw - kWide)) {
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = e[r] * alpha;
        part = rs16<false>(v, lane) * exp2_hw(cw - Rmine);
      } else {
        const INFCL_LDS char* sp = (const INFCL_LDS char*)scur + 32 * h;
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const f32x4 r4 = *(const INFCL_LDS f32x4*)(sp + 64 * (q4 >> 1) + 16 * (q4 & 1));
#pragma unroll
          for (int c = 0; c < 4; ++c) v[4 * q4 + c] = exp2_hw(yv(4 * q4 + c) - r4[c]);
        }
        part = rs16<false>(v, lane);
      }
      float Rw = Rmine;
      const bool mine_bad = !lazy_ok(part) || (Lmine + part < kTinyBound && j0 + jl < b && wave_any_row);
      if (wave_any(mine_bad)) {
        // bounds failure: the wave's partial against its own column maxima
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = yv(r);
        const float mx = rs16<true>(v, lane);
        if ((lane & 1) == 0) cw_[wave][jl] = mx;
        const INFCL_LDS char* mp = (const INFCL_LDS char*)&cw_[wave][0] + 32 * h;
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const f32x4 m4 = *(const INFCL_LDS f32x4*)(mp + 64 * (q4 >> 1) + 16 * (q4 & 1));
#pragma unroll
          for (int c = 0; c < 4; ++c) v[4 * q4 + c] = exp2_hw(yv(4 * q4 + c) - (m4[c] == ninf ? 0.f : m4[c]));
        }
        const float s2 = rs16<false>(v, lane);
        Rw = mx == ninf ? Rmine : mx;
        part = mx == ninf ? 0.f : s2;
      }
      if ((lane & 1) == 0) {  // lanes l and l ^ 1 hold the same column
        cxR_[par][jl][wave] = Rw;
        cxS_[par][jl][wave] = part;
      }
      if (wave_any(rchg)) refresh();
    };

    const int jl_lane = jrow(rs16_index(lane));
    // one tile: GEMM1 of the tile in cur (issuing the DMA of tile jt+1 into
    // nxt between its MFMAs), the pending merge, row statistics, column
    // partial pairs into LDS
    auto body = [&](int jt, const INFCL_LDS char* cur, const INFCL_LDS float* scur, INFCL_LDS char* nxt,
                    INFCL_LDS float* snxt, int par) {
      const int jn = jt + 1 < ct_hi ? jt + 1 : -1;
      const float Rmine = scur[jl_lane], Lmine = scur[256 + jl_lane];
      const float Rold = scur[jc], Lold = scur[256 + jc];
      float prw[NW], psw[NW];
      pairs(par ^ 1, prw, psw);
      const f32x16 sacc = gemm1(cur, jn, nxt, snxt);
      merge(prw, psw);
      stats(jt, sacc, scur, par, Rmine, Lmine);
      pjg = jt * kSweepBN + jc;
      pRold = Rold;
      pLold = Lold;
      wait_dma();  // the next tile and its column pairs are in LDS after the barrier
      __syncthreads();
    };
    for (int jt = ct_lo; jt < ct_hi; jt += 2) {
      body(jt, tA, sA, tB, sB, 0);
      if (jt + 1 < ct_hi) body(jt + 1, tB, sB, tA, sA, 1);
    }
    {
      const int lpar = (ct_hi - 1 - ct_lo) & 1;  // parity of the last tile
      float rw[NW], sw[NW];
      pairs(lpar, rw, sw);
      merge(rw, sw);
    }

    // ---- end of the row block: merge the two lane halves, publish the row pair
    {
      float R = rowR, L = rowL;
      lse2_merge(R, L, shfl_xor(rowR, 32), shfl_xor(rowL, 32));
      if (h == 0 && own_ok) {
        p.rowR[(int64_t)g * p.rstride + (iown - p.r0)] = R;
        p.rowL[(int64_t)g * p.rstride + (iown - p.r0)] = L;
      }
    }
    // column pairs stored in this row block are read by the next one's DMA
    wait_dma();
    __syncthreads();
  }
}

template <int D>
static int launch_fwd2_d(const Fwd2Params& p, bool f16, hipStream_t stream) {
  if (f16)
    hipLaunchKernelGGL((fwd_sweep2<D, true>), dim3(p.Pr * p.Pc), dim3(64 * fwd2_waves(D)), 0, stream, p);
  else
    hipLaunchKernelGGL((fwd_sweep2<D, false>), dim3(p.Pr * p.Pc), dim3(64 * fwd2_waves(D)), 0, stream, p);
  return hipGetLastError() == hipSuccess ? 0 : 1;
}

// 16-bit inputs (bf16 = 0, fp16 = 2) with d a multiple of 128 up to 1024
bool fwd2_supported(int64_t d, int dtype) { return (dtype == 0 || dtype == 2) && d % 128 == 0 && d >= 128 && d <= 1024; }

// Grid of the resident-rows forward for nrows own rows of width d against b
// columns: P_c column groups (one per XCD) times P_r row groups, P_r P_c <= 256
// workgroups (one per CU) with 8 waves or with 4 waves at d > 512, and 512 (two
// per CU) with the 4-wave build option at d <= 512.
void fwd2_grid(int64_t b, int64_t nrows, int64_t d, int* Pr, int* Pc) {
  const int64_t bm = 32 * fwd2_waves(d);
  const int64_t nRB = (nrows + bm - 1) / bm, nCT = (b + kSweepBN - 1) / kSweepBN;
  *Pc = (int)(nCT < 8 ? nCT : 8);
  const int64_t pmax = d > 512 ? 32 : 256 / kF2NW;
  *Pr = (int)(nRB < pmax ? nRB : pmax);
}

int launch_fwd2(const void* img, const void* txt, int64_t b, int64_t d, int dtype, int64_t r0, int64_t nrows,
                const float* scale, float* rowR, float* rowL, float* colR, float* colL, float* udiag, float* ref2,
                hipStream_t stream) {
  const bool f16 = dtype == 2;
  if (f16)
    hipLaunchKernelGGL(fwd2_diag<true>, dim3((unsigned)((b + 31) / 32)), dim3(256), 0, stream, (const __bf16*)img,
                       (const __bf16*)txt, b, d, scale, udiag, ref2);
  else
    hipLaunchKernelGGL(fwd2_diag<false>, dim3((unsigned)((b + 31) / 32)), dim3(256), 0, stream, (const __bf16*)img,
                       (const __bf16*)txt, b, d, scale, udiag, ref2);
  if (hipGetLastError() != hipSuccess) return 1;
  Fwd2Params p;
  p.img = (const __bf16*)img;
  p.txt = (const __bf16*)txt;
  p.b = b;
  p.scale = scale;
  p.ref2 = ref2;
  p.rowR = rowR;
  p.rowL = rowL;
  p.colR = colR;
  p.colL = colL;
  p.r0 = (int)r0;
  p.rend = (int)(r0 + nrows);
  p.rstride = nrows;
  fwd2_grid(b, nrows, d, &p.Pr, &p.Pc);
  p.nRB = (int)((nrows + 32 * fwd2_waves(d) - 1) / (32 * fwd2_waves(d)));
  p.nCT = (int)((b + kSweepBN - 1) / kSweepBN);
  switch (d) {
    case 128: return launch_fwd2_d<128>(p, f16, stream);
    case 256: return launch_fwd2_d<256>(p, f16, stream);
    case 384: return launch_fwd2_d<384>(p, f16, stream);
    case 512: return launch_fwd2_d<512>(p, f16, stream);
    case 640: return launch_fwd2_d<640>(p, f16, stream);
    case 768: return launch_fwd2_d<768>(p, f16, stream);
    case 896: return launch_fwd2_d<896>(p, f16, stream);
    case 1024: return launch_fwd2_d<1024>(p, f16, stream);
  }
  return 2;
}

}  // namespace infcl
