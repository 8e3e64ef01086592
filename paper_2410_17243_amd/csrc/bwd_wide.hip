// Backward sweep for wide rows (16-bit inputs: bf16 or fp16, d = 768 or
// 1024) in a single pass (gfx950): bwd_wide below, the serial form, serves
// d = 1024; bwd_wide3 further down, the pipelined form, serves d = 768.
//
// Same quantities as the 128-row sweep (Sec. 3.1, Eq. 6-8 completed for both
// halves of the loss and the scale; the appendix's in-GPU backward recomputes
// every tile from the saved log-sum-exp vectors).  At these widths the
// gradient accumulators of 128 own rows (128 x d fp32) do not fit the
// register file, so a workgroup owns 64 rows instead: 64 x d fp32 is 192 or
// 256 AGPRs per wave.  GEMM1's own operand is then split by contraction: the
// wave pair (2 ob, 2 ob + 1) holds own block ob (32 rows), each wave one half
// of the features (d/8 VGPRs), and computes a partial S^T block over its half.
// Per tile:
//   GEMM1   partial S^T (32 swept x 32 own) over the wave's feature half
//           (and the DMA of the next tile's log-sum-exp slot);
//   join    each wave hands the partner the 8 accumulator entries the
//           partner finishes (LDS), then adds the partner's half of its own 8;
//   G'      two exp2 per entry for the wave's 8 entries, the diagonal from
//           expm1 terms, the dscale contribution; rounded to the input
//           type into the shared G' block (64 own x 32 swept).  The DMA of
//           the next tile (all four waves) is issued here, between the
//           entries: in this phase, which has no MFMAs, its instructions cost
//           far less than between GEMM1's MFMAs (a whole-tile phase trace at
//           d = 768, when this form served it: GEMM1 took 3170 cycles with
//           the DMA and 1300 without);
//   GEMM2   each wave multiplies all 64 own rows' G' by its quarter of the
//           features of the tile (transposing LDS reads), accumulating in
//           AGPRs.
// Three barriers per tile (join, G' block, buffer turn-over).
#include <type_traits>

#include "bwd.hpp"


namespace infcl {

constexpr int kWideBM = 64;  // own rows per workgroup

template <int D, bool F16, bool G16>
__global__ void __launch_bounds__(256, 1) bwd_wide(BwdParams p) {
  using GO = GradOut<G16, F16>;  // gradient element type
  constexpr int KS = D / 16;  // 16-wide contraction steps of the full width
  constexpr int KH = KS / 2;  // steps of one wave (half the features)
  constexpr int ROWG = D * 2;
  constexpr int TILEB = kBwdBN * ROWG;
  constexpr int NIW = TILEB / 4096;  // 1 KiB DMA instructions per wave and tile
  constexpr int FBW = D / 128;       // 32-feature blocks of GEMM2 per wave
  constexpr int kPre = 4;
  static_assert(KH % 8 == 0, "feature halves start on a 128-feature segment");
  static_assert(2 * TILEB + 2 * 1024 + kWideBM * kBwdBN * 2 + 4 * 64 * 32 + 2048 <= 160 * 1024, "LDS budget");
  __shared__ __attribute__((aligned(1024))) char tA_[TILEB];
  __shared__ __attribute__((aligned(1024))) char tB_[TILEB];
  __shared__ __attribute__((aligned(1024))) float lA_[256];
  __shared__ __attribute__((aligned(1024))) float lB_[256];
  // G' of the workgroup's 64 own rows for one tile: 64-byte rows (32 swept
  // rows, input type) whose four 16-byte chunks are XOR-swizzled by (row >> 2) & 3
  __shared__ __attribute__((aligned(1024))) char gp_[kWideBM * kBwdBN * 2];
  // join: per wave and lane the 8 partial entries its partner finishes
  __shared__ __attribute__((aligned(16))) float xs_[4][64][8];
  __shared__ double red[256];
  INFCL_LDS char* const tA = (INFCL_LDS char*)tA_;
  INFCL_LDS char* const tB = (INFCL_LDS char*)tB_;
  INFCL_LDS float* const lA = (INFCL_LDS float*)lA_;
  INFCL_LDS float* const lB = (INFCL_LDS float*)lB_;
  INFCL_LDS char* const gp = (INFCL_LDS char*)gp_;

  const int lane = __lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ob = wave >> 1, kh = wave & 1;  // own block, feature half of GEMM1
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t b = p.b;
  const int64_t wg0 = p.own_off + (int64_t)blockIdx.x * kWideBM;  // own_off is a multiple of 32
  const int64_t own0 = wg0 + 32 * ob;                              // this wave's own block
  const int64_t iown = own0 + l32;
  const bool own_ok = iown < p.own_end;
  const int64_t irow = own_ok ? iown : p.own_end - 1;
  const bool wave_rows_ok = own0 + 32 <= p.own_end;
  const int ntile = (int)((b + kBwdBN - 1) / kBwdBN);

  const float s = p.scale[0];
  const float k2 = s * kLog2e;
  const float dl = p.dloss ? p.dloss[0] : 1.0f;
  // fp16: G' is rounded after scaling by alpha = g16[0], divided out at the end
  const float g16a = F16 ? p.g16[0] : 1.0f;
  const float kfin = dl * s / (2.0f * (float)b) * (F16 ? p.g16[1] : 1.0f);

  // own operand of GEMM1: row irow, features kh d/2 + 16 s2 + 8h .. +8
  bf16x8 ownf[KH];
  {
    const __bf16* src = (const __bf16*)p.own + irow * D + kh * (D / 2) + 8 * h;
#pragma unroll
    for (int s2 = 0; s2 < KH; ++s2) ownf[s2] = *(const bf16x8*)(src + 16 * s2);
  }
  const float aO = own_ok ? p.lse_own[iown] * kLog2e : 0.f;
  const float uO = own_ok ? p.udiag[iown] : 0.f;
  const float gdiag = own_ok ? expm1f(-p.ell_own[iown]) + expm1f(-p.ell_swept[iown]) : 0.f;

  auto opaque_lane = [&]() {
    int lo = lane;
    asm volatile("" : "+v"(lo));
    return lo;
  };
  auto tile_rsrc = [&](int jt) {
    const int64_t j0 = (int64_t)(jt < 0 ? 0 : jt) * kBwdBN;
    return rsrc_words((const char*)p.swept + j0 * ROWG, jt < 0 ? 0 : (b - j0) * ROWG);
  };
  auto lse_rsrc = [&](int jt) {
    const int64_t j0 = (int64_t)(jt < 0 ? 0 : jt) * kBwdBN;
    return rsrc_words(p.lse2_swept + j0, jt < 0 ? 0 : (b - j0) * 4);
  };
  auto lse_lane_off = [&]() { return 16u * (uint32_t)(opaque_lane() & 7); };
  // Per-lane address parts are rebuilt at each use from an opaque lane id:
  // at d = 1024 all 512 registers are taken, so a value held across the loop
  // would be spilled, and a scratch reload waits for all DMA in flight.
  auto dma_lo = [&]() { return sweep_dma_lane_off(opaque_lane(), wave, ROWG); };
  // The kh = 1 wave loads the tile's rows 16..31 into MFMA rows 0..15 and
  // rows 0..15 into 16..31 (row index XOR 16; the row does not enter the bank
  // of a chunk): accumulator entries 0..7 of either wave are then the ones it
  // finishes (tile rows 16 kh + 8 h + i), entries 8..15 the ones it hands over.
  auto make_offA = [&](int lo, int (&o)[8]) {
    const int rA = sweep_perm(lo & 31) ^ (16 * kh);
#pragma unroll
    for (int k = 0; k < 8; ++k) o[k] = sweep_seg_off(rA, 2 * k + (lo >> 5));
  };
  // GEMM2's transposing reads (tile base + offB[t][fbw] + 16 kSegRow s2) and
  // G' fragments (G' block + offG[s2])
  auto make_offBG = [&](int lo, int (&oB)[2][FBW], int (&oG)[2]) {
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int fbw = 0; fbw < FBW; ++fbw) oB[t][fbw] = sweep_tr_off(lo, t, wave * FBW + fbw);
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) oG[s2] = gp_chunk_off(lo & 31, 2 * s2 + (lo >> 5));
  };

  double ds_acc = 0.0;
  f32x16 dacc[2 * FBW];
#pragma unroll
  for (int i = 0; i < 2 * FBW; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dacc[i][r] = 0.f;

  // ---- GEMM1 over this wave's feature half of the tile in cur; issues the
  // DMA of tile dtile's log-sum-exp slot
  auto gemm1 = [&](const INFCL_LDS char* cur, int dtile, INFCL_LDS float* dlse) {
    int offA[8];
    make_offA(opaque_lane(), offA);
    const INFCL_LDS char* half = cur + kSeg * (kh * KH / 8);
    const u32x4 drl = lse_rsrc(dtile);
    f32x16 sacc;
    bf16x8 ring[kPre];
#pragma unroll
    for (int i = 0; i < kPre; ++i) ring[i] = *(const INFCL_LDS bf16x8*)(half + offA[i & 7] + kSeg * (i >> 3));
    __builtin_amdgcn_sched_group_barrier(0x100, kPre, 0);
#pragma unroll
    for (int s2 = 0; s2 < KH; ++s2) {
      mfma16_vgpr<F16, false>(sacc, ring[s2 % kPre], ownf[s2], s2 == 0, s2 == KH - 1);  // unpadded: scan-checked
      if (s2 == 1) dma16_asm(drl, dlse, lse_lane_off());
      if (s2 + kPre < KH) {
        const int n = s2 + kPre;
        ring[s2 % kPre] = *(const INFCL_LDS bf16x8*)(half + offA[n & 7] + kSeg * (n >> 3));
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
    }
    return sacc;
  };

  // ---- join, G' of the wave's 8 entries (entry i <-> swept row
  // 16 kh + 8h + i of the tile) into the G' block, with the DMA of tile
  // dtile into ddst spread over the entries; returns dscale's share
  auto join_gp = [&](int jt, const INFCL_LDS float* lcur, const f32x16& sacc, int dtile,
                     INFCL_LDS char* ddst) -> float {
    float mine[8], other[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      mine[i] = sacc[i];
      other[i] = sacc[8 + i];
    }
    *(INFCL_LDS f32x4*)&xs_[wave][lane][0] = f32x4{other[0], other[1], other[2], other[3]};
    *(INFCL_LDS f32x4*)&xs_[wave][lane][4] = f32x4{other[4], other[5], other[6], other[7]};
    __syncthreads();
    const f32x4 q0 = *(const INFCL_LDS f32x4*)&xs_[wave ^ 1][lane][0];
    const f32x4 q1 = *(const INFCL_LDS f32x4*)&xs_[wave ^ 1][lane][4];
    const INFCL_LDS float* lp = lcur + 16 * kh + 8 * h;
    const f32x4 L0 = *(const INFCL_LDS f32x4*)lp;
    const f32x4 L1 = *(const INFCL_LDS f32x4*)(lp + 4);
    const int64_t j0 = (int64_t)jt * kBwdBN;
    const bool special = (j0 == own0) || (j0 + kBwdBN > b) || !wave_rows_ok;
    float ds_tile = 0.f;
    bf16x8 ga;
    const u32x4 drs = tile_rsrc(dtile);
    const uint32_t dlo = dma_lo();
#pragma unroll
    for (int i = 0; i < 8; ++i) {
#pragma unroll
      for (int u = 0; u < (NIW + 7) / 8; ++u) {  // DMA instructions i, i + 8, ...
        const int kk = i + 8 * u;
        // the lane offset in a VGPR, the instruction's part as the scalar
        // offset: only the first instruction follows the lane offset's
        // arithmetic closely enough to need the full padding
        if (kk == 0)
          dma16_asm(drs, ddst + 1024 * wave, dlo, sweep_dma_kk_off(0, wave, ROWG));
        else if (kk < NIW)
          dma16_asm_w1(drs, ddst + 1024 * (wave + 4 * kk), dlo, sweep_dma_kk_off(kk, wave, ROWG));
      }
      const float x = mine[i] + (i < 4 ? q0[i] : q1[i - 4]);
      const float Lj = i < 4 ? L0[i] : L1[i - 4];
      const float pO = exp2_hw(__builtin_fmaf(x, k2, -aO));
      const float pS = exp2_hw(__builtin_fmaf(x, k2, -Lj));
      float gg = pO + pS;
      float dsv = pO * (x - uO);
      if (special) {
        const int64_t j = j0 + 16 * kh + 8 * h + i;
        const bool ok = (bool)(own_ok & (j < b));
        const bool dg = j == iown;
        gg = dg ? gdiag : (ok ? gg : 0.f);
        dsv = (ok & !dg) ? dsv : 0.f;
      }
      ds_tile += dsv;
      ga[i] = to16<F16>(F16 ? gg * g16a : gg);
    }
    const int row = 32 * ob + l32;
    *(INFCL_LDS bf16x8*)(gp + gp_chunk_off(row, 2 * kh + h)) = ga;
    return ds_tile;
  };

  // ---- GEMM2: all 64 own rows' G' x this wave's quarter of the tile's
  // features (transposing reads of the segment-blocked tile)
  auto gemm2 = [&](const INFCL_LDS char* cur) {
    int offB[2][FBW], offG[2];
    make_offBG(opaque_lane(), offB, offG);
    auto readB = [&](int g, s16x4 (&bq)[2]) {
      const int s2 = g / FBW;
#pragma unroll
      for (int t = 0; t < 2; ++t)
        bq[t] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (INFCL_LDS s16x4*)(cur + offB[t][g % FBW] + 16 * kSegRow * s2));
    };
    // one group (contraction half s2, feature block fbw) per stage, the
    // transposing reads two stages ahead; stages are separate scheduling
    // regions, which keeps the read-ahead (and the registers) bounded
    bf16x8 A[2];
    s16x4 bq[3][2];
    readB(0, bq[0]);
    readB(1, bq[1]);
#pragma unroll
    for (int g = 0; g < 2 * FBW; ++g) {
      const int s2 = g / FBW, fbw = g % FBW;
      if (fbw == 0) {
#pragma unroll
        for (int o2 = 0; o2 < 2; ++o2)
          A[o2] = *(const INFCL_LDS bf16x8*)(gp + 2048 * o2 + offG[s2]);
      }
      if (g + 2 < 2 * FBW) readB(g + 2, bq[(g + 2) % 3]);
      const s16x4* q = bq[g % 3];
      const s16x8 bb = {q[0][0], q[0][1], q[0][2], q[0][3], q[1][0], q[1][1], q[1][2], q[1][3]};
#pragma unroll
      for (int o2 = 0; o2 < 2; ++o2)
        dacc[o2 * FBW + fbw] = mfma16<F16>(A[o2], __builtin_bit_cast(bf16x8, bb), dacc[o2 * FBW + fbw]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // ---- sweep: tile jt in cur (LSE slot lcur); the DMA of tile jt+1 goes to
  // nxt during GEMM1
  auto body = [&](int jt, const INFCL_LDS char* cur, const INFCL_LDS float* lcur, INFCL_LDS char* nxt,
                  INFCL_LDS float* lnxt) {
    const int dtile = jt + 1 < ntile ? jt + 1 : -1;
    const f32x16 sacc = gemm1(cur, dtile, lnxt);
    ds_acc += (double)join_gp(jt, lcur, sacc, dtile, nxt);
    __syncthreads();  // the G' block is complete
    gemm2(cur);
    wait_dma();
    __syncthreads();  // tile jt+1 landed; cur, the G' block and the join area are free
  };
  {
    const u32x4 rs = tile_rsrc(0);
    const uint32_t lo = dma_lo();
#pragma unroll
    for (int kk = 0; kk < NIW; ++kk) dma16_asm(rs, tA + 1024 * (wave + 4 * kk), lo + sweep_dma_kk_off(kk, wave, ROWG));
    dma16_asm(lse_rsrc(0), lA, lse_lane_off());
  }
  wait_dma();
  __syncthreads();
  // one body with the buffers picked per tile (an unrolled pair of bodies
  // doubles the live ranges and spills at these widths)
  for (int jt = 0; jt < ntile; ++jt) {
    const bool odd = (jt & 1) != 0;
    body(jt, odd ? tB : tA, odd ? lB : lA, odd ? tA : tB, odd ? lA : lB);
  }

  // ---- write dOwn: accumulator dacc[o2 FBW + fbw] lane holds feature l32 of
  // block (wave FBW + fbw), rows 8(r>>2) + 4h + (r&3) of own block o2
  const bool all_ok = wg0 + kWideBM <= p.own_end;
#pragma unroll
  for (int o2 = 0; o2 < 2; ++o2) {
    auto* dst = (typename GO::type*)p.dOwn + (wg0 - p.own_off + 32 * o2 + 4 * h) * D + 32 * (wave * FBW) + l32;
#pragma unroll
    for (int fbw = 0; fbw < FBW; ++fbw)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = wg0 + 32 * o2 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (all_ok || row < p.own_end) dst[(8 * (r >> 2) + (r & 3)) * D + 32 * fbw] = GO::cvt(kfin * dacc[o2 * FBW + fbw][r]);
      }
  }

  // ---- dscale partial of this workgroup: fixed-order reduction
  red[threadIdx.x] = ds_acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) p.ds_part[blockIdx.x] = red[0];
}

// ---------------------------------------------------------------------------
// Pipelined form for d = 768, where three swept tiles fit in LDS (3 x 48 KiB).
// Same quantities and the same per-entry arithmetic as bwd_wide; the work of
// three tiles overlaps in each iteration t, with two barriers per tile:
//   stage 1  GEMM1 of tile t+1 (partial S^T over the wave's feature half),
//            with the G' entries of tile t (joined in the previous stage 2)
//            computed between its MFMAs: exponentials issued among MFMAs of
//            the same wave cost little up to about two per MFMA, where the
//            serial form spends a phase without MFMAs on them;
//            then G' of tile t into the G' block, the partner's half of tile
//            t+1 into the join area, and the DMA of tile t+2.  The DMA sits in
//            this phase without MFMAs on purpose: issued among either stage's
//            MFMAs each 1 KiB instruction cost about 200 cycles (phase trace at
//            d = 768), against about 95 here.  An LDS-DMA instruction holds
//            the issuing wave until the CU's path accepts it, and the MFMAs
//            behind it wait too, even MFMAs that read no LDS;
//   barrier  (G' block of tile t complete, join data of tile t+1 visible)
//   stage 2  GEMM2 of tile t, then the read of the partner's half of tile t+1;
//            wait for the DMA;
//   barrier  (tile t+2 landed; tile t's buffer, the G' block and the join
//            area are free).
// A tile's buffer is written by its DMA in iteration t-2 (after the barrier
// that ends iteration t-3, i.e. after the last reads of the tile three places
// earlier), read by GEMM1 in iteration t-1 and by GEMM2 in iteration t.  The
// swept log-sum-exp values a lane needs for tile t are loaded into registers
// in iteration t-1.
// At d = 1024 three tiles (3 x 64 KiB) do not fit in LDS: bwd_wide serves it.
// It serves d = 768 at every batch size: measured against bwd_wide, 4% faster
// at b = 131072 (192 MiB of swept rows, inside the 256 MiB last-level
// cache) and 1.5-1.6% faster at b = 163840, 262144 and 1048576, where the
// tiles come from HBM.
template <int D, bool F16, bool G16>
__global__ void __launch_bounds__(256, 1) bwd_wide3(BwdParams p) {
  using GO = GradOut<G16, F16>;  // gradient element type
  constexpr int KS = D / 16;
  constexpr int KH = KS / 2;
  constexpr int ROWG = D * 2;
  constexpr int TILEB = kBwdBN * ROWG;
  constexpr int NIW = TILEB / 4096;  // 1 KiB DMA instructions per wave and tile
  constexpr int FBW = D / 128;       // 32-feature blocks of GEMM2 per wave
#ifndef INFCL_W3_PRE
#define INFCL_W3_PRE 8
#endif
  constexpr int kPre = INFCL_W3_PRE;
  constexpr int NG = 2 * FBW;  // GEMM2 groups
  static_assert(KH % 8 == 0 && KH >= 8, "feature halves start on a 128-feature segment");
  static_assert(3 * TILEB + kWideBM * kBwdBN * 2 + 4 * 64 * 8 * 4 <= 160 * 1024, "LDS budget");
  __shared__ __attribute__((aligned(1024))) char tiles_[3 * TILEB];
  __shared__ __attribute__((aligned(1024))) char gp_[kWideBM * kBwdBN * 2];
  __shared__ __attribute__((aligned(16))) float xs_[4][64][8];
  INFCL_LDS char* const tiles = (INFCL_LDS char*)tiles_;
  INFCL_LDS char* const gp = (INFCL_LDS char*)gp_;

  const int lane = __lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ob = wave >> 1, kh = wave & 1;
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t b = p.b;
  const int64_t wg0 = p.own_off + (int64_t)blockIdx.x * kWideBM;
  const int64_t own0 = wg0 + 32 * ob;
  const int64_t iown = own0 + l32;
  const bool own_ok = iown < p.own_end;
  const int64_t irow = own_ok ? iown : p.own_end - 1;
  const bool wave_rows_ok = own0 + 32 <= p.own_end;
  const int ntile = (int)((b + kBwdBN - 1) / kBwdBN);

  const float s = p.scale[0];
  const float k2 = s * kLog2e;
  const float dl = p.dloss ? p.dloss[0] : 1.0f;
  const float g16a = F16 ? p.g16[0] : 1.0f;
  const float kfin = dl * s / (2.0f * (float)b) * (F16 ? p.g16[1] : 1.0f);

  bf16x8 ownf[KH];
  {
    const __bf16* src = (const __bf16*)p.own + irow * D + kh * (D / 2) + 8 * h;
#pragma unroll
    for (int s2 = 0; s2 < KH; ++s2) ownf[s2] = *(const bf16x8*)(src + 16 * s2);
  }
  const float aO = own_ok ? p.lse_own[iown] * kLog2e : 0.f;
  const float uO = own_ok ? p.udiag[iown] : 0.f;
  const float gdiag = own_ok ? expm1f(-p.ell_own[iown]) + expm1f(-p.ell_swept[iown]) : 0.f;

  // Per-lane address parts, computed once: the kernel has registers to spare
  // at d = 768, and rebuilding them per tile costs several hundred VALU
  // cycles in phases without MFMAs.
  const uint32_t dma_lo = sweep_dma_lane_off(lane, wave, ROWG);
  // GEMM1's swept fragments: tile base + kSeg (n >> 3) + offA[n & 7].  The
  // kh = 1 wave loads the tile's rows 16..31 into MFMA rows 0..15 and rows
  // 0..15 into 16..31 (row index XOR 16; the row does not enter the bank of
  // a chunk, so the reads stay conflict free): then accumulator entries 0..7
  // of either wave are the ones it finishes (tile rows 16 kh + 8 h + i) and
  // entries 8..15 the ones it hands over, with no selection by kh.
  int offA[8];
  {
    const int rA = sweep_perm(l32) ^ (16 * kh);
#pragma unroll
    for (int k = 0; k < 8; ++k) offA[k] = sweep_seg_off(rA, 2 * k + h);
  }
  int offB[2][FBW];  // GEMM2's transposing reads: tile base + offB + 16 kSegRow s2
  int offG[2];       // GEMM2's G' fragments of feature step s2
  {
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int fbw = 0; fbw < FBW; ++fbw) offB[tt][fbw] = sweep_tr_off(lane, tt, wave * FBW + fbw);
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) offG[s2] = gp_chunk_off(l32, 2 * s2 + h);
  }
  auto tile_rsrc = [&](int jt) {
    const int64_t j0 = (int64_t)(jt < 0 ? 0 : jt) * kBwdBN;
    return rsrc_words((const char*)p.swept + j0 * ROWG, jt < 0 ? 0 : (b - j0) * ROWG);
  };
  auto tbuf = [&](int t) { return tiles + TILEB * (t % 3); };
  // The fragment addresses of GEMM1 in the buffer stage 1 reads next (pA)
  // and of GEMM2 in the buffer stage 2 reads next (pB), advanced with the
  // buffer rotation before the barrier that ends each iteration, so that no
  // address arithmetic sits between a barrier and the MFMAs after it.
  const INFCL_LDS char* pA[8];
  const INFCL_LDS char* pB[2][FBW];
#pragma unroll
  for (int k = 0; k < 8; ++k) pA[k] = tbuf(0) + kSeg * (kh * KH / 8) + offA[k];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt)
#pragma unroll
    for (int fbw = 0; fbw < FBW; ++fbw) pB[tt][fbw] = tbuf(0) + offB[tt][fbw];
  auto rot = [&](int t) { return TILEB * ((t + 1) % 3 - t % 3); };  // buffer of tile t -> of tile t+1
  auto advance_pA = [&](int t1) {
    const int delta = rot(t1);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      pA[k] += delta;
      asm volatile("" : "+v"(pA[k]));
    }
  };
  auto advance_pB = [&](int t) {
    const int delta = rot(t);
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int fbw = 0; fbw < FBW; ++fbw) {
        pB[tt][fbw] += delta;
        asm volatile("" : "+v"(pB[tt][fbw]));
      }
  };
  // DMA instruction kk of tile jt into its buffer
  auto dma_part = [&](int jt, int kk) {
    dma16_asm(tile_rsrc(jt < ntile ? jt : -1), tbuf(jt) + 1024 * (wave + 4 * kk),
              dma_lo + sweep_dma_kk_off(kk, wave, ROWG));
  };
  auto dma_part_w1 = [&](int jt, int kk) {
    dma16_asm_w1(tile_rsrc(jt < ntile ? jt : -1), tbuf(jt) + 1024 * (wave + 4 * kk),
                 dma_lo + sweep_dma_kk_off(kk, wave, ROWG));
  };
  // The log-sum-exp values of the 8 swept rows 16 kh + 8 h + i of tile jt
  // whose G' entries the lane forms go straight into registers, one tile
  // ahead (range-checked buffer loads: zeros past b).  Through an LDS slot
  // that every wave filled by DMA the backward took 1% longer.
  auto load_L = [&](int jt, f32x4& A, f32x4& B) {
    const int64_t j0 = (int64_t)jt * kBwdBN;
    const bool in = jt < ntile;
    const int64_t rem = in ? (b - j0) * 4 : 0;
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(p.lse2_swept + (in ? j0 : 0)), (short)0, (int)(rem < 128 ? rem : 128), 0x00020000);
    const int vo = 4 * (16 * kh + 8 * h);
    A = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, vo, 0, 0));
    B = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, vo + 16, 0, 0));
  };

  double ds_acc = 0.0;
  f32x16 dacc[2 * FBW];
#pragma unroll
  for (int i = 0; i < 2 * FBW; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dacc[i][r] = 0.f;

  // G' entry of the lane's own row against swept row with base-2 LSE Lj
  auto gp_entry = [&](float x, float Lj, float& ds) {
    const float pO = exp2_hw(__builtin_fmaf(x, k2, -aO));
    const float pS = exp2_hw(__builtin_fmaf(x, k2, -Lj));
    ds = __builtin_fmaf(pO, x - uO, ds);
    return F16 ? (pO + pS) * g16a : pO + pS;
  };

  // ---- stage 1: GEMM1 of tile t1 (partial S^T over this wave's feature
  // half); between its MFMAs, the G' entries of tile t from the joined values
  // x (LSE values L0, L1 read from tile t's slot).  Returns the accumulator
  // of tile t1.
  auto stage1 = [&](const float (&x)[8], const f32x4& L0, const f32x4& L1, float (&gv)[8], float& ds_t,
                    bool with_gp) {
    f32x16 sacc;
    bf16x8 ring[kPre];
#pragma unroll
    for (int i = 0; i < kPre; ++i) ring[i] = *(const INFCL_LDS bf16x8*)(pA[i & 7] + kSeg * (i >> 3));
    __builtin_amdgcn_sched_group_barrier(0x100, kPre, 0);
#pragma unroll
    for (int s2 = 0; s2 < KH; ++s2) {
      mfma16_vgpr<F16, false>(sacc, ring[s2 % kPre], ownf[s2], s2 == 0, s2 == KH - 1);  // unpadded: scan-checked
      if (s2 + kPre < KH) {
        const int n = s2 + kPre;
        ring[s2 % kPre] = *(const INFCL_LDS bf16x8*)(pA[n & 7] + kSeg * (n >> 3));
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      if (with_gp && s2 % 3 == 1) {
        const int i = s2 / 3;  // 8 entries over the 24 MFMAs
        gv[i] = gp_entry(x[i], i < 4 ? L0[i] : L1[i - 4], ds_t);
        // kept here: the compiler would otherwise move part of the entry's
        // arithmetic past the MFMAs, into the phase after them
        asm volatile("" : "+v"(gv[i]), "+v"(ds_t));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    return sacc;
  };

  // ---- stage 2: GEMM2 of tile t (all 64 own rows' G' x this wave's quarter of
  // the tile's features, transposing reads two groups ahead)
  auto stage2 = [&]() {
    auto readB = [&](int g, s16x4 (&bq)[2]) {
      const int s2 = g / FBW;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
        bq[tt] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((INFCL_LDS s16x4*)(pB[tt][g % FBW] + 16 * kSegRow * s2));
    };
    bf16x8 A[2];
    s16x4 bq[3][2];
    readB(0, bq[0]);
    readB(1, bq[1]);
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const int s2 = g / FBW, fbw = g % FBW;
      if (fbw == 0) {
#pragma unroll
        for (int o2 = 0; o2 < 2; ++o2)
          A[o2] = *(const INFCL_LDS bf16x8*)(gp + 2048 * o2 + offG[s2]);
      }
      if (g + 2 < NG) readB(g + 2, bq[(g + 2) % 3]);
      const s16x4* q = bq[g % 3];
      const s16x8 bb = {q[0][0], q[0][1], q[0][2], q[0][3], q[1][0], q[1][1], q[1][2], q[1][3]};
#pragma unroll
      for (int o2 = 0; o2 < 2; ++o2)
        dacc[o2 * FBW + fbw] = mfma16<F16>(A[o2], __builtin_bit_cast(bf16x8, bb), dacc[o2 * FBW + fbw]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // ---- prologue: tiles 0 and 1 in flight, GEMM1 of tile 0, its join
  float x[8];
  {
#pragma unroll
    for (int kk = 0; kk < NIW; ++kk) dma_part(0, kk);
#pragma unroll
    for (int kk = 0; kk < NIW; ++kk) dma_part(1, kk);
    wait_dma();
    __syncthreads();
    float gv0[8], ds0 = 0.f;
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    float x0[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    const f32x16 sacc = stage1(x0, z, z, gv0, ds0, false);
    advance_pA(0);
    float mine[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) mine[i] = sacc[i];
    *(INFCL_LDS f32x4*)&xs_[wave][lane][0] = f32x4{sacc[8], sacc[9], sacc[10], sacc[11]};
    *(INFCL_LDS f32x4*)&xs_[wave][lane][4] = f32x4{sacc[12], sacc[13], sacc[14], sacc[15]};
    __syncthreads();
    const f32x4 q0 = *(const INFCL_LDS f32x4*)&xs_[wave ^ 1][lane][0];
    const f32x4 q1 = *(const INFCL_LDS f32x4*)&xs_[wave ^ 1][lane][4];
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = mine[i] + (i < 4 ? q0[i] : q1[i - 4]);
    __syncthreads();
  }

  f32x4 Lc0, Lc1, Ln0, Ln1;  // log-sum-exp values of tiles t and t+1
  load_L(0, Lc0, Lc1);
  for (int t = 0; t < ntile; ++t) {
    load_L(t + 1, Ln0, Ln1);
    // ---- stage 1
    float mine[8];
    {
      const f32x4 L0 = Lc0, L1 = Lc1;
      float gv[8], ds_t = 0.f;
      const f32x16 sacc = stage1(x, L0, L1, gv, ds_t, true);
      const int64_t j0 = (int64_t)t * kBwdBN;
      if ((j0 == own0) || (j0 + kBwdBN > b) || !wave_rows_ok) {
        // tile on the diagonal or past the ragged end: masked entries
        ds_t = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int64_t j = j0 + 16 * kh + 8 * h + i;
          const float Lj = i < 4 ? L0[i] : L1[i - 4];
          float dsv = 0.f;
          float gg = gp_entry(x[i], Lj, dsv);
          const bool ok = (bool)(own_ok & (j < b));
          const bool dg = j == iown;
          gg = dg ? gdiag * (F16 ? g16a : 1.0f) : (ok ? gg : 0.f);
          ds_t += (ok & !dg) ? dsv : 0.f;
          gv[i] = gg;
        }
      }
      ds_acc += (double)ds_t;
      bf16x8 ga;
#pragma unroll
      for (int i = 0; i < 8; ++i) ga[i] = to16<F16>(gv[i]);
      const int row = 32 * ob + l32;
      *(INFCL_LDS bf16x8*)(gp + gp_chunk_off(row, 2 * kh + h)) = ga;
#pragma unroll
      for (int i = 0; i < 8; ++i) mine[i] = sacc[i];
      *(INFCL_LDS f32x4*)&xs_[wave][lane][0] = f32x4{sacc[8], sacc[9], sacc[10], sacc[11]};
      *(INFCL_LDS f32x4*)&xs_[wave][lane][4] = f32x4{sacc[12], sacc[13], sacc[14], sacc[15]};
#pragma unroll
      for (int kk = 0; kk < NIW; ++kk) dma_part_w1(t + 2, kk);
    }
    __syncthreads();  // G' block of tile t complete; join data of tile t+1 visible
    // ---- stage 2
    stage2();
    {
      const f32x4 q0 = *(const INFCL_LDS f32x4*)&xs_[wave ^ 1][lane][0];
      const f32x4 q1 = *(const INFCL_LDS f32x4*)&xs_[wave ^ 1][lane][4];
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = mine[i] + (i < 4 ? q0[i] : q1[i - 4]);
    }
    advance_pA(t + 1);
    advance_pB(t);
    wait_dma();
    __syncthreads();  // tile t+2 landed; tile t's buffer, the G' block and the join area are free
    Lc0 = Ln0;
    Lc1 = Ln1;
  }

  // ---- write dOwn (as bwd_wide)
  const bool all_ok = wg0 + kWideBM <= p.own_end;
#pragma unroll
  for (int o2 = 0; o2 < 2; ++o2) {
    auto* dst = (typename GO::type*)p.dOwn + (wg0 - p.own_off + 32 * o2 + 4 * h) * D + 32 * (wave * FBW) + l32;
#pragma unroll
    for (int fbw = 0; fbw < FBW; ++fbw)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = wg0 + 32 * o2 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (all_ok || row < p.own_end) dst[(8 * (r >> 2) + (r & 3)) * D + 32 * fbw] = GO::cvt(kfin * dacc[o2 * FBW + fbw][r]);
      }
  }

  // ---- dscale partial: fixed-order reduction in the (now free) join area
  double* red = (double*)&xs_[0][0][0];
  red[threadIdx.x] = ds_acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) p.ds_part[blockIdx.x] = red[0];
}

bool bwd_wide_supported(int64_t d, int dtype) { return (dtype == 0 || dtype == 2) && (d == 768 || d == 1024); }

int bwd_wide_workgroups(int64_t nown) { return (int)((nown + kWideBM - 1) / kWideBM); }

int launch_bwd_wide(const BwdParams& p, int nwg, bool f16, hipStream_t stream) {
  auto go = [&](auto f16c, auto g16c) {
    constexpr bool F = decltype(f16c)::value, G = decltype(g16c)::value;
    if (p.d == 768)
      hipLaunchKernelGGL((bwd_wide3<768, F, G>), dim3(nwg), dim3(256), 0, stream, p);
    else
      hipLaunchKernelGGL((bwd_wide<1024, F, G>), dim3(nwg), dim3(256), 0, stream, p);
    return hipGetLastError() == hipSuccess ? 0 : 1;
  };
  using T = std::true_type;
  using N = std::false_type;
  if (p.d != 768 && p.d != 1024) return 2;
  if (f16) return p.gdt ? go(T{}, T{}) : go(T{}, N{});
  return p.gdt ? go(N{}, T{}) : go(N{}, N{});
}

}  // namespace infcl
