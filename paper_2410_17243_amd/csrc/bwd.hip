// Backward sweeps of the tiled symmetric InfoNCE loss (gfx950).
//
// What is computed (paper Sec. 3.1, Eq. 6-8, completed for both halves of the
// symmetric loss, the text side and the scale; the appendix's in-GPU backward
// algorithm recomputes every tile from the saved log-sum-exp vectors):
//   dL/dx_ij = (1/2b) (P^r_ij + P^c_ij) - (1/b) delta_ij,
//   P^r_ij = exp(x_ij - r_i),  P^c_ij = exp(x_ij - c_j),
//   dimg = k * G' txt,   dtxt = k * G'^T img,
//   with G' = P^r + P^c off the diagonal, G'_ii = expm1(-(r_i-x_ii)) + expm1(-(c_i-x_ii)),
//   k = dloss * s / (2b), and
//   ds = dloss/(2b) * sum_{i != j} [P^r_ij (u_ij - u_ii) + P^c_ij (u_ij - u_jj)],  u = <img_i, txt_j>.
//
// Design (differs from the paper's single pass that read-modify-writes the text
// gradient tile in HBM for every tile): one kernel template, launched twice.
// The launch that "owns" the image rows keeps dimg rows in registers and sweeps
// all text rows; the second launch swaps the roles.  The similarity tile is
// recomputed in each launch, but no gradient leaves the registers before the
// sweep ends and no atomics are used.  A workgroup owns 128 rows (32 per wave)
// and sweeps 32-row tiles of the other side.  Per tile and wave:
//   GEMM1  S^T(32 swept x 32 own) = swept_tile * own^T   (own operand held in
//          registers for the whole sweep, swept rows read from LDS with a
//          row permutation that makes the accumulator usable as GEMM2's operand)
//   G'     two exp2 per entry (log2 domain), the diagonal from expm1 terms
//   GEMM2  16-bit inputs: the four waves' G' blocks are exchanged through LDS and each
//          wave multiplies all 128 own rows by its quarter of the features;
//          fp32: each wave multiplies its own 32 rows by all features.
// Feature widths whose accumulators do not fit the register file are split in
// passes; each pass recomputes GEMM1.
//
// Memory pipeline.  Tiles arrive by LDS DMA (buffer loads that write LDS).
// Each tile buffer, its log-sum-exp slot and the G' buffers are separate LDS
// objects and the tile loop is unrolled over the buffer rotation, so every
// LDS address is tied to one object at compile time: the compiler can then
// see that the reads of the current tiles never alias the DMA in flight and
// does not stall them on it.  The DMA instructions of the next tile are
// spread over the MFMAs of GEMM1 (a burst fills the address queue and stalls
// every wave at issue).
#include <type_traits>

#include "bwd.hpp"

namespace infcl {

constexpr int kBwdBM = 128;  // own rows per workgroup (32 per wave)
constexpr int kGpBytes = kBwdBM * kBwdBN * 2;  // one 16-bit G' exchange buffer

// LDS read-ahead (steps) of GEMM1 (build-time tuning knob).
#ifndef INFCL_BWD_G1_PRE
#define INFCL_BWD_G1_PRE 4
#endif

template <typename TIN, int D, int FB, bool PIPE, bool G16>
__global__ void __launch_bounds__(256, 1) bwd_sweep(BwdParams p) {
  constexpr int ES = sizeof(TIN);
  constexpr bool F16 = std::is_same<TIN, _Float16>::value;  // fp16 (else bf16) when ES == 2
  static_assert(ES == 2 || !G16, "16-bit gradients come with 16-bit inputs");
  using GO = GradOut<G16, F16>;  // gradient element type
  constexpr int KS = D / 16;            // 16-wide contraction steps of GEMM1
  constexpr int ROWG = D * ES;          // bytes per row in HBM
  constexpr int TILEB = kBwdBN * ROWG;  // bytes per swept tile
  constexpr int NIW = TILEB / 4096;     // 1 KiB DMA instructions per wave and tile
  constexpr int FBW = ES == 2 ? FB / 4 : FB;  // 32-feature blocks per wave and pass
  constexpr int NACC = ES == 2 ? 4 * FBW : FB;
  constexpr int NPASS = D / (32 * FB);
  constexpr int GPN = ES == 2 ? (PIPE ? 2 : 1) : 0;  // G' exchange buffers
  static_assert(!PIPE || ES == 2, "the pipelined schedule is for 16-bit inputs only");
  static_assert(D % (32 * FB) == 0, "pass width must divide d");
  static_assert(ES == 4 || FB % 4 == 0, "16-bit pass width is a multiple of 128 features");
  static_assert(D % 64 == 0 && KS % NIW == 0, "tile DMA layout");
  static_assert((PIPE ? 3 : 2) * TILEB + 3 * 1024 + GPN * kGpBytes + 2048 <= 160 * 1024, "LDS budget");
  __shared__ __attribute__((aligned(1024))) char tA_[TILEB];
  __shared__ __attribute__((aligned(1024))) char tB_[TILEB];
  __shared__ __attribute__((aligned(1024))) char tC_[PIPE ? TILEB : 16];
  // log-sum-exp slots: 32 values used; the rest of the 1 KiB catches the zeros
  // that the other lanes of the (branch-free) slot DMA write
  __shared__ __attribute__((aligned(1024))) float lA_[256];
  __shared__ __attribute__((aligned(1024))) float lB_[256];
  __shared__ __attribute__((aligned(1024))) float lC_[256];
  __shared__ __attribute__((aligned(1024))) char gp_[GPN ? GPN * kGpBytes : 16];
  __shared__ double red[256];
  INFCL_LDS char* const tA = (INFCL_LDS char*)tA_;
  INFCL_LDS char* const tB = (INFCL_LDS char*)tB_;
  INFCL_LDS char* const tC = (INFCL_LDS char*)tC_;
  INFCL_LDS float* const lA = (INFCL_LDS float*)lA_;
  INFCL_LDS float* const lB = (INFCL_LDS float*)lB_;
  INFCL_LDS float* const lC = (INFCL_LDS float*)lC_;
  INFCL_LDS char* const gp = (INFCL_LDS char*)gp_;

  const int lane = __lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform (SGPR)
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t b = p.b;
  const int64_t wg0 = p.own_off + (int64_t)blockIdx.x * kBwdBM;  // own_off is a multiple of 32
  const int64_t own0 = wg0 + 32 * wave;                            // this wave's first own row
  const int64_t iown = own0 + l32;                                 // this lane's own row
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

  // own operand of GEMM1, held for the whole sweep: row irow, slots 8h..8h+7 of each step
  typedef typename std::conditional<ES == 2, bf16x8, f32x4>::type frag_t;
  constexpr int FR = ES == 2 ? 1 : 2;  // 16-byte loads per step and lane
  frag_t ownf[KS][FR];
  {
    const char* src = (const char*)p.own + (irow * D) * ES;
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2)
#pragma unroll
      for (int u = 0; u < FR; ++u) ownf[s2][u] = *(const frag_t*)(src + (16 * s2 + 8 * h) * ES + 16 * u);
  }
  const float aO = own_ok ? p.lse_own[iown] * kLog2e : 0.f;
  const float uO = own_ok ? p.udiag[iown] : 0.f;
  const float gdiag = own_ok ? expm1f(-p.ell_own[iown]) + expm1f(-p.ell_swept[iown]) : 0.f;

  auto opaque_lane = [&]() {
    int lo = lane;
    asm volatile("" : "+v"(lo));
    return lo;
  };

  // ---- DMA of swept tile jt into the segment-blocked layout of dst.
  // Instruction k = wave + 4 kk fills LDS bytes [1024 k, 1024 k + 1024): segment
  // k >> 3, rows 4 (k & 7) .. +3; lane L fills row 4 (k & 7) + (L >> 4), physical
  // chunk L & 15, i.e. logical chunk (L & 15) ^ g(row).  Since g(row) =
  // 4 (L >> 4) + (k & 3) and k & 3 = wave, the per-lane part of every source
  // offset is one constant and the rest is wave-uniform.  The DMA lane offsets
  // are rebuilt from an opaque lane id at each use: all 512 registers are in
  // use at d = 512, a value held across the loop would be spilled, and a
  // scratch reload waits for all DMA in flight.  Rows past b fall outside the
  // resource and load as zeros (their G' is masked); jt < 0 loads zeros only.
  auto dma_lane_off = [&]() { return sweep_dma_lane_off(opaque_lane(), wave, ROWG); };
  auto dma_kk_off = [&](int kk) { return sweep_dma_kk_off(kk, wave, ROWG); };
  auto tile_rsrc = [&](int jt) {
    const int64_t j0 = (int64_t)(jt < 0 ? 0 : jt) * kBwdBN;
    return rsrc_words((const char*)p.swept + j0 * ROWG, jt < 0 ? 0 : (b - j0) * ROWG);
  };
  auto lse_rsrc = [&](int jt) {
    const int64_t j0 = (int64_t)(jt < 0 ? 0 : jt) * kBwdBN;
    return rsrc_words(p.lse2_swept + j0, jt < 0 ? 0 : (b - j0) * 4);
  };
  // The log-sum-exp slot of a tile is loaded by every wave with the full wave
  // (no divergent branch in the middle of GEMM1): lanes 8k..8k+7 all fetch the
  // tile's 32 values, so the 1 KiB slot holds 8 copies (the first is read).
  // All waves write the same bytes.
  auto lse_lane_off = [&]() { return 16u * (uint32_t)(opaque_lane() & 7); };
  auto issue_tile = [&](int jt, INFCL_LDS char* dst, INFCL_LDS float* ldst) {
    const u32x4 rs = tile_rsrc(jt);
    const uint32_t lo = dma_lane_off();
#pragma unroll
    for (int kk = 0; kk < NIW; ++kk) dma16_asm(rs, dst + 1024 * (wave + 4 * kk), lo + dma_kk_off(kk));
    dma16_asm(lse_rsrc(jt), ldst, lse_lane_off());
  };

  // ---- per-lane LDS offsets of GEMM1's swept fragments; every read is one
  // of these plus an immediate
  auto make_offA = [&](int lo, int (&offA)[8]) {
    const int l32o = lo & 31, ho = lo >> 5;
    const int rA = sweep_perm(l32o);
#pragma unroll
    for (int k = 0; k < 8; ++k) offA[k] = sweep_seg_off(rA, ES == 2 ? (2 * k + ho) : (4 * (k >> 1) + 2 * ho + (k & 1)));
  };

  double ds_acc = 0.0;

  // ---- GEMM1 of the tile in cur: S^T block, MFMA row m <-> swept row perm(m).
  // LDS fragments are read kPre steps ahead of their MFMA through a register
  // ring.  With with_dma, the loads of tile dtile into (ddst, dlse) are issued
  // between the MFMAs, one 1 KiB instruction per KS / NIW steps.
  // 16-bit inputs: GEMM1's fragment offsets are computed once and held in
  // registers (rebuilt per tile they cost about 2.5% of the backward at
  // d = 512; the fp32 form has no registers to spare and rebuilds them)
  constexpr bool HA = ES == 2;
  int offA_h[8];
  if constexpr (HA) make_offA(lane, offA_h);
  auto gemm1 = [&](const INFCL_LDS char* cur, bool with_dma, int dtile, INFCL_LDS char* ddst,
                   INFCL_LDS float* dlse) {
    int offA[8];
    if constexpr (HA) {
#pragma unroll
      for (int k = 0; k < 8; ++k) offA[k] = offA_h[k];
    } else {
      make_offA(opaque_lane(), offA);
    }
    u32x4 drs = tile_rsrc(-1), drl = lse_rsrc(-1);
    uint32_t dlo = 0;
    if (with_dma) {
      drs = tile_rsrc(dtile);
      drl = lse_rsrc(dtile);
      dlo = dma_lane_off();
    }
    auto dma_step = [&](int s2) {
      if (!with_dma) return;
      constexpr int SPI = KS / NIW;  // steps per DMA instruction
      if ((s2 + 1) % SPI == 0) {
        const int kk = (s2 + 1) / SPI - 1;
        dma16_asm(drs, ddst + 1024 * (wave + 4 * kk), dlo + dma_kk_off(kk));
      }
      if (s2 == (KS > 1 ? 1 : 0)) dma16_asm(drl, dlse, lse_lane_off());
    };
    f32x16 sacc;
    if constexpr (ES == 2) {
      constexpr int kPre = KS < INFCL_BWD_G1_PRE ? KS : INFCL_BWD_G1_PRE;
      bf16x8 ring[kPre];
#pragma unroll
      for (int i = 0; i < kPre; ++i) ring[i] = *(const INFCL_LDS bf16x8*)(cur + offA[i & 7] + kSeg * (i >> 3));
      __builtin_amdgcn_sched_group_barrier(0x100, kPre, 0);
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2) {
        // one pass: no leading padding (its sources are LDS loads and the own
        // rows, never restored just before; the build's scan checks it)
        mfma16_vgpr<F16, (NPASS > 1)>(sacc, ring[s2 % kPre], ownf[s2][0], s2 == 0, s2 == KS - 1);
        dma_step(s2);
        if (s2 + kPre < KS) {
          const int n = s2 + kPre;
          ring[s2 % kPre] = *(const INFCL_LDS bf16x8*)(cur + offA[n & 7] + kSeg * (n >> 3));
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
      }
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[r] = 0.f;
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2) {
        const int kb = 2 * (s2 & 3);
        f32x4 a0 = *(const INFCL_LDS f32x4*)(cur + offA[kb] + kSeg * (s2 >> 2));
        f32x4 a1 = *(const INFCL_LDS f32x4*)(cur + offA[kb + 1] + kSeg * (s2 >> 2));
#pragma unroll
        for (int t = 0; t < 4; ++t) sacc = mfma_f32(a0[t], ownf[s2][0][t], sacc);
#pragma unroll
        for (int t = 0; t < 4; ++t) sacc = mfma_f32(a1[t], ownf[s2][1][t], sacc);
        dma_step(s2);
      }
    }
    return sacc;
  };

  // ---- G' of swept tile jt from its S^T block (log2 domain); entry r <->
  // swept row j = 16 (r>>3) + 8h + (r&7) of the tile.  Returns the dscale
  // contribution.  Tiles touching the diagonal or the ragged end take the
  // masked path (uniform branch).
  auto tile_special = [&](int jt) {
    const int64_t j0 = (int64_t)jt * kBwdBN;
    return (j0 == own0) || (j0 + kBwdBN > b) || !wave_rows_ok;
  };
  auto epilogue = [&](int jt, const INFCL_LDS float* lsep, const f32x16& sacc, float (&gv)[16]) -> float {
    const int64_t j0 = (int64_t)jt * kBwdBN;
    float ds_tile = 0.f;
    if (!tile_special(jt)) {
      const INFCL_LDS char* lp = (const INFCL_LDS char*)lsep + 32 * h;
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const f32x4 v = *(const INFCL_LDS f32x4*)(lp + 64 * (q4 >> 1) + 16 * (q4 & 1));
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int r = 4 * q4 + c;
          const float pO = exp2_hw(__builtin_fmaf(sacc[r], k2, -aO));
          const float pS = exp2_hw(__builtin_fmaf(sacc[r], k2, -v[c]));
          gv[r] = pO + pS;
          ds_tile = __builtin_fmaf(pO, sacc[r] - uO, ds_tile);
        }
      }
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t j = j0 + 16 * (r >> 3) + 8 * h + (r & 7);
        const bool jok = j < b;
        const float aSr = p.lse2_swept[jok ? j : b - 1];
        const float pO = exp2_hw(__builtin_fmaf(sacc[r], k2, -aO));
        const float pS = exp2_hw(__builtin_fmaf(sacc[r], k2, -aSr));
        const bool ok = own_ok && jok;
        const bool dg = (j == iown);
        float gg = ok ? pO + pS : 0.f;
        gg = dg ? gdiag : gg;
        gv[r] = gg;
        ds_tile += (ok && !dg) ? pO * (sacc[r] - uO) : 0.f;
      }
    }
    return ds_tile;
  };
  auto to_h16 = [&](const float (&gv)[16], bf16x8 (&ga)[2]) {
#pragma unroll
    for (int r = 0; r < 16; ++r) ga[r >> 3][r & 7] = to16<F16>(F16 ? gv[r] * g16a : gv[r]);
  };

  // G' exchange buffer (the input's 16-bit type): [128 own rows][32 swept rows], 64-byte rows whose
  // four 16-byte chunks are XOR-swizzled by (row >> 2) & 3.
  auto put_gp = [&](INFCL_LDS char* gpb, const bf16x8 (&ga)[2]) {
    const int lo = opaque_lane();
    const int row = 32 * wave + (lo & 31);
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
      *(INFCL_LDS bf16x8*)(gpb + gp_chunk_off(row, 2 * s2 + (lo >> 5))) = ga[s2];
  };

  // GEMM2's per-lane offsets, computed once where the sweep makes one pass
  // (its feature blocks are then fixed): another 2.5% at d = 512
  constexpr bool HB = ES == 2 && NPASS == 1;
  int offBh[2][FBW], offGh[2];
  if constexpr (HB) {
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int fbw = 0; fbw < FBW; ++fbw) offBh[t][fbw] = sweep_tr_off(lane, t, wave * FBW + fbw);
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) offGh[s2] = gp_chunk_off(l32, 2 * s2 + h);
  }
  for (int pass = 0; pass < NPASS; ++pass) {
    // 16-bit: dacc[ob * FBW + fbw] holds own block ob (rows 32 ob .. of the
    // workgroup) x feature block (pass FB + wave FBW + fbw).
    // fp32: dacc[fb] holds this wave's own rows x feature block (pass FB + fb).
    f32x16 dacc[NACC];
#pragma unroll
    for (int i = 0; i < NACC; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) dacc[i][r] = 0.f;

    // ---- 16-bit GEMM2 of the tile in cur with the G' in gpb, as an explicit
    // software pipeline over its 2 FBW groups (contraction half s2, feature
    // block fbw; 4 MFMAs each, one per own block): stage g issues the LDS reads
    // of group g + 2 and then the MFMAs of group g.  With epi the stages also
    // compute the G' of the next tile (sacc, log-sum-exp values in lnext), a
    // share per stage, into ga.  The stages are separate scheduling regions.
    auto gemm2_staged = [&](bool epi, const INFCL_LDS char* cur, const INFCL_LDS char* gpb,
                            const INFCL_LDS float* lnext, const f32x16& sacc, bf16x8 (&ga)[2]) -> float {
      constexpr int NG = 2 * FBW;
      constexpr int PD = 2;
      constexpr int EPS = (16 + NG - 1) / NG;  // G' entries per stage
      constexpr int NL = EPS > 2 ? 4 : 2;      // live log-sum-exp blocks
      const int lo = opaque_lane();
      const int ho = lo >> 5;
      const INFCL_LDS char* lp = (const INFCL_LDS char*)lnext + 32 * ho;
      auto readL = [&](int q4) { return *(const INFCL_LDS f32x4*)(lp + 64 * (q4 >> 1) + 16 * (q4 & 1)); };
      auto first_stage = [](int q) { return (4 * q) / EPS; };  // first stage using LSE block q
      auto readA = [&](int s2, bf16x8 (&A)[4]) {
#pragma unroll
        for (int ob = 0; ob < 4; ++ob)
          A[ob] = *(const INFCL_LDS bf16x8*)(gpb + 2048 * ob + (HB ? offGh[s2] : gp_chunk_off(lo & 31, 2 * s2 + ho)));
      };
      auto readB = [&](int g, s16x4 (&bq)[2]) {
        const int s2 = g / FBW, fbw = g % FBW;
        const int fbabs = pass * FB + wave * FBW + fbw;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int off = HB ? offBh[t][fbw] + 16 * s2 * kSegRow
                             : sweep_tr_off(lo, t, fbabs) + 16 * kSegRow * s2;
          bq[t] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((INFCL_LDS s16x4*)(cur + off));
        }
      };
      // A holds G' of contraction half 0 until the last stage of that half has
      // issued its MFMAs, then half 1 (read straight after).
      bf16x8 A[4];
      s16x4 Bq[PD + 1][2];
      f32x4 Lq[NL];
      readA(0, A);
      if (epi) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (first_stage(q) == 0) Lq[q % NL] = readL(q);
      }
#pragma unroll
      for (int g = 0; g < PD && g < NG; ++g) readB(g, Bq[g]);
      __builtin_amdgcn_sched_barrier(0);
      float ds_tile = 0.f;
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        if (g + PD < NG) readB(g + PD, Bq[(g + PD) % (PD + 1)]);
        if (epi) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (first_stage(q) == g + 1) Lq[q % NL] = readL(q);
#pragma unroll
          for (int i = 0; i < EPS; ++i) {
            const int r = g * EPS + i;
            if (r < 16) {
              const float x = sacc[r];
              const float pO = exp2_hw(__builtin_fmaf(x, k2, -aO));
              const float pS = exp2_hw(__builtin_fmaf(x, k2, -Lq[(r >> 2) % NL][r & 3]));
              ga[r >> 3][r & 7] = to16<F16>(F16 ? (pO + pS) * g16a : pO + pS);
              ds_tile = __builtin_fmaf(pO, x - uO, ds_tile);
            }
          }
        }
        const int fbw = g % FBW;
        const s16x4* bq = Bq[g % (PD + 1)];
        const s16x8 bb = {bq[0][0], bq[0][1], bq[0][2], bq[0][3], bq[1][0], bq[1][1], bq[1][2], bq[1][3]};
#pragma unroll
        for (int ob = 0; ob < 4; ++ob)
          dacc[ob * FBW + fbw] = mfma16<F16>(A[ob], __builtin_bit_cast(bf16x8, bb), dacc[ob * FBW + fbw]);
        if (g == FBW - 1) readA(1, A);
        __builtin_amdgcn_sched_barrier(0);
      }
      return ds_tile;
    };

    // ---- fp32 GEMM2: this wave's own rows x all the pass's features; step r
    // contracts swept row jr(r, h) of each lane half.
    auto gemm2_f32 = [&](const INFCL_LDS char* cur, const float (&gv)[16]) {
#pragma unroll
      for (int fb = 0; fb < FB; ++fb) {
        const int fbabs = pass * FB + fb;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = sweep_perm(8 * (r >> 2) + 4 * h + (r & 3));
          const int cf = 8 * fbabs + (l32 >> 2);
          float bv = *(const INFCL_LDS float*)(cur + sweep_chunk_off(j, cf) + (l32 & 3) * 4);
          dacc[fb] = mfma_f32(gv[r], bv, dacc[fb]);
        }
      }
    };

    if constexpr (PIPE) {
      // Software pipeline over tiles: iteration jt runs GEMM1 of tile jt+1
      // (issuing the loads of tile jt+2), then GEMM2 of tile jt together with
      // the G' of tile jt+1.  Three tile buffers rotate; G' buffers alternate.
      // Past the last tile, GEMM1 runs on a stale buffer and the G' step takes
      // the masked path (tile rows >= b), so it yields zeros.
      issue_tile(0, tA, lA);
      issue_tile(ntile > 1 ? 1 : -1, tB, lB);
      wait_dma();
      __syncthreads();
      {
        const f32x16 sacc = gemm1(tA, false, -1, tC, lC);
        float gv[16];
        const float d0 = epilogue(0, lA, sacc, gv);
        if (pass == 0) ds_acc += (double)d0;
        bf16x8 ga[2];
        to_h16(gv, ga);
        put_gp(gp, ga);
      }
      __syncthreads();
      auto body = [&](int jt, const INFCL_LDS char* cur, INFCL_LDS char* nxt, const INFCL_LDS float* lnxt,
                      INFCL_LDS char* fre, INFCL_LDS float* lfre) {
        const bool next = jt + 1 < ntile;
        const f32x16 sacc = gemm1(nxt, true, jt + 2 < ntile ? jt + 2 : -1, fre, lfre);
        __builtin_amdgcn_sched_barrier(0);
        bf16x8 ga[2];
        float dn = gemm2_staged(true, cur, gp + (jt & 1) * kGpBytes, lnxt, sacc, ga);
        // pin the unmasked G' here: otherwise it is sunk into the not-special
        // branch below and computed after GEMM2 instead of alongside it
        asm volatile("" : "+v"(ga[0]), "+v"(ga[1]), "+v"(dn));
        __builtin_amdgcn_sched_barrier(0);
        if (tile_special(jt + 1)) {
          float gv[16];
          dn = epilogue(jt + 1, lnxt, sacc, gv);
          to_h16(gv, ga);
        }
        if (pass == 0 && next) ds_acc += (double)dn;
        put_gp(gp + ((jt + 1) & 1) * kGpBytes, ga);
        wait_dma();
        __syncthreads();
      };
      // Unrolled over the buffer rotation without tests in between: a tile
      // index past the end is a tile of rows past b, fully masked (zero G').
      for (int jt = 0; jt < ntile; jt += 3) {
        body(jt, tA, tB, lB, tC, lC);
        body(jt + 1, tB, tC, lC, tA, lA);
        body(jt + 2, tC, tA, lA, tB, lB);
      }
    } else {
      // Two tile buffers: GEMM1 of tile jt (issuing the loads of tile jt+1),
      // G', GEMM2.
      issue_tile(0, tA, lA);
      wait_dma();
      __syncthreads();
      auto body = [&](int jt, const INFCL_LDS char* cur, const INFCL_LDS float* lcur, INFCL_LDS char* nxt,
                      INFCL_LDS float* lnxt) {
        const f32x16 sacc = gemm1(cur, true, jt + 1 < ntile ? jt + 1 : -1, nxt, lnxt);
        float gv[16];
        const float d0 = epilogue(jt, lcur, sacc, gv);
        if (pass == 0) ds_acc += (double)d0;
        if constexpr (ES == 2) {
          bf16x8 ga[2];
          to_h16(gv, ga);
          put_gp(gp, ga);
          __syncthreads();
          gemm2_staged(false, cur, gp, lcur, sacc, ga);
        } else {
          gemm2_f32(cur, gv);
        }
        wait_dma();
        __syncthreads();
      };
      // Unrolled over the buffer pair without a test in between: a tile
      // index past the end is a tile of rows past b, fully masked (zero G').
      for (int jt = 0; jt < ntile; jt += 2) {
        body(jt, tA, lA, tB, lB);
        body(jt + 1, tB, lB, tA, lA);
      }
    }

    // ---- write dOwn: lane holds feature l32 of a 32-feature block, rows 8(r>>2)+4h+(r&3)
    if constexpr (ES == 2) {
      const bool all_ok = wg0 + kBwdBM <= p.own_end;
#pragma unroll
      for (int ob = 0; ob < 4; ++ob) {
        auto* dst = (typename GO::type*)p.dOwn + (wg0 - p.own_off + 32 * ob + 4 * h) * D + 32 * (pass * FB + wave * FBW) + l32;
#pragma unroll
        for (int fbw = 0; fbw < FBW; ++fbw)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int64_t row = wg0 + 32 * ob + 8 * (r >> 2) + 4 * h + (r & 3);
            if (all_ok || row < p.own_end) dst[(8 * (r >> 2) + (r & 3)) * D + 32 * fbw] = GO::cvt(kfin * dacc[ob * FBW + fbw][r]);
          }
      }
    } else {
      auto* dst = (typename GO::type*)p.dOwn + (own0 - p.own_off + 4 * h) * D + 32 * pass * FB + l32;
#pragma unroll
      for (int fb = 0; fb < FB; ++fb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t row = own0 + 8 * (r >> 2) + 4 * h + (r & 3);
          if (wave_rows_ok || row < p.own_end) dst[(8 * (r >> 2) + (r & 3)) * D + 32 * fb] = GO::cvt(kfin * dacc[fb][r]);
        }
    }
    // the next pass reuses the tile buffers
    __syncthreads();
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

// dscale = dloss / (2b) * (sum of both launches' partials), fixed order; into
// dscale (fp32) and/or dscale64 (fp64), whichever is given
__global__ void __launch_bounds__(256) dscale_finish(const double* part, int64_t n, int64_t b, const float* dloss,
                                                     float* dscale, double* dscale64) {
  __shared__ double red[256];
  double s = 0.0;
  for (int64_t k = threadIdx.x; k < n; k += 256) s += part[k];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double dl = dloss ? (double)dloss[0] : 1.0;
    const double v = red[0] * dl / (2.0 * (double)b);
    if (dscale) *dscale = (float)v;
    if (dscale64) *dscale64 = v;
  }
}

// Pass width: largest FB (32-feature blocks) dividing d/32 whose accumulators
// (16 FB registers) fit next to the own operand (d/4 or d/2 registers); for
// 16-bit inputs FB is also a multiple of 4 (see the transposing-read addressing).
// Build-time tuning knobs: the register budget shared by the own operand and
// the gradient accumulators, and whether the three-buffer pipeline is used
// (16-bit widths whose three tiles fit in LDS).
#ifndef INFCL_BWD_REG_BUDGET
#define INFCL_BWD_REG_BUDGET 384
#endif
#ifndef INFCL_BWD_PIPE
#define INFCL_BWD_PIPE 1
#endif

template <typename TIN, int D>
static int launch_bwd_d(const BwdParams& p, int nwg, hipStream_t stream) {
  constexpr int ES = sizeof(TIN);
  constexpr int OWNREGS = D * ES / 8;
  constexpr int NB32 = D / 32;
  constexpr int FBMAX = (INFCL_BWD_REG_BUDGET - OWNREGS) / 16;
  constexpr int FB = [] {
    int best = ES == 4 ? 1 : 4;  // 16-bit: at least one 128-feature group
    for (int f = 1; f <= NB32; ++f)
      if (NB32 % f == 0 && f <= FBMAX && (ES == 4 || f % 4 == 0)) best = f;
    return best;
  }();
  static_assert(ES == 4 || FB % 4 == 0, "16-bit pass width must be a multiple of 128 features");
  constexpr int TILEB = kBwdBN * D * ES;
  constexpr bool PIPE = INFCL_BWD_PIPE != 0 && ES == 2 && 3 * (TILEB + 128) + 2 * kGpBytes + 2048 <= 160 * 1024;
  if constexpr (ES == 2) {
    if (p.gdt) {
      hipLaunchKernelGGL((bwd_sweep<TIN, D, FB, PIPE, true>), dim3(nwg), dim3(256), 0, stream, p);
      return hipGetLastError() == hipSuccess ? 0 : 1;
    }
  }
  hipLaunchKernelGGL((bwd_sweep<TIN, D, FB, PIPE, false>), dim3(nwg), dim3(256), 0, stream, p);
  return hipGetLastError() == hipSuccess ? 0 : 1;
}

template <typename TIN>
static int launch_bwd_t(const BwdParams& p, int nwg, hipStream_t stream) {
  const int64_t d = p.d;
  if constexpr (sizeof(TIN) == 2) {
    switch (d) {
      case 128: return launch_bwd_d<TIN, 128>(p, nwg, stream);
      case 256: return launch_bwd_d<TIN, 256>(p, nwg, stream);
      case 384: return launch_bwd_d<TIN, 384>(p, nwg, stream);
      case 512: return launch_bwd_d<TIN, 512>(p, nwg, stream);
      case 640: return launch_bwd_d<TIN, 640>(p, nwg, stream);
      case 896: return launch_bwd_d<TIN, 896>(p, nwg, stream);
      // 768 and 1024 take the single-pass wide-row sweep
    }
  } else {
    switch (d) {
      case 64: return launch_bwd_d<TIN, 64>(p, nwg, stream);
      case 128: return launch_bwd_d<TIN, 128>(p, nwg, stream);
      case 192: return launch_bwd_d<TIN, 192>(p, nwg, stream);
      case 256: return launch_bwd_d<TIN, 256>(p, nwg, stream);
      case 320: return launch_bwd_d<TIN, 320>(p, nwg, stream);
      case 384: return launch_bwd_d<TIN, 384>(p, nwg, stream);
      case 448: return launch_bwd_d<TIN, 448>(p, nwg, stream);
      case 512: return launch_bwd_d<TIN, 512>(p, nwg, stream);
    }
  }
  return 2;
}

// fp16 inputs: G' is rounded to fp16 after multiplication by a power of two
// alpha, and the fp32 accumulators are multiplied by 1/alpha at the end (exact
// scaling, the role loss scaling plays in mixed-precision training): without
// it the G' of a well-separated batch (loss near zero) lies below fp16's
// smallest subnormal, 2^-24, and the gradients would vanish.  alpha maps a
// bound B on every |G'| to at most 2^14 (fp16's largest finite value is about
// 2^16): off the diagonal P^r_ij <= 1 - P^r_ii = -expm1(-l^r_i) and
// P^c_ij <= -expm1(-l^c_j), and |G'_ii| <= -expm1(-l^r_i) - expm1(-l^c_i), so
// B = max_i(-expm1(-l^r_i)) + max_j(-expm1(-l^c_j)).
// Per-block maxima (fixed-order tree) of the two terms, then alpha.
__global__ void __launch_bounds__(256) g16_bound_part(const float* aux, int64_t b, float* part) {
  __shared__ float sr[256], sc[256];
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  sr[threadIdx.x] = i < b ? -expm1f(-aux[i]) : 0.f;
  sc[threadIdx.x] = i < b ? -expm1f(-aux[b + i]) : 0.f;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) {
      sr[threadIdx.x] = fmaxf(sr[threadIdx.x], sr[threadIdx.x + w]);
      sc[threadIdx.x] = fmaxf(sc[threadIdx.x], sc[threadIdx.x + w]);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = sr[0];
    part[2 * blockIdx.x + 1] = sc[0];
  }
}
__global__ void __launch_bounds__(256) g16_scale_finish(const float* part, int64_t nblk, float* g16) {
  __shared__ float sr[256], sc[256];
  float mr = 0.f, mc = 0.f;
  for (int64_t k = threadIdx.x; k < nblk; k += 256) {
    mr = fmaxf(mr, part[2 * k]);
    mc = fmaxf(mc, part[2 * k + 1]);
  }
  sr[threadIdx.x] = mr;
  sc[threadIdx.x] = mc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) {
      sr[threadIdx.x] = fmaxf(sr[threadIdx.x], sr[threadIdx.x + w]);
      sc[threadIdx.x] = fmaxf(sc[threadIdx.x], sc[threadIdx.x + w]);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const float B = sr[0] + sc[0];
    int k = 0;
    if (B > 0.f) {
      int e;
      (void)frexpf(B, &e);  // B = m 2^e, m in [0.5, 1): alpha B = m 2^14 < 2^14
      k = 14 - e;
      k = k > 100 ? 100 : k;
    }
    g16[0] = ldexpf(1.f, k);
    g16[1] = ldexpf(1.f, -k);
  }
}

// Log-sum-exp vectors rescaled to base 2 (the swept side is streamed through
// LDS next to every tile and used as is).
__global__ void __launch_bounds__(256) lse_to_log2(const float* lse_r, const float* lse_c, float* l2r, float* l2c,
                                                   int64_t b) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < b) {
    l2r[i] = lse_r[i] * kLog2e;
    l2c[i] = lse_c[i] * kLog2e;
  }
}

bool bwd_wide_supported(int64_t d, int dtype);
int bwd_wide_workgroups(int64_t nown);
int launch_bwd_wide(const BwdParams& p, int nwg, bool f16, hipStream_t stream);

// Backward: 16-bit inputs with d = 768 or 1024 take the single-pass wide-row sweep
// (64 own rows per workgroup), everything else the 128-row sweep above.  Own
// rows are [r0, r0 + nrows) of both sides (all b for the whole batch; a
// shard's samples otherwise, with dimg/dtxt [nrows, d]: fp32, or with gdt = 1
// the 16-bit input type); lse_r, lse_c and aux cover all b samples.  dscale
// (fp32) and/or dscale64 (fp64) receive this call's share, dloss/(2b) times its
// partial sums.
int launch_bwd(const void* img, const void* txt, int64_t b, int64_t d, int dtype, int64_t r0, int64_t nrows,
               const float* scale, const float* lse_r, const float* lse_c, const float* aux, const float* dloss,
               void* dimg, void* dtxt, int gdt, float* dscale, double* dscale64, float* lse2, double* ds_part,
               float* g16, hipStream_t stream) {
  const bool wide = bwd_wide_supported(d, dtype);
  const int nwg = wide ? bwd_wide_workgroups(nrows) : (int)((nrows + kBwdBM - 1) / kBwdBM);
  auto launch = [&](const BwdParams& q) {
    if (wide) return launch_bwd_wide(q, nwg, dtype == 2, stream);
    if (dtype == 0) return launch_bwd_t<__bf16>(q, nwg, stream);
    if (dtype == 2) return launch_bwd_t<_Float16>(q, nwg, stream);
    return launch_bwd_t<float>(q, nwg, stream);
  };
  float* l2r = lse2;
  float* l2c = lse2 + b;
  const unsigned nblk = (unsigned)((b + 255) / 256);
  hipLaunchKernelGGL(lse_to_log2, dim3(nblk), dim3(256), 0, stream, lse_r, lse_c, l2r, l2c, b);
  if (hipGetLastError() != hipSuccess) return 1;
  if (dtype == 2) {  // g16 = (alpha, 1/alpha) followed by 2 nblk block maxima
    hipLaunchKernelGGL(g16_bound_part, dim3(nblk), dim3(256), 0, stream, aux, b, g16 + 2);
    hipLaunchKernelGGL(g16_scale_finish, dim3(1), dim3(256), 0, stream, (const float*)(g16 + 2), (int64_t)nblk, g16);
    if (hipGetLastError() != hipSuccess) return 1;
  }
  BwdParams p;
  p.g16 = g16;
  p.b = b;
  p.d = d;
  p.scale = scale;
  p.udiag = aux + 2 * b;
  p.dloss = dloss;
  p.own_off = r0;
  p.own_end = r0 + nrows;
  p.gdt = gdt;
  // launch 1: own = image rows (dimg), swept = text rows
  p.own = img;
  p.swept = txt;
  p.lse_own = lse_r;
  p.lse2_swept = l2c;
  p.ell_own = aux;
  p.ell_swept = aux + b;
  p.dOwn = dimg;
  p.ds_part = ds_part;
  int rc = launch(p);
  if (rc) return rc;
  // launch 2: own = text rows (dtxt), swept = image rows
  p.own = txt;
  p.swept = img;
  p.lse_own = lse_c;
  p.lse2_swept = l2r;
  p.ell_own = aux + b;
  p.ell_swept = aux;
  p.dOwn = dtxt;
  p.ds_part = ds_part + nwg;
  rc = launch(p);
  if (rc) return rc;
  hipLaunchKernelGGL(dscale_finish, dim3(1), dim3(256), 0, stream, (const double*)ds_part, (int64_t)2 * nwg, b,
                     dloss, dscale, dscale64);
  return hipGetLastError() == hipSuccess ? 0 : 1;
}

bool bwd_supported(int64_t d, int dtype) {
  if (dtype == 0 || dtype == 2) return d % 128 == 0 && d >= 128 && d <= 1024;
  return d % 64 == 0 && d >= 64 && d <= 512;
}

}  // namespace infcl
