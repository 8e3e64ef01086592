// Backward sweeps of the tiled symmetric InfoNCE loss (gfx950).
//
// What is computed (paper Sec. 3.1, Eq. 6-8, completed for both halves of the
// symmetric loss, the text side and the scale; the appendix's in-GPU backward
// algorithm recomputes every tile from the saved log-sum-exp vectors):
//   dL/dx_ij = (1/2b) (P^r_ij + P^c_ij) - (1/b) delta_ij,
//   P^r_ij = exp(x_ij - r_i),  P^c_ij = exp(x_ij - c_j),
//   dimg = dloss * s * G img-side = k * G' txt,   dtxt = k * G'^T img,
//   with G' = P^r + P^c off the diagonal, G'_ii = expm1(-(r_i-x_ii)) + expm1(-(c_i-x_ii)),
//   k = dloss * s / (2b), and
//   ds = dloss/(2b) * sum_{i != j} [P^r_ij (u_ij - u_ii) + P^c_ij (u_ij - u_jj)],  u = <img_i, txt_j>.
//
// Design (differs from the paper's single pass that read-modify-writes the text
// gradient tile in HBM for every tile): one kernel template, launched twice.
// The launch that "owns" the image rows keeps dimg rows in registers and sweeps
// all text rows; the second launch swaps the roles (owns text rows, sweeps
// image rows).  The similarity tile is recomputed in each launch, but no
// gradient ever leaves the registers before the sweep ends and no atomics are
// used.  Per tile and wave:
//   GEMM1  S^T(32 swept x 32 own) = swept_tile * own^T   (own operand held in
//          registers for the whole sweep, swept rows read from LDS with a
//          row permutation that makes the accumulator usable as GEMM2's operand)
//   G'     two exp2 per entry (log2 domain), the diagonal from expm1 terms
//   GEMM2  dOwn(32 own x FP features) += G'(bf16) * swept_tile, the swept tile
//          read feature-major through the transposing LDS read.
// Feature widths whose accumulators do not fit the register file are split in
// passes of FP features; each pass recomputes GEMM1.
#include <type_traits>

#include "common.hpp"

namespace infcl {

struct BwdParams {
  const void* own;    // [b, d] rows whose gradient this launch produces
  const void* swept;  // [b, d] the other modality
  int64_t b, d;
  const float* scale;
  const float* lse_own;    // [b]
  const float* lse_swept;  // [b]
  const float* ell_own;    // [b]  r_i - x_ii of the own side
  const float* ell_swept;  // [b]
  const float* udiag;      // [b]  <img_i, txt_i>
  const float* dloss;      // device scalar or nullptr (= 1)
  float* dOwn;             // [b, d]
  double* ds_part;         // [gridDim.x]
};

constexpr int kBwdBM = 128;  // own rows per workgroup (32 per wave)

// LDS read-ahead (steps) of the two products and the number of independent
// accumulation chains of the first one (build-time tuning knobs).
#ifndef INFCL_BWD_G1_PRE
#define INFCL_BWD_G1_PRE 4
#endif
#ifndef INFCL_BWD_G1_CHAINS
#define INFCL_BWD_G1_CHAINS 1
#endif
#ifndef INFCL_BWD_G2_PRE
#define INFCL_BWD_G2_PRE 3
#endif
constexpr int kBwdBN = 32;   // swept rows per tile

// Chunk swizzle for the swept tile (rows of >= 16 chunks): 16 rows reading one
// logical chunk, and the 4 rows x 4 chunks of a transposing read, are both
// spread over all 64 banks.
__device__ __forceinline__ int bwd_g(int r) { return 4 * (r & 3) + ((r >> 2) & 3); }
// GEMM1 row permutation: MFMA row m loads swept row perm(m) (bits 2 and 3
// swapped), so that accumulator register 8s+t of lane half h holds swept row
// 16s + 8h + t -- exactly the contraction slot t of GEMM2 step s.
__device__ __forceinline__ int bwd_perm(int m) { return (m & 0x13) | ((m & 4) << 1) | ((m & 8) >> 1); }

template <typename TIN, int D, int FB, bool PIPE, int RING>
__global__ void __launch_bounds__(256, 1) bwd_sweep(BwdParams p) {
  constexpr int ES = sizeof(TIN);
  constexpr int EPC = 16 / ES;          // elements per 16-byte chunk
  constexpr int KS = D / 16;            // 16-wide contraction steps of GEMM1
  constexpr int CPR = D * ES / 16;      // 16-byte chunks per swept row
  constexpr int ROWB = CPR * 16;        // bytes per swept row in LDS
  constexpr int TILEB = kBwdBN * ROWB;  // bytes per swept tile
  constexpr int NI = TILEB / 1024;      // 1 KiB DMA instructions per tile
  constexpr int NIW = NI / 4;           // ... per wave
  constexpr int FP = 32 * FB;           // features per pass
  constexpr int NPASS = D / FP;
  // three tile buffers (t in GEMM2, t+1 in GEMM1, t+2 loading) when they fit,
  // otherwise two (GEMM1 -> G' -> GEMM2 per tile while the next tile loads)
  // PIPE: three tile buffers (t in GEMM2, t+1 in GEMM1, t+2 loading).
  // Otherwise a ring of RING buffers: GEMM1 -> G' -> GEMM2 per tile while the
  // next RING-1 tiles load (clamped to what fits in LDS).
  constexpr int GPB = ES == 2 ? kBwdBM * kBwdBN * 2 : 0;  // G' exchange buffer bytes
  constexpr int RINGFIT = (160 * 1024 - 2048 - GPB) / (TILEB + 128);
  constexpr int NBUF = PIPE ? 3 : (RING < RINGFIT ? RING : RINGFIT);
  static_assert(NBUF >= 2, "at least two tile buffers");
  static_assert(D % FP == 0, "pass width must divide d");
  static_assert(CPR % 16 == 0 && NI % 4 == 0, "rows must hold a multiple of 16 chunks");
  static_assert(NBUF * (TILEB + 128) + GPB + 2048 <= 160 * 1024, "LDS budget");
  __shared__ __attribute__((aligned(1024))) char lds_[NBUF * TILEB + NBUF * 128 + GPB];
  INFCL_LDS char* lds = (INFCL_LDS char*)lds_;
  INFCL_LDS char* lse_lds = lds + NBUF * TILEB;  // 32 swept log-sum-exp values per buffer

  const int lane = __lane_id();
  const int wave = threadIdx.x >> 6;
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t b = p.b;
  const int64_t own0 = (int64_t)blockIdx.x * kBwdBM + 32 * wave;  // this wave's first own row
  const int64_t iown = own0 + l32;                                // this lane's own row
  const bool own_ok = iown < b;
  const int64_t irow = own_ok ? iown : b - 1;
  const bool wave_rows_ok = own0 + 32 <= b;
  const int ntile = (int)((b + kBwdBN - 1) / kBwdBN);

  const float s = p.scale[0];
  const float k2 = s * kLog2e;
  const float dl = p.dloss ? p.dloss[0] : 1.0f;
  const float kfin = dl * s / (2.0f * (float)b);

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

  // ---- DMA of a swept tile: instruction k = wave + 4 kk writes LDS bytes
  // [1024 k, 1024 k + 1024) of the buffer; lane L fills physical chunk 64 k + L,
  // i.e. row r = (64 k + L) / CPR, physical chunk pc = (64 k + L) % CPR, which
  // holds logical chunk pc ^ g(r).  The per-lane source offsets are recomputed
  // at every issue from an opaque copy of the lane id: hoisted out of the loop
  // they would be spilled, and a scratch reload waits for all in-flight DMA.
  auto issue_tile = [&](int jt, int buf) {
    const int64_t j0 = (int64_t)jt * kBwdBN;
    INFCL_LDS char* dst = lds + buf * TILEB;
    int lo = lane;
    asm volatile("" : "+v"(lo));
    // rows past b fall outside the resource and load as zeros (their G' is masked)
    const __amdgpu_buffer_rsrc_t rs = make_rsrc((const char*)p.swept + j0 * (D * ES), (b - j0) * (D * ES));
#pragma unroll
    for (int kk = 0; kk < NIW; ++kk) {
      const int F = 64 * (wave + 4 * kk) + lo;
      const int r = F / CPR, pc = F % CPR;
      const uint32_t off = (uint32_t)(r * D * ES + (pc ^ bwd_g(r)) * 16);
      dma16b(rs, (INFCL_LDS void*)(dst + 1024 * (wave + 4 * kk)), off, 0);
    }
    if (wave == 0 && lane < 8) {
      const __amdgpu_buffer_rsrc_t rl = make_rsrc(p.lse_swept + j0, (b - j0) * 4);
      dma16b(rl, (INFCL_LDS void*)(lse_lds + 128 * buf), 16u * lo, 0);
    }
  };

  // ---- per-lane LDS offsets; every read below is one of these plus an
  // immediate.  They are rebuilt from an opaque lane id inside every tile
  // iteration (see issue_tile for why nothing lane-dependent may stay live).
  auto make_offA = [&](int lo, int (&offA)[8]) {
    const int l32o = lo & 31, ho = lo >> 5;
    const int rA = bwd_perm(l32o);
    const int gA = bwd_g(rA);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int cl = ES == 2 ? (2 * k + ho) : (4 * (k >> 1) + 2 * ho + (k & 1));
      offA[k] = rA * ROWB + 16 * (cl ^ gA);
    }
  };
  auto make_offT = [&](int lo, int (&offT)[2][4]) {
    const int g4 = lo >> 4, l16 = lo & 15;
    const int e = l16 >> 2, qq = l16 & 3, nb16 = g4 & 1, hh = g4 >> 1;
    const int lb = 2 * nb16 + (qq >> 1);
    const int fo = (qq & 1) * 8;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int fm = 0; fm < 4; ++fm)
        offT[t][fm] = (8 * hh + e) * ROWB + 16 * (4 * (fm ^ e) + (lb ^ ((t + 2 * hh) & 3))) + fo;
  };
  auto opaque_lane = [&]() {
    int lo = lane;
    asm volatile("" : "+v"(lo));
    return lo;
  };

  double ds_acc = 0.0;

  // GEMM1 of swept tile jt (in buffer buf): S^T block, MFMA row m <-> swept row j0 + perm(m).
  // bf16: LDS fragments are read kPre steps ahead of their MFMA through a
  // register ring, and the steps alternate between two accumulators so that
  // consecutive MFMAs are independent; the scheduling groups pin the order
  // MFMA, read, MFMA, read, ...
  auto gemm1 = [&](int buf) {
    const INFCL_LDS char* cur = lds + buf * TILEB;
    int offA[8];
    make_offA(opaque_lane(), offA);
    f32x16 sacc;
    if constexpr (ES == 2) {
      constexpr int kPre = KS < INFCL_BWD_G1_PRE ? KS : INFCL_BWD_G1_PRE;
      constexpr int NCH = INFCL_BWD_G1_CHAINS;
      f32x16 acc2[NCH];
#pragma unroll
      for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc2[c][r] = 0.f;
      bf16x8 ring[kPre];
#pragma unroll
      for (int i = 0; i < kPre; ++i) ring[i] = *(const INFCL_LDS bf16x8*)(cur + offA[i & 7] + 256 * (i >> 3));
      __builtin_amdgcn_sched_group_barrier(0x100, kPre, 0);
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2) {
        const bf16x8 a = ring[s2 % kPre];
        acc2[s2 % NCH] = mfma_bf16(a, ownf[s2][0], acc2[s2 % NCH]);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (s2 + kPre < KS) {
          const int n = s2 + kPre;
          ring[s2 % kPre] = *(const INFCL_LDS bf16x8*)(cur + offA[n & 7] + 256 * (n >> 3));
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v = acc2[0][r];
#pragma unroll
        for (int c = 1; c < NCH; ++c) v += acc2[c][r];
        sacc[r] = v;
      }
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[r] = 0.f;
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2) {
        const int kb = 2 * (s2 & 3);
        f32x4 a0 = *(const INFCL_LDS f32x4*)(cur + offA[kb] + 256 * (s2 >> 2));
        f32x4 a1 = *(const INFCL_LDS f32x4*)(cur + offA[kb + 1] + 256 * (s2 >> 2));
#pragma unroll
        for (int t = 0; t < 4; ++t) sacc = mfma_f32(a0[t], ownf[s2][0][t], sacc);
#pragma unroll
        for (int t = 0; t < 4; ++t) sacc = mfma_f32(a1[t], ownf[s2][1][t], sacc);
      }
    }
    return sacc;
  };

  // G' of swept tile jt from its S^T block (log2 domain); entry r <-> swept row
  // j = j0 + 16 (r>>3) + 8h + (r&7).  Returns the dscale contribution.
  auto epilogue = [&](int jt, int buf, const f32x16& sacc, float (&gv)[16]) -> float {
    const int64_t j0 = (int64_t)jt * kBwdBN;
    float ds_tile = 0.f;
    const bool special = (j0 == own0) || (j0 + kBwdBN > b) || !wave_rows_ok;
    if (!special) {
      float aS[16];
      const INFCL_LDS char* lp = lse_lds + 128 * buf + 32 * (opaque_lane() >> 5);
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const f32x4 v = *(const INFCL_LDS f32x4*)(lp + 64 * (q4 >> 1) + 16 * (q4 & 1));
#pragma unroll
        for (int c = 0; c < 4; ++c) aS[4 * q4 + c] = v[c] * kLog2e;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float pO = exp2_hw(__builtin_fmaf(sacc[r], k2, -aO));
        const float pS = exp2_hw(__builtin_fmaf(sacc[r], k2, -aS[r]));
        gv[r] = pO + pS;
        ds_tile = __builtin_fmaf(pO, sacc[r] - uO, ds_tile);
      }
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t j = j0 + 16 * (r >> 3) + 8 * h + (r & 7);
        const bool jok = j < b;
        const float aSr = p.lse_swept[jok ? j : b - 1] * kLog2e;
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

  // G' exchange buffer (bf16): [128 own rows][32 swept rows], 64-byte rows whose
  // four 16-byte chunks are XOR-swizzled by (row >> 2) & 3.
  constexpr int FBW = ES == 2 ? FB / 4 : FB;  // 32-feature blocks per wave and pass (bf16)
  INFCL_LDS char* gp_lds = lse_lds + NBUF * 128;
  auto gp_off = [](int row, int c) { return row * 64 + 16 * (c ^ ((row >> 2) & 3)); };

  for (int pass = 0; pass < NPASS; ++pass) {
    // bf16: dacc[ob * FBW + fbw] holds own block ob (rows 32 ob .. of the
    // workgroup) x feature block (pass FB + wave FBW + fbw).
    // fp32: dacc[fb] holds this wave's own rows x feature block (pass FB + fb).
    f32x16 dacc[ES == 2 ? 4 * FBW : FB];
#pragma unroll
    for (int i = 0; i < (ES == 2 ? 4 * FBW : FB); ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) dacc[i][r] = 0.f;

    // bf16 GEMM2: every wave multiplies the G' of all four waves (from LDS) by
    // its quarter of the pass's features of the swept tile (transposing reads).
    auto gemm2_bf16 = [&](int buf) {
      const INFCL_LDS char* cur = lds + buf * TILEB;
      const int lo = opaque_lane();
      const int l32o = lo & 31, ho = lo >> 5;
      const int g4 = lo >> 4, l16 = lo & 15;
      const int e = l16 >> 2, qq = l16 & 3, nb16 = g4 & 1, hh = g4 >> 1;
      const int lb = 2 * nb16 + (qq >> 1);
      const int fo = (qq & 1) * 8;
      // B-fragment offsets of this wave's feature blocks (read t = 0, 1)
      int offB[2][FBW];
#pragma unroll
      for (int fbw = 0; fbw < FBW; ++fbw) {
        const int fbabs = pass * FB + wave * FBW + fbw;
#pragma unroll
        for (int t = 0; t < 2; ++t)
          offB[t][fbw] = (8 * hh + 4 * t + e) * ROWB +
                         16 * (16 * (fbabs >> 2) + 4 * ((fbabs & 3) ^ e) + (lb ^ ((t + 2 * hh) & 3))) + fo;
      }
      typedef short s16x8 __attribute__((ext_vector_type(8)));
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        bf16x8 A[4];
#pragma unroll
        for (int ob = 0; ob < 4; ++ob) A[ob] = *(const INFCL_LDS bf16x8*)(gp_lds + gp_off(32 * ob + l32o, 2 * s2 + ho));
#pragma unroll
        for (int fbw = 0; fbw < FBW; ++fbw) {
          const int imm = 16 * s2 * ROWB;
          s16x4 b0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((INFCL_LDS s16x4*)(cur + offB[0][fbw] + imm));
          s16x4 b1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((INFCL_LDS s16x4*)(cur + offB[1][fbw] + imm));
          const s16x8 bb = {b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
#pragma unroll
          for (int ob = 0; ob < 4; ++ob)
            dacc[ob * FBW + fbw] = mfma_bf16(A[ob], __builtin_bit_cast(bf16x8, bb), dacc[ob * FBW + fbw]);
        }
      }
    };

    // fp32 GEMM2: this wave's own rows x all the pass's features; step r
    // contracts swept row jr(r, h) of each lane half.
    auto gemm2_f32 = [&](int buf, const float (&gv)[16]) {
      const INFCL_LDS char* cur = lds + buf * TILEB;
#pragma unroll
      for (int fb = 0; fb < FB; ++fb) {
        const int fbabs = pass * FB + fb;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = bwd_perm(8 * (r >> 2) + 4 * h + (r & 3));
          const int cf = 8 * fbabs + (l32 >> 2);
          float bv = *(const INFCL_LDS float*)(cur + j * ROWB + 16 * (cf ^ bwd_g(j)) + (l32 & 3) * 4);
          dacc[fb] = mfma_f32(gv[r], bv, dacc[fb]);
        }
      }
    };

    // DMA instructions this wave issues per tile (wave 0 also copies the tile's
    // log-sum-exp values): the wait before a tile's last barrier lets the
    // NBUF-2 younger tiles stay in flight.
    for (int k = 0; k < NBUF - 1; ++k)
      if (k < ntile) issue_tile(k, k);
    wait_dma();
    __syncthreads();
    int bcur = 0;
    for (int jt = 0; jt < ntile; ++jt) {
      const int bload = bcur == 0 ? NBUF - 1 : bcur - 1;  // buffer of tile jt-1, free since the last barrier
      if (jt + NBUF - 1 < ntile) issue_tile(jt + NBUF - 1, bload);
      float gv[16];
      f32x16 sacc = gemm1(bcur);
      const float d0 = epilogue(jt, bcur, sacc, gv);
      if (pass == 0) ds_acc += (double)d0;
      if constexpr (ES == 2) {
        // publish this wave's G' rows (bf16): chunk 2 s2 + h of row 32 wave + l32
        const int lo = opaque_lane();
        const int rowg = 32 * wave + (lo & 31);
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          bf16x8 ga;
#pragma unroll
          for (int t = 0; t < 8; ++t) ga[t] = (__bf16)gv[8 * s2 + t];
          *(INFCL_LDS bf16x8*)(gp_lds + gp_off(rowg, 2 * s2 + (lo >> 5))) = ga;
        }
        __syncthreads();
        gemm2_bf16(bcur);
      } else {
        gemm2_f32(bcur, gv);
      }
      // tile jt+1 must be in LDS; tiles jt+2 .. jt+NBUF-1 may still load
      const int younger = (ntile - 1 - (jt + 1)) < (NBUF - 2) ? (ntile - 1 - (jt + 1)) : (NBUF - 2);
      if (younger <= 0) {
        wait_dma();
      } else {
        wait_dma_allow(younger * (NIW + (wave == 0 ? 1 : 0)));
      }
      __syncthreads();
      bcur = bcur == NBUF - 1 ? 0 : bcur + 1;
    }

    // ---- write dOwn: lane holds feature l32 of a 32-feature block, rows 8(r>>2)+4h+(r&3)
    if constexpr (ES == 2) {
      const int64_t wg0 = (int64_t)blockIdx.x * kBwdBM;
      const bool all_ok = wg0 + kBwdBM <= b;
#pragma unroll
      for (int ob = 0; ob < 4; ++ob) {
        float* dst = p.dOwn + (wg0 + 32 * ob + 4 * h) * D + 32 * (pass * FB + wave * FBW) + l32;
#pragma unroll
        for (int fbw = 0; fbw < FBW; ++fbw)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int64_t row = wg0 + 32 * ob + 8 * (r >> 2) + 4 * h + (r & 3);
            if (all_ok || row < b) dst[(8 * (r >> 2) + (r & 3)) * D + 32 * fbw] = kfin * dacc[ob * FBW + fbw][r];
          }
      }
    } else {
      float* dst = p.dOwn + (own0 + 4 * h) * D + 32 * pass * FB + l32;
#pragma unroll
      for (int fb = 0; fb < FB; ++fb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t row = own0 + 8 * (r >> 2) + 4 * h + (r & 3);
          if (wave_rows_ok || row < b) dst[(8 * (r >> 2) + (r & 3)) * D + 32 * fb] = kfin * dacc[fb][r];
        }
    }
  }

  // ---- dscale partial of this workgroup: fixed-order reduction
  __shared__ double red[256];
  red[threadIdx.x] = ds_acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) p.ds_part[blockIdx.x] = red[0];
}

// dscale = dloss / (2b) * (sum of both launches' partials), fixed order
__global__ void __launch_bounds__(256) dscale_finish(const double* part, int64_t n, int64_t b, const float* dloss,
                                                     float* dscale) {
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
    *dscale = (float)(red[0] * dl / (2.0 * (double)b));
  }
}

// Pass width: largest FB (32-feature blocks) dividing d/32 whose accumulators
// (16 FB registers) fit next to the own operand (d/4 or d/2 registers); for
// bf16 FB is also a multiple of 4 (see the transposing-read addressing).
// Build-time tuning knobs: the register budget shared by the own operand and
// the gradient accumulators, and whether the three-buffer pipeline is used.
#ifndef INFCL_BWD_REG_BUDGET
#define INFCL_BWD_REG_BUDGET 384
#endif
#ifndef INFCL_BWD_PIPE
#define INFCL_BWD_PIPE 0
#endif
#ifndef INFCL_BWD_RING
#define INFCL_BWD_RING 2
#endif

template <typename TIN, int D>
static int launch_bwd_d(const BwdParams& p, int nwg, hipStream_t stream) {
  constexpr int ES = sizeof(TIN);
  constexpr int OWNREGS = D * ES / 8;
  constexpr int NB32 = D / 32;
  constexpr int FBMAX = (INFCL_BWD_REG_BUDGET - OWNREGS) / 16;
  constexpr int FB = [] {
    int best = ES == 4 ? 1 : 4;  // bf16: at least one 128-feature group
    for (int f = 1; f <= NB32; ++f)
      if (NB32 % f == 0 && f <= FBMAX && (ES == 4 || f % 4 == 0)) best = f;
    return best;
  }();
  static_assert(ES == 4 || FB % 4 == 0, "bf16 pass width must be a multiple of 128 features");
  hipLaunchKernelGGL((bwd_sweep<TIN, D, FB, INFCL_BWD_PIPE != 0, INFCL_BWD_RING>), dim3(nwg), dim3(256), 0, stream, p);
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
      case 768: return launch_bwd_d<TIN, 768>(p, nwg, stream);
      case 896: return launch_bwd_d<TIN, 896>(p, nwg, stream);
      case 1024: return launch_bwd_d<TIN, 1024>(p, nwg, stream);
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

int launch_bwd(const void* img, const void* txt, int64_t b, int64_t d, int dtype, const float* scale,
               const float* lse_r, const float* lse_c, const float* aux, const float* dloss, float* dimg, float* dtxt,
               float* dscale, double* ds_part, hipStream_t stream) {
  const int nwg = (int)((b + kBwdBM - 1) / kBwdBM);
  BwdParams p;
  p.b = b;
  p.d = d;
  p.scale = scale;
  p.udiag = aux + 2 * b;
  p.dloss = dloss;
  // launch 1: own = image rows (dimg), swept = text rows
  p.own = img;
  p.swept = txt;
  p.lse_own = lse_r;
  p.lse_swept = lse_c;
  p.ell_own = aux;
  p.ell_swept = aux + b;
  p.dOwn = dimg;
  p.ds_part = ds_part;
  int rc = dtype == 0 ? launch_bwd_t<__bf16>(p, nwg, stream) : launch_bwd_t<float>(p, nwg, stream);
  if (rc) return rc;
  // launch 2: own = text rows (dtxt), swept = image rows
  p.own = txt;
  p.swept = img;
  p.lse_own = lse_c;
  p.lse_swept = lse_r;
  p.ell_own = aux + b;
  p.ell_swept = aux;
  p.dOwn = dtxt;
  p.ds_part = ds_part + nwg;
  rc = dtype == 0 ? launch_bwd_t<__bf16>(p, nwg, stream) : launch_bwd_t<float>(p, nwg, stream);
  if (rc) return rc;
  hipLaunchKernelGGL(dscale_finish, dim3(1), dim3(256), 0, stream, (const double*)ds_part, (int64_t)2 * nwg, b,
                     dloss, dscale);
  return hipGetLastError() == hipSuccess ? 0 : 1;
}

bool bwd_supported(int64_t d, int dtype) {
  if (dtype == 0) return d % 128 == 0 && d >= 128 && d <= 1024;
  return d % 64 == 0 && d >= 64 && d <= 512;
}

}  // namespace infcl
