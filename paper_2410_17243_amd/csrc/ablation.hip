// Ablation: the single-launch backward of the appendix's in-GPU algorithm
// (gfx950), set against the two-launch backward of infcl_bwd.
//
// The appendix's backward keeps the image gradient of a row block on chip and,
// for every column tile j, reads the text-gradient tile dT^j from memory, adds
// the block's contribution and writes it back; S and G' are computed once per
// tile.  With row blocks in parallel that update is an atomic add.  This
// kernel does exactly that:
//   - a workgroup owns 64 image rows (the wide sweep's layout: the wave pair
//     (2 ob, 2 ob + 1) holds own block ob, each wave one half of the features;
//     the image gradients of the 64 rows stay in AGPRs for the whole sweep);
//   - per text tile of 32 rows: S^T (GEMM1, joined across the wave pair), G'
//     (both halves of the loss and both dscale terms), dI += G' T (GEMM2 as in
//     the wide sweep) and dT^j += G'^T I (the own rows' transposed fragments,
//     loaded once, as the B operand; G'^T gathered from the G' block), added
//     into dtxt with hardware fp32 atomics;
//   - start tiles are staggered over the workgroups, so that at any time the
//     workgroups add into different tiles.
// 64 own rows is what the register file allows next to the dT product's own
// operand at d = 512 (the two-launch sweep owns 128).  Each text element then
// receives ceil(b / 64) atomic additions: 32 GiB of atomic payload at
// b = 32768, d = 512, against 128 MiB of gradients written once by the
// two-launch backward, which instead recomputes GEMM1 in its second launch.
//
// Results agree with infcl_bwd to rounding; the order of the atomic additions
// varies from run to run, so dtxt is not bitwise reproducible.
#include "bwd.hpp"
#include "infcl_ablation.h"

namespace infcl {

constexpr int kSingleBM = 64;  // own image rows per workgroup

__global__ void dscale_finish(const double* part, int64_t n, int64_t b, const float* dloss, float* dscale,
                              double* dscale64);
__global__ void lse_to_log2(const float* lse_r, const float* lse_c, float* l2r, float* l2c, int64_t b);

struct SingleParams {
  const __bf16* img;   // own rows i, [b, d]
  const __bf16* txt;   // swept rows j, [b, d]
  int64_t b;
  const float* scale;
  const float* lse_r;  // [b] natural log
  const float* l2c;    // [b] c_j log2(e)
  const float* ell_r;  // [b]
  const float* ell_c;  // [b]
  const float* udiag;  // [b] <img_i, txt_i>
  const float* dloss;
  float* dimg;         // [b, d]
  float* dtxt;         // [b, d], zero on entry, accumulated with atomics
  double* ds_part;     // [gridDim.x]
};

__global__ void __launch_bounds__(256) zero_f32(float* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = 0.f;
}

template <int D>
__global__ void __launch_bounds__(256, 1) bwd_single(SingleParams p) {
  constexpr int KS = D / 16;
  constexpr int KH = KS / 2;
  constexpr int ROWG = D * 2;
  constexpr int TILEB = kBwdBN * ROWG;
  constexpr int NIW = TILEB / 4096;
  constexpr int FBW = D / 128;  // 32-feature blocks per wave (both products)
  constexpr int kPre = 4;
  static_assert(KH % 8 == 0, "feature halves start on a 128-feature segment");
  static_assert(2 * TILEB + 4 * 1024 + kSingleBM * kBwdBN * 2 + 4 * 64 * 8 * 4 + 2048 <= 160 * 1024, "LDS budget");
  __shared__ __attribute__((aligned(1024))) char tA_[TILEB];
  __shared__ __attribute__((aligned(1024))) char tB_[TILEB];
  __shared__ __attribute__((aligned(1024))) float lA_[256];  // c_j log2 e of the tile's rows
  __shared__ __attribute__((aligned(1024))) float lB_[256];
  __shared__ __attribute__((aligned(1024))) float uA_[256];  // u_jj of the tile's rows
  __shared__ __attribute__((aligned(1024))) float uB_[256];
  __shared__ __attribute__((aligned(1024))) char gp_[kSingleBM * kBwdBN * 2];
  __shared__ __attribute__((aligned(16))) float xs_[4][64][8];
  __shared__ double red[256];
  INFCL_LDS char* const tA = (INFCL_LDS char*)tA_;
  INFCL_LDS char* const tB = (INFCL_LDS char*)tB_;
  INFCL_LDS float* const lA = (INFCL_LDS float*)lA_;
  INFCL_LDS float* const lB = (INFCL_LDS float*)lB_;
  INFCL_LDS float* const uA = (INFCL_LDS float*)uA_;
  INFCL_LDS float* const uB = (INFCL_LDS float*)uB_;
  INFCL_LDS char* const gp = (INFCL_LDS char*)gp_;

  const int lane = __lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ob = wave >> 1, kh = wave & 1;
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t b = p.b;
  const int64_t wg0 = (int64_t)blockIdx.x * kSingleBM;
  const int64_t own0 = wg0 + 32 * ob;
  const int64_t iown = own0 + l32;
  const bool own_ok = iown < b;
  const int64_t irow = own_ok ? iown : b - 1;
  const bool wave_rows_ok = own0 + 32 <= b;
  const int ntile = (int)((b + kBwdBN - 1) / kBwdBN);
  // staggered sweep: workgroup w starts at tile w * ntile / gridDim.x
  const int jstart = (int)(((int64_t)blockIdx.x * ntile) / gridDim.x);
  auto tile_at = [&](int k) { return k < ntile ? (jstart + k) % ntile : -1; };

  const float s = p.scale[0];
  const float k2 = s * kLog2e;
  const float dl = p.dloss ? p.dloss[0] : 1.0f;
  const float kfin = dl * s / (2.0f * (float)b);

  // GEMM1's own operand: row irow, features kh d/2 + 16 s2 + 8h .. +8
  bf16x8 ownf[KH];
  {
    const __bf16* src = p.img + irow * D + kh * (D / 2) + 8 * h;
#pragma unroll
    for (int s2 = 0; s2 < KH; ++s2) ownf[s2] = *(const bf16x8*)(src + 16 * s2);
  }
  // the dT product's B operand, fixed for the sweep: for feature block
  // fb = wave FBW + f and own rows 16 kq + 8h .. +8 of the workgroup, lane
  // holds feature 32 fb + l32 of those 8 rows (rows past b read as zero)
  bf16x8 ownT[4][FBW];
#pragma unroll
  for (int kq = 0; kq < 4; ++kq)
#pragma unroll
    for (int f = 0; f < FBW; ++f) {
      const int n = 32 * (wave * FBW + f) + l32;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int64_t r = wg0 + 16 * kq + 8 * h + e;
        ownT[kq][f][e] = r < b ? p.img[r * D + n] : (__bf16)0.f;
      }
    }
  const float aO = own_ok ? p.lse_r[iown] * kLog2e : 0.f;
  const float uO = own_ok ? p.udiag[iown] : 0.f;
  const float gdiag = own_ok ? expm1f(-p.ell_r[iown]) + expm1f(-p.ell_c[iown]) : 0.f;

  auto opaque_lane = [&]() {
    int lo = lane;
    asm volatile("" : "+v"(lo));
    return lo;
  };
  auto tile_rsrc = [&](int jt) {
    const int64_t j0 = (int64_t)(jt < 0 ? 0 : jt) * kBwdBN;
    return rsrc_words((const char*)p.txt + j0 * ROWG, jt < 0 ? 0 : (b - j0) * ROWG);
  };
  auto vec_rsrc = [&](const float* v, int jt) {
    const int64_t j0 = (int64_t)(jt < 0 ? 0 : jt) * kBwdBN;
    return rsrc_words(v + j0, jt < 0 ? 0 : (b - j0) * 4);
  };
  auto slot_lane_off = [&]() { return 16u * (uint32_t)(opaque_lane() & 7); };
  auto issue_slots = [&](int jt, INFCL_LDS float* l, INFCL_LDS float* u) {
    dma16_asm(vec_rsrc(p.l2c, jt), l, slot_lane_off());
    dma16_asm(vec_rsrc(p.udiag, jt), u, slot_lane_off());
  };

  double ds_acc = 0.0;
  f32x16 dacc[2 * FBW];
#pragma unroll
  for (int i = 0; i < 2 * FBW; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dacc[i][r] = 0.f;

  // ---- GEMM1: partial S^T (32 swept x 32 own) over this wave's feature half
  auto gemm1 = [&](const INFCL_LDS char* cur) {
    int offA[8];
    {
      const int lo = opaque_lane();
      const int rA = sweep_perm(lo & 31);
#pragma unroll
      for (int k = 0; k < 8; ++k) offA[k] = sweep_seg_off(rA, 2 * k + (lo >> 5));
    }
    const INFCL_LDS char* half = cur + kSeg * (kh * KH / 8);
    f32x16 sacc;
    bf16x8 ring[kPre];
#pragma unroll
    for (int i = 0; i < kPre; ++i) ring[i] = *(const INFCL_LDS bf16x8*)(half + offA[i & 7] + kSeg * (i >> 3));
    __builtin_amdgcn_sched_group_barrier(0x100, kPre, 0);
#pragma unroll
    for (int s2 = 0; s2 < KH; ++s2) {
      mfma16_vgpr<false>(sacc, ring[s2 % kPre], ownf[s2], s2 == 0, s2 == KH - 1);
      if (s2 + kPre < KH) {
        const int n = s2 + kPre;
        ring[s2 % kPre] = *(const INFCL_LDS bf16x8*)(half + offA[n & 7] + kSeg * (n >> 3));
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
    }
    return sacc;
  };

  // ---- join, G' of the wave's 8 entries (entry i <-> swept row
  // 16 kh + 8h + i of the tile) into the G' block, with the DMA of tile dtile
  // spread over the entries; returns dscale's share (both terms)
  auto join_gp = [&](int jt, const INFCL_LDS float* lcur, const INFCL_LDS float* ucur, const f32x16& sacc,
                     int dtile, INFCL_LDS char* ddst) -> float {
    float mine[8], other[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      mine[i] = kh ? sacc[8 + i] : sacc[i];
      other[i] = kh ? sacc[i] : sacc[8 + i];
    }
    *(INFCL_LDS f32x4*)&xs_[wave][lane][0] = f32x4{other[0], other[1], other[2], other[3]};
    *(INFCL_LDS f32x4*)&xs_[wave][lane][4] = f32x4{other[4], other[5], other[6], other[7]};
    __syncthreads();
    const f32x4 q0 = *(const INFCL_LDS f32x4*)&xs_[wave ^ 1][lane][0];
    const f32x4 q1 = *(const INFCL_LDS f32x4*)&xs_[wave ^ 1][lane][4];
    const INFCL_LDS float* lp = lcur + 16 * kh + 8 * h;
    const f32x4 L0 = *(const INFCL_LDS f32x4*)lp;
    const f32x4 L1 = *(const INFCL_LDS f32x4*)(lp + 4);
    const INFCL_LDS float* up = ucur + 16 * kh + 8 * h;
    const f32x4 U0 = *(const INFCL_LDS f32x4*)up;
    const f32x4 U1 = *(const INFCL_LDS f32x4*)(up + 4);
    const int64_t j0 = (int64_t)jt * kBwdBN;
    const bool special = (j0 == own0) || (j0 + kBwdBN > b) || !wave_rows_ok;
    float ds_tile = 0.f;
    bf16x8 ga;
    const u32x4 drs = tile_rsrc(dtile);
    const uint32_t dlo = sweep_dma_lane_off(opaque_lane(), wave, ROWG);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
#pragma unroll
      for (int u = 0; u < (NIW + 7) / 8; ++u) {
        const int kk = i + 8 * u;
        if (kk < NIW) dma16_asm(drs, ddst + 1024 * (wave + 4 * kk), dlo + sweep_dma_kk_off(kk, wave, ROWG));
      }
      const float x = mine[i] + (i < 4 ? q0[i] : q1[i - 4]);
      const float Lj = i < 4 ? L0[i] : L1[i - 4];
      const float uS = i < 4 ? U0[i] : U1[i - 4];
      const float pO = exp2_hw(__builtin_fmaf(x, k2, -aO));
      const float pS = exp2_hw(__builtin_fmaf(x, k2, -Lj));
      float gg = pO + pS;
      float dsv = __builtin_fmaf(pO, x - uO, pS * (x - uS));
      if (special) {
        const int64_t j = j0 + 16 * kh + 8 * h + i;
        const bool ok = (bool)(own_ok & (j < b));
        const bool dg = j == iown;
        gg = dg ? gdiag : (ok ? gg : 0.f);
        dsv = (ok & !dg) ? dsv : 0.f;
      }
      ds_tile += dsv;
      ga[i] = (__bf16)gg;
    }
    const int row = 32 * ob + l32;
    *(INFCL_LDS bf16x8*)(gp + gp_chunk_off(row, 2 * kh + h)) = ga;
    return ds_tile;
  };

  // ---- dI: all 64 own rows' G' x this wave's quarter of the tile's features
  auto gemm2 = [&](const INFCL_LDS char* cur) {
    const int lo = opaque_lane();
    const int ho = lo >> 5;
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      bf16x8 A[2];
#pragma unroll
      for (int o2 = 0; o2 < 2; ++o2)
        A[o2] = *(const INFCL_LDS bf16x8*)(gp + 2048 * o2 + gp_chunk_off(lo & 31, 2 * s2 + ho));
#pragma unroll
      for (int fbw = 0; fbw < FBW; ++fbw) {
        const int fbabs = wave * FBW + fbw;
        s16x4 bq[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int off = sweep_tr_off(lo, t, fbabs) + 16 * kSegRow * s2;
          bq[t] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((INFCL_LDS s16x4*)(cur + off));
        }
        const s16x8 bb = {bq[0][0], bq[0][1], bq[0][2], bq[0][3], bq[1][0], bq[1][1], bq[1][2], bq[1][3]};
#pragma unroll
        for (int o2 = 0; o2 < 2; ++o2)
          dacc[o2 * FBW + fbw] = mfma_bf16(A[o2], __builtin_bit_cast(bf16x8, bb), dacc[o2 * FBW + fbw]);
      }
    }
  };

  // ---- dT^j += G'^T I over the 64 own rows for this wave's quarter of the
  // features, added into dtxt with fp32 atomics.  A operand: lane holds swept
  // row l32 and own rows 16 kq + 8h .. +8, gathered from the G' block.
  auto gemm_dt = [&](int jt) {
    f32x16 tacc[FBW];
#pragma unroll
    for (int f = 0; f < FBW; ++f)
#pragma unroll
      for (int r = 0; r < 16; ++r) tacc[f][r] = 0.f;
    const INFCL_LDS unsigned short* g16 = (const INFCL_LDS unsigned short*)gp;
#pragma unroll
    for (int kq = 0; kq < 4; ++kq) {
      bf16x8 a;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int r = 16 * kq + 8 * h + e;  // own row of the workgroup
        const int off = r * 32 + 8 * (((l32 >> 3)) ^ ((r >> 2) & 3)) + (l32 & 7);  // in 16-bit units
        a[e] = __builtin_bit_cast(__bf16, g16[off]);
      }
#pragma unroll
      for (int f = 0; f < FBW; ++f) tacc[f] = mfma_bf16(a, ownT[kq][f], tacc[f]);
    }
    const int64_t j0 = (int64_t)jt * kBwdBN;
#pragma unroll
    for (int f = 0; f < FBW; ++f) {
      const int n = 32 * (wave * FBW + f) + l32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t j = j0 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (j < b) unsafeAtomicAdd(p.dtxt + j * D + n, kfin * tacc[f][r]);
      }
    }
  };

  // ---- sweep
  {
    const int t0 = tile_at(0);
    const u32x4 rs = tile_rsrc(t0);
    const uint32_t lo = sweep_dma_lane_off(opaque_lane(), wave, ROWG);
#pragma unroll
    for (int kk = 0; kk < NIW; ++kk) dma16_asm(rs, tA + 1024 * (wave + 4 * kk), lo + sweep_dma_kk_off(kk, wave, ROWG));
    issue_slots(t0, lA, uA);
  }
  wait_dma();
  __syncthreads();
  for (int k = 0; k < ntile; ++k) {
    const bool odd = (k & 1) != 0;
    INFCL_LDS char* cur = odd ? tB : tA;
    INFCL_LDS char* nxt = odd ? tA : tB;
    const int jt = tile_at(k), jn = tile_at(k + 1);
    issue_slots(jn, odd ? lA : lB, odd ? uA : uB);
    const f32x16 sacc = gemm1(cur);
    ds_acc += (double)join_gp(jt, odd ? lB : lA, odd ? uB : uA, sacc, jn, nxt);
    __syncthreads();  // the G' block is complete
    gemm2(cur);
    gemm_dt(jt);
    wait_dma();
    __syncthreads();  // tile k+1 landed; cur, the G' block and the join area are free
  }

  // ---- dimg
  const bool all_ok = wg0 + kSingleBM <= b;
#pragma unroll
  for (int o2 = 0; o2 < 2; ++o2) {
    float* dst = p.dimg + (wg0 + 32 * o2 + 4 * h) * D + 32 * (wave * FBW) + l32;
#pragma unroll
    for (int fbw = 0; fbw < FBW; ++fbw)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = wg0 + 32 * o2 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (all_ok || row < b) dst[(8 * (r >> 2) + (r & 3)) * D + 32 * fbw] = kfin * dacc[o2 * FBW + fbw][r];
      }
  }
  red[threadIdx.x] = ds_acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) p.ds_part[blockIdx.x] = red[0];
}

}  // namespace infcl

extern "C" int infcl_ablation_bwd_single(const void* img, const void* txt, int64_t b, int64_t d, int dtype,
                                         const float* scale, const float* lse_r, const float* lse_c,
                                         const float* aux, const float* dloss, float* dimg, float* dtxt,
                                         float* dscale, void* workspace, size_t ws_bytes, void* stream) {
  using namespace infcl;
  auto al = [](const void* q, uintptr_t a) { return q != nullptr && ((uintptr_t)q % a) == 0; };
  if (b < 1 || d < 1 || !al(img, 16) || !al(txt, 16) || !al(scale, 4) || !al(lse_r, 16) || !al(lse_c, 16) ||
      !al(aux, 16) || !al(dimg, 16) || !al(dtxt, 16) || !al(dscale, 4) || !al(workspace, 256) ||
      (dloss != nullptr && ((uintptr_t)dloss % 4) != 0))
    return 1;
  if (dtype != 0 || (d != 256 && d != 512) || b > ((int64_t)1 << 30)) return 2;
  const int64_t nwg = (b + kSingleBM - 1) / kSingleBM;
  const size_t lse2_bytes = ((size_t)2 * b * sizeof(float) + 255) & ~(size_t)255;
  if (ws_bytes < lse2_bytes + (size_t)nwg * sizeof(double)) return 3;
  float* l2r = (float*)workspace;
  float* l2c = l2r + b;
  double* ds_part = (double*)((char*)workspace + lse2_bytes);
  hipStream_t st = (hipStream_t)stream;
  const unsigned nblk = (unsigned)((b + 255) / 256);
  hipLaunchKernelGGL(lse_to_log2, dim3(nblk), dim3(256), 0, st, lse_r, lse_c, l2r, l2c, b);
  hipLaunchKernelGGL(zero_f32, dim3(2048), dim3(256), 0, st, dtxt, b * d);
  SingleParams p;
  p.img = (const __bf16*)img;
  p.txt = (const __bf16*)txt;
  p.b = b;
  p.scale = scale;
  p.lse_r = lse_r;
  p.l2c = l2c;
  p.ell_r = aux;
  p.ell_c = aux + b;
  p.udiag = aux + 2 * b;
  p.dloss = dloss;
  p.dimg = dimg;
  p.dtxt = dtxt;
  p.ds_part = ds_part;
  if (d == 256)
    hipLaunchKernelGGL(bwd_single<256>, dim3((unsigned)nwg), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(bwd_single<512>, dim3((unsigned)nwg), dim3(256), 0, st, p);
  hipLaunchKernelGGL(dscale_finish, dim3(1), dim3(256), 0, st, (const double*)ds_part, nwg, b, dloss, dscale,
                     (double*)nullptr);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}
