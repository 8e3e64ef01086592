// Forward sweep of the tiled symmetric InfoNCE loss for fp32 inputs (gfx950),
// and the finalize shared by both forward sweeps.  (16-bit inputs take the
// resident-rows sweep of fwd2.hip.)
//
// What is computed (paper Sec. 3.1, Eq. 2-5; the in-GPU forward algorithm of
// Sec. 3.2): for every row i and column j of S = s * img * txt^T, the
// off-diagonal log-sum-exp of row i and of column j, without storing S.
//
// Work decomposition (differs from the paper's one-row-block-per-thread-block
// design: here a persistent 2-D grid of workgroups shares the column
// statistics without atomics):
//   - A workgroup tile covers BI = 64 rows i (image rows) x BJ = 256 columns j
//     (text rows).  The MFMA computes the transposed block S^T (M = j, N = i),
//     so each lane owns a fixed i and 16 consecutive-ish j's per 32x32 block.
//   - Workgroup (q, g) of a P_r x P_c grid sweeps row tiles q, q+P_r, ... and,
//     for each, the column tiles of column group g.  Row statistics stay in
//     registers across the sweep (one running pair per lane and row, merged
//     across lanes only when the row tile is done); column statistics are
//     reduced across lanes every tile and merged into the group's own slice
//     colR/colL[q][j] in global memory (only this workgroup touches it).
//   - The finalize kernel merges the partial pairs of every row and column in
//     a fixed order and evaluates the per-sample terms in fp64.
//   - Workgroups of one column group are launched with the same index modulo
//     8, so they run on one XCD and share its L2 for the text tiles.
//
// Online log-sum-exp (Eq. 4-5) with lazy references: each running pair keeps a
// reference R (a value actually seen, so l >= 1 after the first one) and adds
// exp2(y - R) for new values y; a tile whose partial sum exceeds 2^64 (or is
// not finite, e.g. while R is still -inf) is redone with the exact max-rescaled
// merge.  The paper's merge starts from 0; the identity of the merge is the
// empty sum (R = -inf, l = 0), which is what is used here.
#include "common.hpp"

namespace infcl {

struct FwdParams {
  const void* img;  // rows i, [b, d]
  const void* txt;  // rows j, [b, d]
  int64_t b, d;
  const float* scale;
  float* rowR;  // [Pc * 4][rstride]   per (column group, wave) partial row pairs, by own row - r0
  float* rowL;
  float* colR;  // [Pr][b]       per row group partial column pairs
  float* colL;
  float* udiag;  // [b]  <img_i, txt_i> as accumulated by the MFMA
  int Pr, Pc;
  int nRT, nCT;
  int64_t r0, rend;  // own rows [r0, rend) (a shard of the batch; 0 and b for the whole batch)
  int64_t rstride;   // rend - r0
};

constexpr int kFwdBI = 64;    // rows i per workgroup tile
constexpr int kFwdBJ = 256;   // columns j per workgroup tile
constexpr int kFwdRows = kFwdBI + kFwdBJ;
constexpr int kFwdStageBytes = kFwdRows * 128;  // 128 bytes of every row per stage

// Chunk swizzle for 128-byte rows: 16 consecutive rows reading the same logical
// 16-byte chunk hit 16 distinct bank groups.
__device__ __forceinline__ int fwd_swz(int r, int c) { return c ^ ((r >> 1) & 7); }

// Per-lane source offsets of the K-stage DMA: instruction k (= wave + 4 kk)
// fills tile rows 8k..8k+7; lane L copies logical chunk fwd_swz(r, L & 7) of row
// r = 8k + L/8 to physical chunk L & 7.  Rows 0..63 are image rows, 64..319 text rows.
struct FwdDmaOffsets {
  uint32_t off[kFwdRows / 8 / 4];
};

__device__ __forceinline__ FwdDmaOffsets fwd_dma_offsets(int64_t d, int es, int wave, int lane) {
  FwdDmaOffsets o;
#pragma unroll
  for (int kk = 0; kk < kFwdRows / 8 / 4; ++kk) {
    const int k = wave + 4 * kk;
    const int r = 8 * k + (lane >> 3);
    const int rl = kk < 2 ? r : r - kFwdBI;  // row within the image or the text tile
    o.off[kk] = (uint32_t)(rl * d * es + 16 * fwd_swz(r, lane & 7));
  }
  return o;
}

// Issue the DMA of one K-stage (128 bytes of each of the 320 tile rows).  Rows
// past b fall outside the buffer resources and load as zeros (they are masked).
__device__ __forceinline__ void fwd_stage_dma(const FwdParams& p, const FwdDmaOffsets& o, int64_t i0, int64_t j0,
                                              int st, INFCL_LDS char* buf, int wave) {
  const int64_t b = p.b, rowb = p.d * (int64_t)sizeof(float);
  const u32x4 ri = rsrc_words((const char*)p.img + i0 * rowb, (p.rend - i0) * rowb);
  const u32x4 rt = rsrc_words((const char*)p.txt + j0 * rowb, (b - j0) * rowb);
  const uint32_t soff = (uint32_t)st * 128u;
#pragma unroll
  for (int kk = 0; kk < kFwdRows / 8 / 4; ++kk)
    dma16_asm(kk < 2 ? ri : rt, buf + 1024 * (wave + 4 * kk), o.off[kk], soff);
}

// MFMA work of one K-stage: acc[mb][nb] += S^T block (j block mb, i block nb).
// A 16-wide fp32 contraction step is 64 bytes; lane half h holds floats 8h..8h+7.
__device__ __forceinline__ void fwd_stage_mfma(const INFCL_LDS char* buf, f32x16 (&acc)[2][2], int wave, int lane) {
  const int l32 = lane & 31, h = lane >> 5;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    f32x4 a[2][2], bb[2][2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = 4 * s + 2 * h + u;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        int r = kFwdBI + 64 * wave + 32 * mb + l32;
        a[mb][u] = *(const INFCL_LDS f32x4*)(buf + r * 128 + fwd_swz(r, c) * 16);
      }
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        int r = 32 * nb + l32;
        bb[nb][u] = *(const INFCL_LDS f32x4*)(buf + r * 128 + fwd_swz(r, c) * 16);
      }
    }
#pragma unroll
    for (int t = 0; t < 8; ++t)
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          acc[mb][nb] = mfma_f32(a[mb][t >> 2][t & 3], bb[nb][t >> 2][t & 3], acc[mb][nb]);
  }
}

// One butterfly step of the reduce-scatter below: lanes exchange the half of
// their HALF*2 live values that the partner keeps (partner = lane ^ HALF).
template <bool kMax, int HALF>
__device__ __forceinline__ void rs_step(float (&v)[32], int l32) {
  const bool bit = (l32 & HALF) != 0;
#pragma unroll
  for (int t = 0; t < HALF; ++t) {
    const float send = bit ? v[t] : v[t + HALF];
    const float keep = bit ? v[t + HALF] : v[t];
    const float recv = shfl_xor(send, HALF);
    v[t] = kMax ? fmaxf(keep, recv) : keep + recv;
  }
}

// Reduce-scatter over the 32 lanes of each wave half: on entry v[t] is this
// lane's partial for value index t (0..31); on exit the result is the total over
// the 32 lanes for index t = lane % 32 (sum, or max when kMax).
template <bool kMax>
__device__ __forceinline__ float half_reduce_scatter(float (&v)[32], int lane) {
  const int l32 = lane & 31;
#pragma unroll
  for (int t = 0; t < 16; ++t) {
    // odd 16-lane rows of x swap with even rows of y: lanes with bit 4 clear end
    // with (own v[t], partner v[t]); lanes with bit 4 set with (partner v[t+16], own v[t+16])
    auto sw = __builtin_amdgcn_permlane16_swap(__float_as_uint(v[t]), __float_as_uint(v[t + 16]), false, false);
    const float x = __uint_as_float(sw[0]), y = __uint_as_float(sw[1]);
    v[t] = kMax ? fmaxf(x, y) : x + y;
  }
  rs_step<kMax, 8>(v, l32);
  rs_step<kMax, 4>(v, l32);
  rs_step<kMax, 2>(v, l32);
  rs_step<kMax, 1>(v, l32);
  return v[0];
}

// Epilogue of one workgroup tile.  acc[mb][nb][r] <-> column
// j = jw + 32 mb + 8 (r>>2) + (r&3), row i = i0 + 32 nb + l32, jw = j0 + 64 wave + 4 h.
// The exponent of an entry is fma(acc, kk, -reference): unmasked tiles pass the
// raw dot products with kk = s log2(e); tiles touching the diagonal or the
// ragged end pass y = s log2(e) <.,.> with excluded entries set to -inf and kk = 1.
template <bool MASKED>
__device__ __forceinline__ void fwd_epilogue(const FwdParams& p, const f32x16 (&acc)[2][2], float (&rowR)[2],
                                             float (&rowL)[2], int64_t j0, int q, bool first_row_tile, float k2,
                                             int wave, int lane) {
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t b = p.b;
  const int64_t jw = j0 + 64 * wave + 4 * h;
  const float ninf = -__builtin_inff();
  const float kk = MASKED ? 1.0f : k2;
  auto jof = [&](int mb, int r) -> int64_t { return jw + 32 * mb + 8 * (r >> 2) + (r & 3); };

  // ---- row statistics: per lane and row, lazy reference with an exact fallback
  {
    float t[2];
    bool bad = false;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      float s = 0.f;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += exp2_hw(__builtin_fmaf(acc[mb][nb][r], kk, -rowR[nb]));
      t[nb] = s;
      bad |= !lazy_ok(s);
    }
    if (!wave_any(bad)) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) rowL[nb] += t[nb];
    } else {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        float m = rowR[nb];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) m = fmaxf(m, acc[mb][nb][r] * kk);
        const float ms = m == ninf ? 0.f : m;
        float s2 = rowL[nb] * exp2_hw(rowR[nb] - ms);
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) s2 += exp2_hw(__builtin_fmaf(acc[mb][nb][r], kk, -ms));
        rowL[nb] = m == ninf ? 0.f : s2;
        rowR[nb] = m;
      }
    }
  }

  // ---- column statistics: reference = the group's running pair for column j
  {
    const int64_t jmine = jof(l32 >> 4, l32 & 15);  // the column this lane reduces to
    float* cR = p.colR + (int64_t)q * b;
    float* cL = p.colL + (int64_t)q * b;
    float Rold = ninf, Lold = 0.f;
    float ref[32];
    if (first_row_tile) {
#pragma unroll
      for (int t = 0; t < 32; ++t) ref[t] = ninf;
    } else if constexpr (!MASKED) {
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const f32x4 v = *(const f32x4*)(cR + jw + 32 * mb + 8 * a);
#pragma unroll
          for (int c = 0; c < 4; ++c) ref[16 * mb + 4 * a + c] = v[c];
        }
      Rold = cR[jmine];
      Lold = cL[jmine];
    } else {
#pragma unroll
      for (int t = 0; t < 32; ++t) {
        const int64_t j = jof(t >> 4, t & 15);
        const float v = cR[j < b ? j : b - 1];
        ref[t] = j < b ? v : ninf;
      }
      const int64_t jc = jmine < b ? jmine : b - 1;
      const float r0 = cR[jc], l0 = cL[jc];
      Rold = jmine < b ? r0 : ninf;
      Lold = jmine < b ? l0 : 0.f;
    }
    float v[32];
#pragma unroll
    for (int t = 0; t < 32; ++t) {
      const int mb = t >> 4, r = t & 15;
      float s = 0.f;
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) s += exp2_hw(__builtin_fmaf(acc[mb][nb][r], kk, -ref[t]));
      // a column whose entries are all excluded so far has ref = -inf and sums
      // exp2(-inf + inf) = NaN here; that sends the tile to the exact path
      v[t] = s;
    }
    const float tot = half_reduce_scatter<false>(v, lane);
    float Rnew = Rold, Lnew = Lold + tot;
    if (wave_any(!lazy_ok(tot))) {
      // exact path: per-column max over this tile, broadcast, rescaled sums
#pragma unroll
      for (int t = 0; t < 32; ++t) {
        const int mb = t >> 4, r = t & 15;
        v[t] = fmaxf(acc[mb][0][r] * kk, acc[mb][1][r] * kk);
      }
      const float mt = half_reduce_scatter<true>(v, lane);
      const float Rn = fmaxf(Rold, mt);
#pragma unroll
      for (int t = 0; t < 32; ++t) {
        const float rn = shfl_idx(Rn, (lane & 32) | t);
        const float rs = rn == ninf ? 0.f : rn;
        const int mb = t >> 4, r = t & 15;
        float s = 0.f;
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) s += exp2_hw(__builtin_fmaf(acc[mb][nb][r], kk, -rs));
        v[t] = s;
      }
      const float tot2 = half_reduce_scatter<false>(v, lane);
      Rnew = Rn;
      Lnew = Rn == ninf ? 0.f : Lold * exp2_hw(Rold - Rn) + tot2;
    }
    if (!MASKED || jmine < b) {
      cR[jmine] = Rnew;
      cL[jmine] = Lnew;
    }
  }
}

__global__ void __launch_bounds__(256, 2) fwd_sweep(FwdParams p) {
  __shared__ __attribute__((aligned(1024))) char lds_[2 * kFwdStageBytes];
  INFCL_LDS char* lds0 = (INFCL_LDS char*)lds_;
  INFCL_LDS char* lds1 = lds0 + kFwdStageBytes;
  const int lane = __lane_id();
  const int wave = threadIdx.x >> 6;
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t b = p.b;
  const int nst = (int)((p.d * (int64_t)sizeof(float)) / 128);  // K-stages per tile (even)

  const int g = blockIdx.x % p.Pc;
  const int q = blockIdx.x / p.Pc;
  const int ct_lo = (int)(((int64_t)g * p.nCT) / p.Pc);
  const int ct_hi = (int)(((int64_t)(g + 1) * p.nCT) / p.Pc);
  const int ncol = ct_hi - ct_lo;
  const int nrow = q < p.nRT ? (p.nRT - 1 - q) / p.Pr + 1 : 0;
  const int ntile = ncol * nrow;
  if (ntile <= 0) return;

  const float k2 = p.scale[0] * kLog2e;
  const float ninf = -__builtin_inff();

  float rowR[2], rowL[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    rowR[nb] = ninf;
    rowL[nb] = 0.f;
  }

  const FwdDmaOffsets dmo = fwd_dma_offsets(p.d, (int)sizeof(float), wave, lane);
  int rr = 0, cc = 0;  // position of the current tile in this workgroup's (row, column) sweep
  fwd_stage_dma(p, dmo, p.r0 + (int64_t)q * kFwdBI, (int64_t)ct_lo * kFwdBJ, 0, lds0, wave);
  wait_dma();
  __syncthreads();

  for (int tau = 0; tau < ntile; ++tau) {
    const int64_t i0 = p.r0 + (int64_t)(q + rr * p.Pr) * kFwdBI;
    const int64_t j0 = (int64_t)(ct_lo + cc) * kFwdBJ;
    const bool has_next = tau + 1 < ntile;
    const int nrr = cc + 1 == ncol ? rr + 1 : rr;
    const int ncc = cc + 1 == ncol ? 0 : cc + 1;
    const int64_t ni0 = p.r0 + (int64_t)(q + nrr * p.Pr) * kFwdBI;
    const int64_t nj0 = (int64_t)(ct_lo + ncc) * kFwdBJ;

    f32x16 acc[2][2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.f;

    for (int st = 0; st < nst; st += 2) {
      fwd_stage_dma(p, dmo, i0, j0, st + 1, lds1, wave);
      fwd_stage_mfma(lds0, acc, wave, lane);
      wait_dma();
      __syncthreads();
      if (st + 2 < nst)
        fwd_stage_dma(p, dmo, i0, j0, st + 2, lds0, wave);
      else if (has_next)
        fwd_stage_dma(p, dmo, ni0, nj0, 0, lds0, wave);
      fwd_stage_mfma(lds1, acc, wave, lane);
      if (st + 2 < nst) {
        wait_dma();
        __syncthreads();
      }
    }

    // the next tile's first stage is in flight while the epilogue runs
    const bool diag = j0 < i0 + kFwdBI && i0 < j0 + kFwdBJ;
    const bool special = diag || (i0 + kFwdBI > p.rend) || (j0 + kFwdBJ > b);
    if (special) {
      const int64_t jw = j0 + 64 * wave + 4 * h;
      if (diag) {
        // the diagonal entry of row i sits in one lane of one wave, in block
        // mb == nb when i0 - j0 is a multiple of 64 (whole batch), in either
        // block for a shard starting at a multiple of 32
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          const int64_t i = i0 + 32 * nb + l32;
          float dv = 0.f;
          bool has = false;
#pragma unroll
          for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const bool hit = jw + 32 * mb + 8 * (r >> 2) + (r & 3) == i;
              dv = hit ? acc[mb][nb][r] : dv;
              has |= hit;
            }
          if (has && i < p.rend) p.udiag[i] = dv;
        }
      }
      // scaled exponents, -inf for the diagonal and for rows/columns past b
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          const int64_t i = i0 + 32 * nb + l32;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int64_t j = jw + 32 * mb + 8 * (r >> 2) + (r & 3);
            const bool ok = i < p.rend && j < b && i != j;
            acc[mb][nb][r] = ok ? acc[mb][nb][r] * k2 : ninf;
          }
        }
      fwd_epilogue<true>(p, acc, rowR, rowL, j0, q, rr == 0, k2, wave, lane);
    } else {
      fwd_epilogue<false>(p, acc, rowR, rowL, j0, q, rr == 0, k2, wave, lane);
    }

    // end of a row tile: merge the two lane halves and publish one pair per wave
    if (cc + 1 == ncol) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        float R = rowR[nb], L = rowL[nb];
        lse2_merge(R, L, shfl_xor(rowR[nb], 32), shfl_xor(rowL[nb], 32));
        const int64_t i = i0 + 32 * nb + l32;
        if (h == 0 && i < p.rend) {
          const int64_t slot = (int64_t)(g * 4 + wave) * p.rstride + (i - p.r0);
          p.rowR[slot] = R;
          p.rowL[slot] = L;
        }
        rowR[nb] = ninf;
        rowL[nb] = 0.f;
      }
    }
    rr = nrr;
    cc = ncc;

    if (has_next) {
      wait_dma();
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------- finalize
// Per-sample terms of samples [r0, r0 + n) (all b for the whole batch, a
// shard's own samples otherwise).  Sample r0 + t takes its row pair from the
// nrowpart partials at rowR/rowL[k rstride + t] and its column pair from the
// ncolpart partials at colR/colL[k cstride + t].
struct FinParams {
  int64_t r0, n;
  const float* scale;
  const float* rowR;
  const float* rowL;
  int nrowpart;
  int64_t rstride;
  const float* colR;
  const float* colL;
  int ncolpart;
  int64_t cstride;
  const float* udiag;  // [b], by sample index
  float* lse_r;        // [n]
  float* lse_c;        // [n]
  float* aux;          // [3n]: l^r, l^c, u_ii
  double* partial;     // [gridDim.x]
};

// natural-log log-sum-exp of n base-2 partial pairs (R, l) at R/L[k stride + t].
// Both passes keep eight loads in flight (one load per iteration, each waited
// for, made the merge latency-bound); an empty pair (R = -inf) is weighted by
// zero.  The sum runs in the same order as a plain loop over k.
__device__ __forceinline__ double merge_parts(const float* R, const float* L, int n, int64_t stride, int64_t t) {
  double M = -__builtin_inf();
#pragma unroll 8
  for (int k = 0; k < n; ++k) M = fmax(M, (double)R[(int64_t)k * stride + t]);
  if (M == -__builtin_inf()) return -__builtin_inf();
  double S = 0.0;
  int k = 0;
  for (; k + 8 <= n; k += 8) {  // the eight pairs' loads first, then their terms
    float r[8], l[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      r[u] = R[(int64_t)(k + u) * stride + t];
      l[u] = L[(int64_t)(k + u) * stride + t];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) S += r[u] != -__builtin_inff() ? (double)l[u] * exp2((double)r[u] - M) : 0.0;
  }
  for (; k < n; ++k) {
    const double r = R[(int64_t)k * stride + t];
    const double l = L[(int64_t)k * stride + t];
    S += r != -__builtin_inf() ? l * exp2(r - M) : 0.0;
  }
  return (M + log2(S)) * 0.6931471805599453;  // natural-log LSE over the off-diagonal entries
}

__device__ __forceinline__ double softplus64(double z) {
  if (z == -__builtin_inf()) return 0.0;
  return fmax(z, 0.0) + log1p(exp(-fabs(z)));
}

__global__ void __launch_bounds__(256) fwd_finalize(FinParams p) {
  __shared__ double red[256];
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  double contrib = 0.0;
  if (t < p.n) {
    const double s = (double)p.scale[0];
    const double u = (double)p.udiag[p.r0 + t];
    const double x = s * u;
    const double offr = merge_parts(p.rowR, p.rowL, p.nrowpart, p.rstride, t);
    const double offc = merge_parts(p.colR, p.colL, p.ncolpart, p.cstride, t);
    const double er = softplus64(offr - x);  // r_i - x_ii, cancellation-free
    const double ec = softplus64(offc - x);
    p.lse_r[t] = (float)(x + er);
    p.lse_c[t] = (float)(x + ec);
    p.aux[t] = (float)er;
    p.aux[p.n + t] = (float)ec;
    p.aux[2 * p.n + t] = (float)u;
    contrib = er + ec;
  }
  red[threadIdx.x] = contrib;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) p.partial[blockIdx.x] = red[0];
}

// Sharded forward: one base-2 pair per column j in [0, b) over this shard's
// rows, merged from the ncolpart row-group partials (colR/colL[k b + j]) in a
// fixed order: out[j] = R, out[b + j] = l.  This is what the column owner
// receives from every shard.
__global__ void __launch_bounds__(256) fwd_col_pairs(const float* colR, const float* colL, int ncolpart, int64_t b,
                                                     float* out) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= b) return;
  float M = -__builtin_inff();
  for (int k = 0; k < ncolpart; ++k) M = fmaxf(M, colR[(int64_t)k * b + j]);
  double S = 0.0;
  if (M != -__builtin_inff())
    for (int k = 0; k < ncolpart; ++k) {
      const float r = colR[(int64_t)k * b + j];
      if (r != -__builtin_inff()) S += (double)colL[(int64_t)k * b + j] * exp2((double)r - (double)M);
    }
  out[j] = M;
  out[b + j] = (float)S;
}

// Fixed-order sum of `n` fp64 partials, times `mul`; one workgroup.
__global__ void __launch_bounds__(256) sum_partials(const double* part, int64_t n, double mul, float* out32,
                                                    double* out64) {
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
    double v = red[0] * mul;
    if (out32) *out32 = (float)v;
    if (out64) *out64 = v;
  }
}

// ------------------------------------------------------------ host launchers
bool fwd2_supported(int64_t d, int dtype);
void fwd2_grid(int64_t b, int64_t nrows, int64_t d, int* Pr, int* Pc);
int launch_fwd2(const void* img, const void* txt, int64_t b, int64_t d, int dtype, int64_t r0, int64_t nrows,
                const float* scale, float* rowR, float* rowL, float* colR, float* colL, float* udiag, float* ref2,
                hipStream_t stream);

// Grid of the streamed-tiles sweep for nrows own rows against b columns: Pc
// column groups (one per XCD when there are enough column tiles) times Pr row
// groups, about two workgroups per compute unit.
void fwd1_grid(int64_t b, int64_t nrows, int* Pr, int* Pc) {
  const int64_t nRT = (nrows + kFwdBI - 1) / kFwdBI, nCT = (b + kFwdBJ - 1) / kFwdBJ;
  *Pc = (int)(nCT < 8 ? nCT : 8);
  *Pr = (int)(nRT < 64 ? nRT : 64);
}

static int launch_fwd1(const void* img, const void* txt, int64_t b, int64_t d, int dtype, int64_t r0, int64_t nrows,
                       const float* scale, hipStream_t stream, float* rowR, float* rowL, float* colR, float* colL,
                       float* udiag, int* nrowpart, int* ncolpart) {
  FwdParams p;
  p.img = img;
  p.txt = txt;
  p.b = b;
  p.d = d;
  p.scale = scale;
  p.rowR = rowR;
  p.rowL = rowL;
  p.colR = colR;
  p.colL = colL;
  p.udiag = udiag;
  fwd1_grid(b, nrows, &p.Pr, &p.Pc);
  p.nRT = (int)((nrows + kFwdBI - 1) / kFwdBI);
  p.nCT = (int)((b + kFwdBJ - 1) / kFwdBJ);
  p.r0 = r0;
  p.rend = r0 + nrows;
  p.rstride = nrows;
  *nrowpart = p.Pc * 4;
  *ncolpart = p.Pr;
  if (dtype != 1) return 2;  // every supported 16-bit width takes the resident-rows sweep
  hipLaunchKernelGGL(fwd_sweep, dim3(p.Pr * p.Pc), dim3(256), 0, stream, p);
  return hipGetLastError() == hipSuccess ? 0 : 1;
}

// The sweep over own rows [r0, r0 + nrows) against all b columns: 16-bit
// inputs with d a multiple of 128 up to 1024 take the resident-rows sweep, everything else the
// streamed-tiles sweep above.  Both leave partial pairs: nrowpart per own row
// (stride nrows, by row - r0) and ncolpart per column (stride b).
static int launch_sweep(const void* img, const void* txt, int64_t b, int64_t d, int dtype, int64_t r0, int64_t nrows,
                        const float* scale, float* rowR, float* rowL, float* colR, float* colL, float* udiag,
                        float* ref2, hipStream_t stream, int* nrowpart, int* ncolpart) {
  if (fwd2_supported(d, dtype)) {
    int Pr2 = 0, Pc2 = 0;
    fwd2_grid(b, nrows, d, &Pr2, &Pc2);
    *nrowpart = Pc2;
    *ncolpart = Pr2;
    return launch_fwd2(img, txt, b, d, dtype, r0, nrows, scale, rowR, rowL, colR, colL, udiag, ref2, stream);
  }
  return launch_fwd1(img, txt, b, d, dtype, r0, nrows, scale, stream, rowR, rowL, colR, colL, udiag, nrowpart,
                     ncolpart);
}

// Row partial count of the sweep over nrows own rows (what the finalize of a
// shard has to merge).
int sweep_rowparts(int64_t b, int64_t d, int dtype, int64_t nrows) {
  int Pr = 0, Pc = 0;
  if (fwd2_supported(d, dtype)) {
    fwd2_grid(b, nrows, d, &Pr, &Pc);
    return Pc;
  }
  fwd1_grid(b, nrows, &Pr, &Pc);
  return Pc * 4;
}

static int launch_finalize(int64_t r0, int64_t n, double loss_mul, const float* scale, float* loss, double* loss64,
                           float* lse_r, float* lse_c, float* aux, const float* rowR, const float* rowL, int nrowpart,
                           int64_t rstride, const float* colR, const float* colL, int ncolpart, int64_t cstride,
                           const float* udiag, double* partial, hipStream_t stream) {
  FinParams f;
  f.r0 = r0;
  f.n = n;
  f.scale = scale;
  f.rowR = rowR;
  f.rowL = rowL;
  f.nrowpart = nrowpart;
  f.rstride = rstride;
  f.colR = colR;
  f.colL = colL;
  f.ncolpart = ncolpart;
  f.cstride = cstride;
  f.udiag = udiag;
  f.lse_r = lse_r;
  f.lse_c = lse_c;
  f.aux = aux;
  f.partial = partial;
  int nfin = (int)((n + 255) / 256);
  hipLaunchKernelGGL(fwd_finalize, dim3(nfin), dim3(256), 0, stream, f);
  if (hipGetLastError() != hipSuccess) return 1;
  hipLaunchKernelGGL(sum_partials, dim3(1), dim3(256), 0, stream, (const double*)partial, (int64_t)nfin, loss_mul,
                     loss, loss64);
  return hipGetLastError() == hipSuccess ? 0 : 1;
}

// Forward over the whole batch: the sweep over all rows, then the finalize of
// every sample and the loss.
int launch_fwd(const void* img, const void* txt, int64_t b, int64_t d, int dtype, const float* scale, float* loss,
               double* loss64, float* lse_r, float* lse_c, float* aux, hipStream_t stream, float* rowR, float* rowL,
               float* colR, float* colL, float* udiag, float* ref2, double* partial) {
  int nrowpart = 0, ncolpart = 0;
  const int rc =
      launch_sweep(img, txt, b, d, dtype, 0, b, scale, rowR, rowL, colR, colL, udiag, ref2, stream, &nrowpart, &ncolpart);
  if (rc != 0) return rc;
  return launch_finalize(0, b, 1.0 / (2.0 * (double)b), scale, loss, loss64, lse_r, lse_c, aux, rowR, rowL, nrowpart,
                         b, colR, colL, ncolpart, b, udiag, partial, stream);
}

// Sharded forward, local part: the sweep over own rows [r0, r0 + nrows), row
// partials left in the workspace, and one base-2 pair per column over the own
// rows written to colpair ([2b]: R then l).
int launch_fwd_shard(const void* img, const void* txt, int64_t b, int64_t d, int dtype, int64_t r0, int64_t nrows,
                     const float* scale, float* colpair, hipStream_t stream, float* rowR, float* rowL, float* colR,
                     float* colL, float* udiag, float* ref2) {
  int nrowpart = 0, ncolpart = 0;
  const int rc = launch_sweep(img, txt, b, d, dtype, r0, nrows, scale, rowR, rowL, colR, colL, udiag, ref2, stream,
                              &nrowpart, &ncolpart);
  if (rc != 0) return rc;
  hipLaunchKernelGGL(fwd_col_pairs, dim3((unsigned)((b + 255) / 256)), dim3(256), 0, stream, (const float*)colR,
                     (const float*)colL, ncolpart, b, colpair);
  return hipGetLastError() == hipSuccess ? 0 : 1;
}

// Sharded forward, owner part: the per-sample terms of own samples [r0, r0 +
// nrows) from the row partials of launch_fwd_shard and the nparts column pairs
// received for the own columns (colpairs: [nparts][2 nrows], R then l), and
// this shard's share of the loss, sum of (l^r + l^c) / (2b), into loss_part.
int launch_fwd_shard_finish(int64_t b, int64_t d, int dtype, int64_t r0, int64_t nrows, int64_t nparts,
                            const float* colpairs, const float* scale, float* lse_r, float* lse_c, float* aux,
                            double* loss_part, hipStream_t stream, const float* rowR, const float* rowL,
                            const float* udiag, double* partial) {
  const int nrowpart = sweep_rowparts(b, d, dtype, nrows);
  return launch_finalize(r0, nrows, 1.0 / (2.0 * (double)b), scale, nullptr, loss_part, lse_r, lse_c, aux, rowR, rowL,
                         nrowpart, nrows, colpairs, colpairs + nrows, (int)nparts, 2 * nrows, udiag, partial, stream);
}

}  // namespace infcl
