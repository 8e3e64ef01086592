// Host-side check of the swept-tile index arithmetic of the sweeps, run on
// the CPU by tests/test_layout.py (no GPU needed: nothing here launches).
//
// Every swept tile (32 rows x rowg bytes) reaches LDS through the DMA
// instructions described in sweep.hpp and is read back by the first
// product's fragment reads and the backward's transposing reads.  The check
// simulates the DMA with the kernels' own offset helpers, recording which
// source byte lands on each LDS byte, and then asks of every read the
// kernels issue whether it fetches the rows and features that its MFMA
// operand needs (written out below from the operand layouts of
// v_mfma_f32_32x32x16_{bf16,f16} and ds_read_b64_tr_b16, independently of
// the helpers).  It also checks bounds, that the DMA is a bijection, the
// G' block offsets, and that the reads are bank-conflict free.
#include "sweep.hpp"

#include <cstdio>
#include <vector>

using namespace infcl;

static int g_fail = 0;
#define CHECK(cond, ...)                         \
  do {                                           \
    if (!(cond)) {                               \
      if (g_fail++ < 20) {                       \
        fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
        fprintf(stderr, __VA_ARGS__);            \
        fputc('\n', stderr);                     \
      }                                          \
    }                                            \
  } while (0)

// LDS byte -> source byte of the tile (row * rowg + byte), -1 if unwritten
static std::vector<long> simulate_dma(int rowg) {
  const int tileb = kSweepBN * rowg;
  const int niw = tileb / 4096;  // 1 KiB instructions per wave (4 waves)
  std::vector<long> owner(tileb, -1);
  std::vector<int> src_hits(tileb, 0);
  CHECK(tileb % 4096 == 0, "rowg %d: tile of %d bytes is not 4 waves x whole 1 KiB instructions", rowg, tileb);
  for (int w = 0; w < 4; ++w)
    for (int kk = 0; kk < niw; ++kk)
      for (int L = 0; L < 64; ++L) {
        const long src = (long)sweep_dma_lane_off(L, w, rowg) + sweep_dma_kk_off(kk, w, rowg);
        const long dst = 1024L * (w + 4 * kk) + 16L * L;  // lane L's 16 bytes of the instruction
        CHECK(src % 16 == 0 && src >= 0 && src + 16 <= tileb, "rowg %d: DMA source %ld out of the tile", rowg, src);
        CHECK(dst + 16 <= tileb, "rowg %d: DMA destination %ld out of the buffer", rowg, dst);
        if (src < 0 || src + 16 > tileb || dst + 16 > tileb) continue;
        for (int i = 0; i < 16; ++i) {
          CHECK(owner[dst + i] < 0, "rowg %d: LDS byte %ld written twice", rowg, dst + i);
          owner[dst + i] = src + i;
          src_hits[src + i]++;
        }
      }
  for (int i = 0; i < tileb; ++i) {
    CHECK(owner[i] >= 0, "rowg %d: LDS byte %d never written", rowg, i);
    CHECK(src_hits[i] == 1, "rowg %d: source byte %d fetched %d times", rowg, i, src_hits[i]);
    if (g_fail > 20) break;
  }
  return owner;
}

// First product, 16-bit inputs: MFMA row m of lane L (m = L & 31) holds
// swept row perm(m) ^ rx, and contraction step n takes features
// 16 n + 8 (L >> 5) .. +7 of it, i.e. bytes 32 n + 16 (L >> 5) .. +15.
// The kernels read it at kSeg (n >> 3) + sweep_seg_off(row, 2 (n & 7) + h).
static void check_fragments16(int rowg, const std::vector<long>& owner) {
  const int ks = rowg / 32;  // contraction steps of 16 features
  for (int rx = 0; rx <= 16; rx += 16)
    for (int n = 0; n < ks; ++n) {
      int bank_use[4][16] = {};
      for (int L = 0; L < 64; ++L) {
        const int h = L >> 5;
        const int row = sweep_perm(L & 31) ^ rx;
        const int addr = kSeg * (n >> 3) + sweep_seg_off(row, 2 * (n & 7) + h);
        CHECK(addr >= 0 && addr + 16 <= (int)owner.size(), "rowg %d: fragment read %d out of the buffer", rowg, addr);
        if (addr < 0 || addr + 16 > (int)owner.size()) continue;
        const long want = (long)row * rowg + 32L * n + 16L * h;
        for (int i = 0; i < 16; ++i)
          CHECK(owner[addr + i] == want + i, "rowg %d rx %d n %d lane %d: fragment byte %d holds %ld, wants %ld", rowg,
                rx, n, L, i, owner[addr + i], want + i);
        bank_use[L >> 4][(addr >> 4) & 15]++;  // 16 lanes per cycle, 16 bytes each
      }
      for (int g = 0; g < 4; ++g)
        for (int b = 0; b < 16; ++b)
          CHECK(bank_use[g][b] == 1, "rowg %d rx %d n %d: lanes %d..%d conflict on bank group %d", rowg, rx, n, 16 * g,
                16 * g + 15, b);
    }
  // MFMA row m <-> swept row perm(m): accumulator register 8 s + t of lane
  // half h (row 8 (r >> 2) + 4 h + (r & 3) of the 32x32 result, r = 8 s + t)
  // is swept row 16 s + 8 h + t.
  for (int h = 0; h < 2; ++h)
    for (int r = 0; r < 16; ++r) {
      const int m = 8 * (r >> 2) + 4 * h + (r & 3);
      CHECK(sweep_perm(m) == 16 * (r >> 3) + 8 * h + (r & 7), "perm(%d) = %d", m, sweep_perm(m));
    }
}

// First product, fp32 inputs: ring slot k of a segment reads chunk
// 4 (k >> 1) + 2 h + (k & 1) of the lane's row; over both lane halves and
// the 8 slots every chunk of the segment is read exactly once.
static void check_fragments32(int rowg, const std::vector<long>& owner) {
  const int nseg = rowg / 256;
  for (int seg = 0; seg < nseg; ++seg)
    for (int m = 0; m < 32; ++m) {
      const int row = sweep_perm(m);
      int hit[16] = {};
      for (int h = 0; h < 2; ++h)
        for (int k = 0; k < 8; ++k) {
          const int cl = 4 * (k >> 1) + 2 * h + (k & 1);
          const int addr = kSeg * seg + sweep_seg_off(row, cl);
          CHECK(addr >= 0 && addr + 16 <= (int)owner.size(), "rowg %d: fp32 fragment read out of the buffer", rowg);
          if (addr < 0 || addr + 16 > (int)owner.size()) continue;
          const long got = owner[addr];
          CHECK(got / rowg == row && got % 16 == 0 && (got % rowg) / 256 == seg,
                "rowg %d: fp32 fragment of row %d, segment %d reads row %ld, byte %ld", rowg, row, seg, got / rowg,
                got % rowg);
          for (int i = 1; i < 16; ++i) CHECK(owner[addr + i] == got + i, "rowg %d: fp32 fragment not one chunk", rowg);
          hit[(got % 256) / 16]++;
        }
      for (int c = 0; c < 16; ++c) CHECK(hit[c] == 1, "rowg %d row %d seg %d: chunk %d read %d times", rowg, row, seg, c, hit[c]);
    }
  // the fp32 second product reads single floats at sweep_chunk_off
  for (int r = 0; r < 32; ++r)
    for (int c = 0; c < rowg / 16; ++c) {
      const int addr = sweep_chunk_off(r, c);
      CHECK(owner[addr] == (long)r * rowg + 16L * c, "rowg %d: chunk %d of row %d at %d holds %ld", rowg, c, r, addr,
            owner[addr]);
    }
}

// Second product (backward), transposing reads: for row group tt of feature
// block fb and contraction half s2, lane L reads swept row
// 16 s2 + 8 (L >> 5) + 4 tt + ((L & 15) >> 2), features
// 32 fb + 16 ((L >> 4) & 1) + 4 (L & 3) .. +3 (8 bytes).
static void check_transposing(int rowg, const std::vector<long>& owner) {
  const int nfb = rowg / 64;  // 32-feature blocks of 16-bit values
  for (int fb = 0; fb < nfb; ++fb)
    for (int tt = 0; tt < 2; ++tt)
      for (int s2 = 0; s2 < 2; ++s2) {
        int bank_use[2][32] = {};
        for (int L = 0; L < 64; ++L) {
          const int addr = sweep_tr_off(L, tt, fb) + 16 * kSegRow * s2;
          CHECK(addr >= 0 && addr % 8 == 0 && addr + 8 <= (int)owner.size(), "rowg %d: transposing read %d", rowg, addr);
          if (addr < 0 || addr + 8 > (int)owner.size()) continue;
          const int row = 16 * s2 + 8 * (L >> 5) + 4 * tt + ((L & 15) >> 2);
          const long want = (long)row * rowg + 64L * fb + 32L * ((L >> 4) & 1) + 8L * (L & 3);
          for (int i = 0; i < 8; ++i)
            CHECK(owner[addr + i] == want + i, "rowg %d fb %d tt %d s2 %d lane %d: byte %d holds %ld, wants %ld", rowg, fb,
                  tt, s2, L, i, owner[addr + i], want + i);
          bank_use[L >> 5][(addr >> 3) & 31]++;  // 32 lanes per cycle, 8 bytes each
        }
        for (int g = 0; g < 2; ++g)
          for (int b = 0; b < 32; ++b)
            CHECK(bank_use[g][b] == 1, "rowg %d fb %d tt %d s2 %d: half-wave %d conflicts on bank pair %d", rowg, fb, tt,
                  s2, g, b);
      }
}

// G' block: 64 own rows x 4 chunks (8 swept columns each), every chunk at
// its own place inside 4 KiB; own block o adds 2048 o (the swizzle depends
// on row bits 2..3 only); each 16-lane group of a fragment read is conflict
// free.
static void check_gp_block() {
  std::vector<int> hit(4096, 0);
  for (int row = 0; row < 64; ++row)
    for (int c = 0; c < 4; ++c) {
      const int a = gp_chunk_off(row, c);
      CHECK(a >= 0 && a % 16 == 0 && a + 16 <= 4096, "G' chunk (%d, %d) at %d", row, c, a);
      if (a < 0 || a + 16 > 4096) continue;
      for (int i = 0; i < 16; ++i) hit[a + i]++;
      CHECK(a == 2048 * (row >> 5) + gp_chunk_off(row & 31, c), "G' row %d: block offset", row);
    }
  for (int i = 0; i < 4096; ++i) CHECK(hit[i] == 1, "G' byte %d covered %d times", i, hit[i]);
  for (int s2 = 0; s2 < 2; ++s2) {
    int bank_use[4][16] = {};
    for (int L = 0; L < 64; ++L) bank_use[L >> 4][(gp_chunk_off(L & 31, 2 * s2 + (L >> 5)) >> 4) & 15]++;
    for (int g = 0; g < 4; ++g)
      for (int b = 0; b < 16; ++b)
        CHECK(bank_use[g][b] <= 1, "G' read s2 %d: lanes %d..%d conflict on bank group %d", s2, 16 * g, 16 * g + 15, b);
  }
}

int main() {
  int shapes = 0;
  for (int rowg = 256; rowg <= 2048; rowg += 256) {  // 16-bit d = 128..1024, fp32 d = 64..512
    const std::vector<long> owner = simulate_dma(rowg);
    check_fragments16(rowg, owner);
    check_fragments32(rowg, owner);
    check_transposing(rowg, owner);
    ++shapes;
  }
  check_gp_block();
  if (g_fail) {
    fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  printf("layout ok (%d row widths)\n", shapes);
  return 0;
}
