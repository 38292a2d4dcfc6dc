// Direct-to-LDS GEMM core for gfx950.
//
// Global tiles are copied into LDS with global_load_lds_dwordx4: one wave
// instruction moves 64 x 16 bytes, lane L's chunk landing at M0 + 16 L.  No
// VGPR staging and no ds_write; the per-lane global address chooses which
// chunk lands where, which is how the LDS swizzles below are applied.
//
// Operand kinds
//   K-major  [ROWS][64] bf16 tile, chunk c of row R at position c ^ swz(R)
//            (the same layout as the register-staged path); fragments are
//            single ds_read_b128.
//   MN-major [64][ROWS] bf16 tile (k-rows, contiguous along M or N); 16-byte
//            chunk c of k-row k at position c ^ (2 (k mod 4)); fragments are
//            two ds_read_b64_tr_b16.  In a 16-lane group, that instruction
//            hands output lane t, element j, the element t mod 4 of source
//            lane 4 j + t / 4; with source lane 4 j + q pointing at
//            tile[k0 + j][n0 + 4 q], lane t receives tile[k0 .. k0 + 3][n0 + t].
//
// Edges.  Rows past the matrix in M or N are clamped to the last row (they only
// feed outputs that are never stored).  Chunks past K read a 16-byte zero page,
// so the K sum is exact; this needs K % 8 == 0 for K-major operands (a chunk
// never straddles K).  Callers fall back to the register-staged path otherwise.
#pragma once
#include "gemm_bf16.hpp"

namespace compact {

__device__ __attribute__((aligned(16))) const uint32_t g_zero16[4] = {0u, 0u, 0u, 0u};

typedef __attribute__((address_space(3))) void lds_void_t;

// LDS byte address of the dynamic shared buffer (it follows static LDS).
__device__ __forceinline__ uint32_t dyn_lds_base() { return __builtin_amdgcn_groupstaticsize(); }

__device__ __forceinline__ void dtl16(const void* g, uint32_t lds_byte) {
  __builtin_amdgcn_global_load_lds(g, reinterpret_cast<lds_void_t*>(static_cast<uintptr_t>(lds_byte)), 16, 0, 0);
}

// s_waitcnt vmcnt(N) with the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// ---------------------------------------------------------------------------
// K-major operand, DTL.  ROWS x 64 tile = ROWS / 8 wave instructions.
// ---------------------------------------------------------------------------
template <int ROWS, int NWAVES>
struct KMajorDTL {
  static constexpr int kInstr = ROWS / 8;             // 1 KB blocks per tile
  static constexpr int kPerWave = kInstr / NWAVES;
  static_assert(kInstr % NWAVES == 0, "tile does not split evenly over waves");
  const uint16_t* base;
  int64_t ld, rows_total, K, row0;

  // Issue the copy of k-tile [k0, k0 + 64) into the stage at LDS byte `stage`.
  __device__ __forceinline__ void issue(int64_t k0, uint32_t stage, int wave, int lane) const {
#pragma unroll
    for (int i = 0; i < kPerWave; ++i) {
      const int I = wave * kPerWave + i;
      const int row = I * 8 + (lane >> 3);
      const int logical = (lane & 7) ^ swz(row);
      int64_t gr = row0 + row;
      gr = gr < rows_total ? gr : rows_total - 1;
      const int64_t gk = k0 + logical * 8;
      const void* src = gk < K ? static_cast<const void*>(base + gr * ld + gk)
                               : static_cast<const void*>(g_zero16);
      dtl16(src, stage + I * 1024);
    }
  }
  // Pull line `line` (0 .. ROWS - 1, one 128-byte row segment each) of k-tile
  // k0 towards the caches: a 16-byte copy into a scratch LDS slot.
  __device__ __forceinline__ const void* touch_addr(int64_t k0, int line) const {
    int64_t gr = row0 + line;
    gr = gr < rows_total ? gr : rows_total - 1;
    return k0 < K ? static_cast<const void*>(base + gr * ld + k0) : static_cast<const void*>(g_zero16);
  }
  static constexpr int kLines = ROWS;
  static constexpr int kLoadsPerWave = kPerWave;
};

// ---------------------------------------------------------------------------
// MN-major operand, DTL.  Element (row, k) at base[k * ld + row]; the tile is
// 64 k-rows of ROWS elements, stored as k-rows in LDS.
// ---------------------------------------------------------------------------
template <int ROWS, int NWAVES>
struct MNMajorDTL {
  static constexpr int kChunksPerK = ROWS / 8;         // 16-byte chunks per k-row
  static constexpr int kKPerInstr = 64 / kChunksPerK;  // k-rows per 1 KB block
  static constexpr int kInstr = 64 / kKPerInstr;
  static constexpr int kPerWave = kInstr / NWAVES;
  static_assert(ROWS >= 64 && ROWS <= 512, "MN-major tile width");
  static_assert(kInstr % NWAVES == 0, "tile does not split evenly over waves");
  const uint16_t* base;
  int64_t ld, rows_total, K, row0;

  __device__ __forceinline__ void issue(int64_t k0, uint32_t stage, int wave, int lane) const {
#pragma unroll
    for (int i = 0; i < kPerWave; ++i) {
      const int I = wave * kPerWave + i;
      const int k = I * kKPerInstr + lane / kChunksPerK;
      const int phys = lane % kChunksPerK;
      const int logical = phys ^ (2 * (k & 3));
      int64_t gr = row0 + logical * 8;
      const int64_t r_last = (rows_total - 1) & ~int64_t(7);
      gr = gr < rows_total ? gr : r_last;
      const int64_t gk = k0 + k;
      const void* src = gk < K ? static_cast<const void*>(base + gk * ld + gr)
                               : static_cast<const void*>(g_zero16);
      dtl16(src, stage + I * 1024);
    }
  }
  // 128-byte lines of the tile: 64 k-rows x (ROWS / 64) lines each.
  __device__ __forceinline__ const void* touch_addr(int64_t k0, int line) const {
    constexpr int kLinesPerK = ROWS / 64;
    const int k = line / kLinesPerK, seg = line % kLinesPerK;
    const int64_t gk = k0 + k;
    int64_t gr = row0 + seg * 64;
    const int64_t r_last = (rows_total - 1) & ~int64_t(7);
    gr = gr < rows_total ? gr : r_last;
    return gk < K ? static_cast<const void*>(base + gk * ld + gr) : static_cast<const void*>(g_zero16);
  }
  static constexpr int kLines = 64 * (ROWS / 64);
  static constexpr int kLoadsPerWave = kPerWave;
};

// Fragment readers.  `tile` is the element offset of the operand tile from the
// start of the dynamic LDS buffer (LDS byte address `lbase`).
// K-major: rows row0 .. row0 + 31, k = kk * 16 + 8 (lane / 32) .. + 7.
struct KFrag {
  __device__ __forceinline__ static u32x4 read(const uint16_t* lds, uint32_t, int tile, int row0, int kk,
                                               int lane) {
    const int row = row0 + (lane & 31);
    return *reinterpret_cast<const u32x4*>(lds + tile + tile_off(row, kk * 16 + (lane >> 5) * 8));
  }
};

// MN-major tile of width ROWS: fragment columns n0 .. n0 + 31,
// k = kk * 16 + 8 (lane / 32) .. + 7, via two transposing reads.
template <int ROWS>
struct MNFrag {
  __device__ __forceinline__ static u32x4 read(const uint16_t*, uint32_t lbase, int tile, int n0, int kk,
                                               int lane) {
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    const int g = lane >> 4, s = lane & 15;
    const int j = s >> 2, q = s & 3;
    const int col = n0 + (g & 1) * 16 + q * 4;
    u32x4 out;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int k = kk * 16 + (g >> 1) * 8 + 4 * h + j;
      const int chunk = (col >> 3) ^ (2 * (k & 3));
      const uint32_t off = static_cast<uint32_t>(tile + k * ROWS + chunk * 8 + (col & 7));
      const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          reinterpret_cast<lds_s16x4*>(static_cast<uintptr_t>(lbase + 2u * off)));
      out[2 * h] = static_cast<uint32_t>(static_cast<uint16_t>(v[0])) |
                   (static_cast<uint32_t>(static_cast<uint16_t>(v[1])) << 16);
      out[2 * h + 1] = static_cast<uint32_t>(static_cast<uint16_t>(v[2])) |
                       (static_cast<uint32_t>(static_cast<uint16_t>(v[3])) << 16);
    }
    return out;
  }
};

// One 16-deep MFMA step with operand-specific fragment readers.
template <int FM, int FN, class FA, class FB>
__device__ __forceinline__ void mma_k16_dtl(const uint16_t* lds, uint32_t lbase, int a_tile, int b_tile,
                                            int a_row0, int b_row0, int lane, int kk,
                                            f32x16 (&acc)[FM][FN]) {
  u32x4 a[FM], b[FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) a[fm] = FA::read(lds, lbase, a_tile, a_row0 + fm * 32, kk, lane);
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) b[fn] = FB::read(lds, lbase, b_tile, b_row0 + fn * 32, kk, lane);
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma32x32x16(a[fm], b[fn], acc[fm][fn]);
}

// Direct-to-LDS main loop, two LDS stages plus a cache prefetch:
//   top of step kt: wait until tile kt has landed (this wave's copies; the
//                   prefetch issued after them may still be out), barrier
//                   (every wave's copies; everyone is done with the other stage);
//                   copy tile kt+1 into the other stage;
//                   touch every line of tile kt+2 (one 16-byte copy per line into
//                   a per-wave scratch slot), so the copy of kt+2 hits the cache;
//                   16-deep MFMA steps on stage kt.
// LDS use: 2 stages + 1 KB scratch per wave, after the stages.
template <int BM, int BN, int WGM, int WGN, class LA, class LB, class FA, class FB>
__device__ __forceinline__ void gemm_mainloop_dtl(const LA& la, const LB& lb, int64_t k_begin, int64_t k_end,
                                                  uint16_t* lds, f32x16 (&acc)[BM / WGM / 32][BN / WGN / 32]) {
  constexpr int NW = WGM * WGN;
  constexpr int FM = BM / WGM / 32, FN = BN / WGN / 32;
  constexpr int kAElems = BM * kBK, kBElems = BN * kBK;
  constexpr int kStage = kAElems + kBElems;  // elements
  constexpr int kTouch = (LA::kLines + LB::kLines) / (NW * 64);  // prefetch lines per lane
  static_assert(kTouch * NW * 64 == LA::kLines + LB::kLines, "prefetch lines split evenly over lanes");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const uint32_t lbase = dyn_lds_base();
  const uint32_t scratch = lbase + 2u * static_cast<uint32_t>(2 * kStage) + 1024u * wave;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[fm][fn][v] = 0.0f;
  const int64_t kt_count = ceil_div(k_end - k_begin, kBK);
  if (kt_count <= 0) return;
  auto touch = [&](int64_t kt) {
    const int64_t k0 = k_begin + kt * kBK;
#pragma unroll
    for (int t = 0; t < kTouch; ++t) {
      const int line = (t * NW + wave) * 64 + lane;
      const void* src = line < LA::kLines ? la.touch_addr(k0, line) : lb.touch_addr(k0, line - LA::kLines);
      dtl16(src, scratch);
    }
  };
  la.issue(k_begin, lbase, wave, lane);
  lb.issue(k_begin, lbase + 2u * kAElems, wave, lane);
  if (kt_count > 1) touch(1);
  for (int64_t kt = 0; kt < kt_count; ++kt) {
    // outstanding in issue order: copies of tile kt, then the touches of kt+1
    if (kt + 1 < kt_count) {
      wait_vmcnt<kTouch>();
    } else {
      wait_vmcnt<0>();
    }
    __syncthreads();
    if (kt + 1 < kt_count) {
      const uint32_t st = lbase + 2u * static_cast<uint32_t>(((kt + 1) & 1) * kStage);
      la.issue(k_begin + (kt + 1) * kBK, st, wave, lane);
      lb.issue(k_begin + (kt + 1) * kBK, st + 2u * kAElems, wave, lane);
      if (kt + 2 < kt_count) touch(kt + 2);
    }
    const int sc = static_cast<int>(kt & 1) * kStage;
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk)
      mma_k16_dtl<FM, FN, FA, FB>(lds, lbase, sc, sc + kAElems, wm * FM * 32, wn * FN * 32, lane, kk, acc);
  }
  __syncthreads();  // every wave is done with the stages before an epilogue reuses LDS
}

// LDS bytes the DTL main loop needs.
__host__ __device__ constexpr int dtl_lds_bytes(int bm, int bn, int nwaves) {
  return 2 * 2 * (bm + bn) * 64 + 1024 * nwaves;
}

}  // namespace compact
