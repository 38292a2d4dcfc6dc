// bf16 MFMA GEMM building blocks for gfx950: tile loaders into LDS, the
// 32x32x16 fragment loop and accumulator walkers.
//
// LDS tile format (both operands): [ROWS][64] bf16, K contiguous, where ROWS
// runs over M (operand A) or N (operand B) and 64 = BK.  Each 16-byte chunk c
// of row R is stored at chunk position c ^ swz(R), swz(R) = (R ^ (R >> 3)) & 7,
// so that the MFMA fragment reads (8 consecutive rows, same chunk) and the
// loader writes hit distinct LDS banks.
#pragma once
#include "common.hpp"
#include "pstream.hpp"

namespace compact {

constexpr int kBK = 64;  // K extent of one LDS tile

__device__ __forceinline__ int swz(int row) { return (row ^ (row >> 3)) & 7; }

// Element offset of (row, k) in a swizzled [ROWS][64] tile; k is a multiple of 4
// when used for 8-byte stores and of 8 for 16-byte accesses.
__device__ __forceinline__ int tile_off(int row, int k) {
  return row * kBK + (((k >> 3) ^ swz(row)) << 3) + (k & 7);
}

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// Keeps the first cnt (0..8) bf16 elements of a 16-byte chunk, zeroes the rest.
__device__ __forceinline__ u32x4 keep_first(u32x4 v, int cnt) {
  const uint32_t m0 = cnt >= 2 ? 0xFFFFFFFFu : (cnt == 1 ? 0x0000FFFFu : 0u);
  const uint32_t m1 = cnt >= 4 ? 0xFFFFFFFFu : (cnt == 3 ? 0x0000FFFFu : 0u);
  const uint32_t m2 = cnt >= 6 ? 0xFFFFFFFFu : (cnt == 5 ? 0x0000FFFFu : 0u);
  const uint32_t m3 = cnt >= 8 ? 0xFFFFFFFFu : (cnt == 7 ? 0x0000FFFFu : 0u);
  v.x &= m0;
  v.y &= m1;
  v.z &= m2;
  v.w &= m3;
  return v;
}

// Loads are branch-free: a tile that lies wholly inside the matrix (a
// workgroup-uniform test) uses plain 16-byte loads; an edge tile clamps each
// chunk address into the matrix and zeroes the elements outside it.  Chunks
// are 8-element aligned, so a chunk that starts inside a row may read up to 7
// elements past the row's last column (never past round_up(cols, 8) <= ld).

// ---------------------------------------------------------------------------
// Operand stored K-contiguous in global memory: element (row, k) at
// base[row * ld + k], rows < rows_total, k < K.  Used for x and dL/do
// (A operands) and for W in dx = dL/do W^T (B operand).
// ---------------------------------------------------------------------------
template <int ROWS, int NT>
struct KMajorLoader {
  static constexpr int kCpr = kBK / 8;
  static constexpr int kPer = ROWS * kCpr / NT;
  static_assert(ROWS * kCpr % NT == 0, "tile does not split evenly over threads");
  const uint16_t* base;
  int64_t ld, rows_total, K, row0;
  u32x4 reg[kPer];

  __device__ __forceinline__ void fetch(int64_t k0, int tid) {
    if (row0 + ROWS <= rows_total && k0 + kBK <= K) {
#pragma unroll
      for (int p = 0; p < kPer; ++p) {
        const int c = tid + p * NT;
        const int row = c / kCpr, kc = c % kCpr;
        reg[p] = load16(base + (row0 + row) * ld + k0 + kc * 8);
      }
    } else {
      const int64_t k_last = (K - 1) & ~int64_t(7);
#pragma unroll
      for (int p = 0; p < kPer; ++p) {
        const int c = tid + p * NT;
        const int row = c / kCpr, kc = c % kCpr;
        const int64_t gr = row0 + row, gk = k0 + kc * 8;
        const bool row_ok = gr < rows_total;
        const int64_t rc = row_ok ? gr : rows_total - 1;
        const int64_t kcl = gk < K ? gk : k_last;
        const int64_t left = K - gk;
        const int cnt = !row_ok || left <= 0 ? 0 : (left >= 8 ? 8 : static_cast<int>(left));
        reg[p] = keep_first(load16(base + rc * ld + kcl), cnt);
      }
    }
  }
  __device__ __forceinline__ void commit(uint16_t* lds, int tid) const {
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int c = tid + p * NT;
      const int row = c / kCpr, kc = c % kCpr;
      *reinterpret_cast<u32x4*>(lds + tile_off(row, kc * 8)) = reg[p];
    }
  }
};

// ---------------------------------------------------------------------------
// Operand stored MN-contiguous: element (row, k) at base[k * ld + row]
// (global matrix [K][rows]).  Loaded as 4(k) x 8(row) blocks and transposed
// in registers.  Used for W in the forward (B[k=i][n=c] = W[i][c]) and for
// z and dL/do in G^ = z^T dL/do.
// ---------------------------------------------------------------------------
template <int ROWS, int NT>
struct MNMajorLoader {
  static constexpr int kRowBlocks = ROWS / 8;
  static constexpr int kBlocks = (kBK / 4) * kRowBlocks;
  static constexpr int kPer = kBlocks / NT;
  static_assert(kBlocks % NT == 0, "tile does not split evenly over threads");
  const uint16_t* base;
  int64_t ld, rows_total, K, row0;
  u32x4 reg[kPer][4];

  __device__ __forceinline__ void fetch(int64_t k0, int tid) {
    if (row0 + ROWS <= rows_total && k0 + kBK <= K) {
#pragma unroll
      for (int p = 0; p < kPer; ++p) {
        const int b = tid + p * NT;
        const int rb = b % kRowBlocks, kb = b / kRowBlocks;
        const uint16_t* src = base + (k0 + kb * 4) * ld + row0 + rb * 8;
#pragma unroll
        for (int q = 0; q < 4; ++q) reg[p][q] = load16(src + q * ld);
      }
    } else {
      const int64_t r_last = (rows_total - 1) & ~int64_t(7);
#pragma unroll
      for (int p = 0; p < kPer; ++p) {
        const int b = tid + p * NT;
        const int rb = b % kRowBlocks, kb = b / kRowBlocks;
        const int64_t gr = row0 + rb * 8;
        const int64_t rcl = gr < rows_total ? gr : r_last;
        const int64_t left = rows_total - gr;
        const int cnt_r = left <= 0 ? 0 : (left >= 8 ? 8 : static_cast<int>(left));
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int64_t gk = k0 + kb * 4 + q;
          const bool k_ok = gk < K;
          const int64_t kcl = k_ok ? gk : K - 1;
          reg[p][q] = keep_first(load16(base + kcl * ld + rcl), k_ok ? cnt_r : 0);
        }
      }
    }
  }
  __device__ __forceinline__ void commit(uint16_t* lds, int tid) const {
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int b = tid + p * NT;
      const int rb = b % kRowBlocks, kb = b / kRowBlocks;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        u32x2 lo, hi;
        lo.x = __builtin_amdgcn_perm(reg[p][1][e], reg[p][0][e], 0x05040100u);
        lo.y = __builtin_amdgcn_perm(reg[p][3][e], reg[p][2][e], 0x05040100u);
        hi.x = __builtin_amdgcn_perm(reg[p][1][e], reg[p][0][e], 0x07060302u);
        hi.y = __builtin_amdgcn_perm(reg[p][3][e], reg[p][2][e], 0x07060302u);
        const int r = rb * 8 + 2 * e;
        *reinterpret_cast<u32x2*>(lds + tile_off(r, kb * 4)) = lo;
        *reinterpret_cast<u32x2*>(lds + tile_off(r + 1, kb * 4)) = hi;
      }
    }
  }
};

// ---------------------------------------------------------------------------
// Projection tile generated on the fly (B operand of z = x P, K = i, N = j):
// LDS row j holds G[k0 .. k0+63][j] as bf16.  One Philox call gives the four
// consecutive rows i = 4p .. 4p+3 of column j, i.e. one 8-byte LDS store.
// identity != 0 gives P = I instead (r == n).
// ---------------------------------------------------------------------------
template <int ROWS, int NT>
struct PGenLoader {
  static constexpr int kQuadsPerRow = kBK / 4;
  static constexpr int kQuads = ROWS * kQuadsPerRow;
  static_assert(kQuads % NT == 0, "tile does not split evenly over threads");
  PhiloxKey key;
  int64_t n, r, col0;  // K extent n, N extent r, first column of the tile
  int identity;
  int64_t k_next;

  // Generation happens in commit(), straight into the LDS buffer that is not
  // being read, so that its VALU work follows the MFMAs of the current tile.
  __device__ __forceinline__ void fetch(int64_t k0, int) { k_next = k0; }
  __device__ __forceinline__ void commit(uint16_t* lds, int tid) const {
#pragma unroll 1
    for (int c = tid; c < kQuads; c += NT) {
      const int row = c / kQuadsPerRow, kq = c % kQuadsPerRow;
      const int64_t j = col0 + row, i0 = k_next + kq * 4;
      float g[4] = {0.f, 0.f, 0.f, 0.f};
      if (j < r && i0 < n) {
        if (identity) {
#pragma unroll
          for (int e = 0; e < 4; ++e) g[e] = (i0 + e == j) ? 1.0f : 0.0f;
        } else {
          pstream_quad(key, static_cast<uint32_t>(i0 >> 2), static_cast<uint32_t>(j), g);
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (i0 + e >= n) g[e] = 0.0f;
        }
      }
      u32x2 v;
      v.x = pack_bf16x2(g[0], g[1]);
      v.y = pack_bf16x2(g[2], g[3]);
      *reinterpret_cast<u32x2*>(lds + tile_off(row, kq * 4)) = v;
    }
  }
};

// ---------------------------------------------------------------------------
// Fragment loop over one 64-deep LDS tile pair.
// ---------------------------------------------------------------------------
template <int FM, int FN>
__device__ __forceinline__ void mma_tile(const uint16_t* As, const uint16_t* Bs, int a_row0,
                                         int b_row0, int lane, f32x16 (&acc)[FM][FN]) {
  const int lr = lane & 31, lh = lane >> 5;
#pragma unroll
  for (int kk = 0; kk < kBK / 16; ++kk) {
    u32x4 a[FM], b[FN];
    const int k = kk * 16 + lh * 8;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int row = a_row0 + fm * 32 + lr;
      a[fm] = *reinterpret_cast<const u32x4*>(As + tile_off(row, k));
    }
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int row = b_row0 + fn * 32 + lr;
      b[fn] = *reinterpret_cast<const u32x4*>(Bs + tile_off(row, k));
    }
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma32x32x16(a[fm], b[fn], acc[fm][fn]);
  }
}

// Calls f(row, col, value) for every accumulator element of the wave tile,
// with row/col relative to the wave tile origin.
template <int FM, int FN, class F>
__device__ __forceinline__ void for_each_acc(const f32x16 (&acc)[FM][FN], int lane, F&& f) {
  const int lr = lane & 31, lh = lane >> 5;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = fm * 32 + (v >> 2) * 8 + lh * 4 + (v & 3);
        const int col = fn * 32 + lr;
        f(row, col, acc[fm][fn][v]);
      }
}

// Generic double-buffered main loop: C(BM x BN) += A(BM x K) B(K x BN) with
// A and B staged through swizzled LDS tiles by the given loaders.
template <int BM, int BN, int WGM, int WGN, class LA, class LB>
__device__ __forceinline__ void gemm_mainloop(LA& la, LB& lb, int64_t k_begin, int64_t k_end,
                                              uint16_t* lds, f32x16 (&acc)[BM / WGM / 32][BN / WGN / 32]) {
  constexpr int NT = WGM * WGN * kWave;
  constexpr int FM = BM / WGM / 32, FN = BN / WGN / 32;
  constexpr int kAElems = BM * kBK, kBElems = BN * kBK;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  // Stage s holds A at lds + s * kStage and B right after it.  Offsets (not a
  // pointer array) keep every access in the LDS address space.
  constexpr int kStage = kAElems + kBElems;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[fm][fn][v] = 0.0f;
  const int64_t kt_count = ceil_div(k_end - k_begin, kBK);
  if (kt_count <= 0) return;
  la.fetch(k_begin, tid);
  lb.fetch(k_begin, tid);
  la.commit(lds, tid);
  lb.commit(lds + kAElems, tid);
  __syncthreads();
  for (int64_t kt = 0; kt < kt_count; ++kt) {
    const int cur = static_cast<int>(kt & 1) * kStage;
    const int nxt = kStage - cur;
    const bool more = kt + 1 < kt_count;
    if (more) {
      la.fetch(k_begin + (kt + 1) * kBK, tid);
      lb.fetch(k_begin + (kt + 1) * kBK, tid);
    }
    mma_tile<FM, FN>(lds + cur, lds + cur + kAElems, wm * FM * 32, wn * FN * 32, lane, acc);
    if (more) {
      la.commit(lds + nxt, tid);
      lb.commit(lds + nxt + kAElems, tid);
    }
    __syncthreads();
  }
}

}  // namespace compact
