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

// Loads are straight-line code: fetch() clamps every chunk address into the
// matrix, issues the load and records how many elements of the chunk are
// valid; commit() zeroes the invalid ones (only on tiles that touch an edge)
// and writes LDS.  Keeping branches out of fetch() lets the compiler wait for
// exactly the loads a commit needs, so loads for later K steps stay in flight.
// Chunks are 8-element aligned, so a chunk that starts inside a row may read up
// to 7 elements past the row's last column (never past round_up(cols, 8) <= ld).

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
  int cnt[kPer];
  bool full;

  __device__ __forceinline__ void fetch(int64_t k0, int tid) {
    full = row0 + ROWS <= rows_total && k0 + kBK <= K;
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
      cnt[p] = !row_ok || left <= 0 ? 0 : (left >= 8 ? 8 : static_cast<int>(left));
      reg[p] = load16(base + rc * ld + kcl);
    }
  }
  __device__ __forceinline__ void commit(uint16_t* lds, int tid) const {
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int c = tid + p * NT;
      const int row = c / kCpr, kc = c % kCpr;
      const u32x4 v = full ? reg[p] : keep_first(reg[p], cnt[p]);
      *reinterpret_cast<u32x4*>(lds + tile_off(row, kc * 8)) = v;
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
  static constexpr int kPer = (kBlocks + NT - 1) / NT;
  static_assert(kBlocks % NT == 0 || kBlocks < NT, "tile does not split evenly over threads");
  static constexpr bool kPartial = kBlocks < NT;  // threads >= kBlocks sit out
  const uint16_t* base;
  int64_t ld, rows_total, K, row0;
  u32x4 reg[kPer][4];
  int cnt[kPer][4];
  bool full;

  __device__ __forceinline__ void fetch(int64_t k0, int tid) {
    full = row0 + ROWS <= rows_total && k0 + kBK <= K;
    if (kPartial && tid >= kBlocks) return;
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
        cnt[p][q] = k_ok ? cnt_r : 0;
        reg[p][q] = load16(base + kcl * ld + rcl);
      }
    }
  }
  __device__ __forceinline__ void commit(uint16_t* lds, int tid) const {
    if (kPartial && tid >= kBlocks) return;
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int b = tid + p * NT;
      const int rb = b % kRowBlocks, kb = b / kRowBlocks;
      u32x4 v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = full ? reg[p][q] : keep_first(reg[p][q], cnt[p][q]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        u32x2 lo, hi;
        lo.x = __builtin_amdgcn_perm(v[1][e], v[0][e], 0x05040100u);
        lo.y = __builtin_amdgcn_perm(v[3][e], v[2][e], 0x05040100u);
        hi.x = __builtin_amdgcn_perm(v[1][e], v[0][e], 0x07060302u);
        hi.y = __builtin_amdgcn_perm(v[3][e], v[2][e], 0x07060302u);
        const int r = rb * 8 + 2 * e;
        *reinterpret_cast<u32x2*>(lds + tile_off(r, kb * 4)) = lo;
        *reinterpret_cast<u32x2*>(lds + tile_off(r + 1, kb * 4)) = hi;
      }
    }
  }
};

// ---------------------------------------------------------------------------
// Projection tile generated on the fly (B operand of z = x P, K = i, N = j):
// LDS row j holds scale x stream elements (k0 .. k0+63, j) as bf16 (scale =
// 1/sqrt(r) for the Gaussian, 1/sqrt(s) for the sparse projection, so the
// tile is P itself, rounded once).  One Philox call gives the four
// consecutive Gaussian rows i = 4p .. 4p+3 of column j, i.e. one 8-byte LDS
// store.  The identity gives P = I (r == n).
// ---------------------------------------------------------------------------
template <int ROWS, int NT>
struct PGenLoader {
  static constexpr int kQuadsPerRow = kBK / 4;
  static constexpr int kQuads = ROWS * kQuadsPerRow;
  static_assert(kQuads % NT == 0, "tile does not split evenly over threads");
  PhiloxKey key;
  int64_t n, r, col0;  // K extent n, N extent r, first column of the tile
  ProjDesc proj;
  float scale;
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
        proj_quad(proj, key, i0, j, g);
        const float sc = proj.kind == kProjIdentity ? 1.0f : scale;
#pragma unroll
        for (int e = 0; e < 4; ++e) g[e] = i0 + e >= n ? 0.0f : g[e] * sc;
      }
      u32x2 v;
      v.x = pack_bf16x2(g[0], g[1]);
      v.y = pack_bf16x2(g[2], g[3]);
      *reinterpret_cast<u32x2*>(lds + tile_off(row, kq * 4)) = v;
    }
  }
};

// ---------------------------------------------------------------------------
// One 16-deep MFMA step over the current LDS stage.
// ---------------------------------------------------------------------------
template <int FM, int FN>
__device__ __forceinline__ void mma_k16(const uint16_t* As, const uint16_t* Bs, int a_row0, int b_row0,
                                        int lane, int kk, f32x16 (&acc)[FM][FN]) {
  const int lr = lane & 31, lh = lane >> 5;
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

// ---------------------------------------------------------------------------
// bf16 tile store through LDS.  Each wave stages its WTM x WTN tile row-major
// in its own LDS region (the GEMM stages are dead once the main loop has
// ended with a barrier), then writes 16-byte chunks so that 16 consecutive
// lanes cover one 256-byte output row.
//
// Staging: an accumulator group (fm, fn, v/4) holds rows R..R+3 of column C in
// one lane.  Lanes 2k and 2k+1 hold columns C and C+1; one DPP swap of a packed
// bf16 pair lets the even lane own rows R, R+1 and the odd lane rows R+2, R+3
// of both columns, so every LDS write is 4 bytes.  Dword d of row `row` sits
// at d ^ (((row >> 1) & 3) << 4), which spreads the four rows one write
// instruction touches over both halves of the banks.
// ---------------------------------------------------------------------------
template <int WTM, int WTN>
__device__ __forceinline__ int stage_dword(int row, int dw) {
  static_assert(WTN % 128 == 0 || WTN == 64, "staging swizzle assumes 64 or 128k columns");
  constexpr int kRowDw = WTN / 2;
  const int sw = WTN >= 128 ? (((row >> 1) & 3) << 4) : (((row >> 1) & 1) << 4);
  return row * kRowDw + (dw ^ sw);
}

template <int BM, int BN, int WGM, int WGN>
__device__ __forceinline__ void store_tile_bf16_lds(const f32x16 (&acc)[BM / WGM / 32][BN / WGN / 32],
                                                    uint16_t* lds, uint16_t* out, int64_t ld,
                                                    int64_t rows, int64_t cols, int64_t row0,
                                                    int64_t col0, float scale) {
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  uint32_t* st = reinterpret_cast<uint32_t*>(lds) + wave * (WTM * WTN / 2);
  const int lr = lane & 31, lh = lane >> 5;
  const bool odd = (lane & 1) != 0;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const uint32_t p01 = pack_bf16x2(acc[fm][fn][4 * g + 0] * scale, acc[fm][fn][4 * g + 1] * scale);
        const uint32_t p23 = pack_bf16x2(acc[fm][fn][4 * g + 2] * scale, acc[fm][fn][4 * g + 3] * scale);
        // even lane sends rows R+2, R+3; odd lane sends rows R, R+1
        const uint32_t snd = odd ? p01 : p23;
        const uint32_t rcv = static_cast<uint32_t>(
            __builtin_amdgcn_mov_dpp(static_cast<int>(snd), 0xB1, 0xF, 0xF, false));  // quad_perm 1,0,3,2
        const int R = fm * 32 + g * 8 + lh * 4;
        const int C = fn * 32 + lr;
        uint32_t w0, w1;
        int r0;
        if (!odd) {  // rows R, R+1; columns C (mine), C+1 (partner)
          w0 = __builtin_amdgcn_perm(rcv, p01, 0x05040100u);
          w1 = __builtin_amdgcn_perm(rcv, p01, 0x07060302u);
          r0 = R;
        } else {     // rows R+2, R+3; columns C-1 (partner), C (mine)
          w0 = __builtin_amdgcn_perm(p23, rcv, 0x05040100u);
          w1 = __builtin_amdgcn_perm(p23, rcv, 0x07060302u);
          r0 = R + 2;
        }
        const int dw = (C & ~1) >> 1;
        st[stage_dword<WTM, WTN>(r0, dw)] = w0;
        st[stage_dword<WTM, WTN>(r0 + 1, dw)] = w1;
      }
  // Read back 16-byte chunks: WTN / 8 chunks per row.
  constexpr int kCpr = WTN / 8;
  constexpr int kChunks = WTM * kCpr;
  const int64_t gr0 = row0 + wm * WTM, gc0 = col0 + wn * WTN;
  const bool interior = gr0 + WTM <= rows && gc0 + WTN <= cols;
#pragma unroll 4
  for (int c = lane; c < kChunks; c += kWave) {
    const int row = c / kCpr, cc = c % kCpr;
    const u32x4 v = *reinterpret_cast<const u32x4*>(st + stage_dword<WTM, WTN>(row, cc * 4));
    const int64_t gr = gr0 + row, gc = gc0 + cc * 8;
    uint16_t* dst = out + gr * ld + gc;
    if (interior) {
      *reinterpret_cast<u32x4*>(dst) = v;
    } else if (gr < rows) {
      if (gc + 8 <= cols) {
        *reinterpret_cast<u32x4*>(dst) = v;
      } else {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
        for (int e = 0; e < 8 && gc + e < cols; ++e)
          dst[e] = static_cast<uint16_t>(w[e >> 1] >> (16 * (e & 1)));
      }
    }
  }
}

// Main loop: C(BM x BN) += A(BM x K) B(K x BN), A and B staged through two
// swizzled LDS stages by the given loaders, with one register stage in front:
//
//   step kt:  MFMAs on stage kt % 2, 16 deep at a time;
//             after the first 16: registers (tile kt+1) -> the other LDS stage
//             (free since the barrier that ended step kt-1);
//             after the second 16: global loads of tile kt+2 -> registers;
//             barrier.
//
// LDS writes and the next global loads are spread between the MFMAs instead of
// arriving as one burst before the barrier.
template <int BM, int BN, int WGM, int WGN, class LA, class LB>
__device__ __forceinline__ void gemm_mainloop(LA& la, LB& lb, int64_t k_begin, int64_t k_end,
                                              uint16_t* lds, f32x16 (&acc)[BM / WGM / 32][BN / WGN / 32]) {
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
  if (kt_count > 1) {
    la.fetch(k_begin + kBK, tid);
    lb.fetch(k_begin + kBK, tid);
  }
  __syncthreads();
  for (int64_t kt = 0; kt < kt_count; ++kt) {
    const int cur = static_cast<int>(kt & 1) * kStage;
    const int nxt = kStage - cur;
    const uint16_t* As = lds + cur;
    const uint16_t* Bs = lds + cur + kAElems;
    mma_k16<FM, FN>(As, Bs, wm * FM * 32, wn * FN * 32, lane, 0, acc);
    if (kt + 1 < kt_count) {
      la.commit(lds + nxt, tid);
      lb.commit(lds + nxt + kAElems, tid);
    }
    mma_k16<FM, FN>(As, Bs, wm * FM * 32, wn * FN * 32, lane, 1, acc);
    if (kt + 2 < kt_count) {
      la.fetch(k_begin + (kt + 2) * kBK, tid);
      lb.fetch(k_begin + (kt + 2) * kBK, tid);
    }
    mma_k16<FM, FN>(As, Bs, wm * FM * 32, wn * FN * 32, lane, 2, acc);
    mma_k16<FM, FN>(As, Bs, wm * FM * 32, wn * FN * 32, lane, 3, acc);
    __syncthreads();
  }
}

// Main loop with two register stages in flight, for contractions with little
// MFMA work per K step (G^ = z^T dL/do at small r): tile j lives in register set
// j % 2 until it is committed to LDS stage j % 2, so the global loads of tiles
// kt+2 and kt+3 are outstanding while tile kt is multiplied.
template <int BM, int BN, int WGM, int WGN, class LA, class LB>
__device__ __forceinline__ void gemm_mainloop_deep(LA (&la)[2], LB (&lb)[2], int64_t k_begin, int64_t k_end,
                                                   uint16_t* lds, f32x16 (&acc)[BM / WGM / 32][BN / WGN / 32]) {
  constexpr int FM = BM / WGM / 32, FN = BN / WGN / 32;
  constexpr int kAElems = BM * kBK, kBElems = BN * kBK;
  constexpr int kStage = kAElems + kBElems;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[fm][fn][v] = 0.0f;
  const int64_t kt_count = ceil_div(k_end - k_begin, kBK);
  if (kt_count <= 0) return;
  la[0].fetch(k_begin, tid);
  lb[0].fetch(k_begin, tid);
  if (kt_count > 1) {
    la[1].fetch(k_begin + kBK, tid);
    lb[1].fetch(k_begin + kBK, tid);
  }
  la[0].commit(lds, tid);
  lb[0].commit(lds + kAElems, tid);
  if (kt_count > 2) {
    la[0].fetch(k_begin + 2 * kBK, tid);
    lb[0].fetch(k_begin + 2 * kBK, tid);
  }
  __syncthreads();
  auto step = [&](int64_t kt, LA& la_next, LB& lb_next) {
    const int cur = static_cast<int>(kt & 1) * kStage;
    const int nxt = kStage - cur;
    const uint16_t* As = lds + cur;
    const uint16_t* Bs = lds + cur + kAElems;
    mma_k16<FM, FN>(As, Bs, wm * FM * 32, wn * FN * 32, lane, 0, acc);
    if (kt + 1 < kt_count) {
      la_next.commit(lds + nxt, tid);
      lb_next.commit(lds + nxt + kAElems, tid);
    }
    mma_k16<FM, FN>(As, Bs, wm * FM * 32, wn * FN * 32, lane, 1, acc);
    if (kt + 3 < kt_count) {
      la_next.fetch(k_begin + (kt + 3) * kBK, tid);
      lb_next.fetch(k_begin + (kt + 3) * kBK, tid);
    }
    mma_k16<FM, FN>(As, Bs, wm * FM * 32, wn * FN * 32, lane, 2, acc);
    mma_k16<FM, FN>(As, Bs, wm * FM * 32, wn * FN * 32, lane, 3, acc);
    __syncthreads();
  };
  for (int64_t kt = 0; kt < kt_count; kt += 2) {
    step(kt, la[1], lb[1]);             // tile kt+1 sits in set 1
    if (kt + 1 < kt_count) step(kt + 1, la[0], lb[0]);  // tile kt+2 sits in set 0
  }
}

}  // namespace compact
