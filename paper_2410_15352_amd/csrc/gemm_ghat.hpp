// G^ = z^T dL/do (the compressed weight gradient) as a split-K bf16 GEMM for
// gfx950: M = r, N = m, K = tokens.  Both operands are token-major in memory
// (z [T][r], dL/do [T][m]), i.e. M- and N-contiguous; they are copied to LDS as
// K rows and read back as MFMA fragments with the transposing LDS read
// ds_read_b64_tr_b16.
//
// Workgroup: 4 waves over one range of tokens (a split), three tile shapes
// (rows of G^ x columns):
//   0: 128 x 256: waves 2 x 2, each 64 x 128 (2 x 4 MFMA 32x32x16
//      fragments), 6 fragment reads per 8 MFMAs;
//   1: 384 x 128 ("tall", for 256 < r that 384-row tiles cover without more
//      padding than 128-row ones, e.g. the down projection at r = 342): waves
//      stacked along the rows, each 96 x 128 (3 x 4 fragments), 7 fragment
//      reads per 12 MFMAs; every column of dL/do is copied and read by one
//      tile instead of by each of three;
//   2: 256 x 256 ("square", for r a multiple of 256 or padded no further than
//      by 128-row tiles, e.g. r = 512 of LLaMA-1B): waves 2 x 2, each 128 x 128
//      (4 x 4 fragments, 256 accumulation registers), 8 fragment reads per 16
//      MFMAs.
// The transposing fragment reads bound the kernel when r is large; shapes 1
// and 2 read fewer bytes per MFMA.
// The fp32 partial tile goes to part[split] and a separate kernel sums the
// splits in a fixed order (deterministic G^).  One launch covers up to 8
// projections of the same tokens (a layer table): the projections of an input
// group then share one grid of about one workgroup per CU, with fewer and
// longer splits than a launch per projection would have.
//
// Pipeline as in gemm_w4.hpp: 32-token K tiles, four LDS stages, copies by
// buffer_load_dwordx4 ... lds issued 3 K tiles ahead (six stages, 5 ahead, time
// the same) and spread over the MFMAs, one barrier per K tile:
//   step 0: read fragments (t, 1); the first half of this wave's copies for
//           K tile t + 3; the MFMAs on fragments (t, 0)
//   step 1: wait for this wave's copies of K tile t + 1 (the copies of K tile
//           t + 2 and the first half of t + 3 may still be in flight);
//           barrier; read fragments (t + 1, 0); the second half of the
//           copies; the MFMAs on fragments (t, 1)
//
// LDS (bytes from the dynamic base): stage s of z^T at s * TM * 64 ([32][TM]
// bf16), stage s of dL/do at 4 * TM * 64 + s * TN * 64 ([32][TN] bf16).
// 16-byte chunk c of K row k sits at c ^ (4 (k mod 4)) (the XOR stays inside
// the aligned group of 16 chunks, so rows of 48 chunks work too).  The
// transposing 64-bit read is served 32 lanes at a time; those lanes touch 4 K
// rows x 64 bytes (4 aligned chunks per row), which this swizzle puts on the
// 64 distinct banks (every row length here is a multiple of 256 bytes).
//
// Edges: tokens past T read as zero (buffer range check); splits are whole K
// tiles, so a split never reads another split's tokens.  Rows of G^ past r and
// columns past m read whatever lies there (finite bf16 values of the same
// buffers, or zero past their end) and only reach partial-sum entries the
// reduction never reads.
#pragma once
#include "gemm_bf16.hpp"
#include "gemm_w4.hpp"

namespace compact {

constexpr int kGhK = 32;                 // K tile (tokens)
constexpr int kGhStages = 4;
constexpr int kGhAhead = kGhStages - 1;  // K tiles copied ahead

// Tile geometry per shape (above).
template <int SHAPE>
struct GhShape {
  static constexpr int kTm = SHAPE == 1 ? 384 : SHAPE == 2 ? 256 : 128;  // rows of G^ (r)
  static constexpr int kTn = SHAPE == 1 ? 128 : 256;                     // columns (m)
  static constexpr int kFm = SHAPE == 1 ? 3 : SHAPE == 2 ? 4 : 2;        // MFMA fragments per wave: rows
  static constexpr int kFn = 4;                                          //   and columns
  static constexpr int kWaveRows = kFm * 32;
  static constexpr int kWaveRowGroups = kTm / kWaveRows;                 // waves along the rows
  static constexpr int kEvery = SHAPE == 2 ? 4 : 3;                      // a copy at every kEvery-th MFMA
  static constexpr int kACopies = kTm * kGhK * 2 / 1024 / 4;  // 1 KB copies per wave per K tile: z^T
  static constexpr int kBCopies = kTn * kGhK * 2 / 1024 / 4;  //   dL/do
  static constexpr int kCopies = kACopies + kBCopies;         // 6, 8, 8
  static constexpr int kAStage = kGhK * kTm * 2;              // 8, 24, 16 KB
  static constexpr int kBStage = kGhK * kTn * 2;              // 16, 8, 16 KB
  static constexpr int kBBase = kGhStages * kAStage;
  static constexpr size_t kLds = size_t(kGhStages) * (kAStage + kBStage);  // 96, 128, 128 KB
  static_assert(kWaveRowGroups * (kTn / 128) == 4, "four waves per tile");
};
constexpr int kGhTm = GhShape<0>::kTm, kGhTn = GhShape<0>::kTn;
constexpr int kGhTallTm = GhShape<1>::kTm, kGhTallTn = GhShape<1>::kTn;
constexpr int kGhSqTm = GhShape<2>::kTm, kGhSqTn = GhShape<2>::kTn;

// One projection of a launch: G^_j = z_j^T dL/do_j.  The projections of one
// launch share the token count and the split plan; in an input group (q, k, v
// or gate, up) z_j and dL/do_j are column slices of the group's z and dL/do.
struct GhatW4Layer {
  const uint16_t* z;   // [T][ldz]
  const uint16_t* dy;  // [T][lddy]
  float* part;         // [splits][tiles_r * 128][tiles_m * 256]
  int ldz, lddy;
  int r, m;
  int tiles_r, tiles_m;
};

constexpr int kGhMaxLayers = 8;

struct GhatW4Params {
  GhatW4Layer layer[kGhMaxLayers];
  int tile_begin[kGhMaxLayers + 1];  // first tile of each layer; tile_begin[count] = tiles per split
  int count;
  int T, splits;
  int split_len;  // tokens per split, a multiple of kGhK
  int shape;      // tile shape (GhShape): 0 128 x 256, 1 384 x 128, 2 256 x 256
};

// Per-lane copy offsets.  A stage of an operand with ROWS columns per K row
// holds ROWS / 8 16-byte chunks per K row; copy block q (1 KB) fills chunks
// 64 q .. 64 q + 63 of the stage in order, so lane L lands at linear chunk
// 64 q + L: K row (64 q + L) / (ROWS / 8), physical chunk the remainder.  Each
// lane fetches the logical chunk phys ^ (4 (k mod 4)).  Offsets are bytes from
// the operand's first token of the split and first column of the tile.
__device__ __forceinline__ int gh_off(int ld, int krow, int chunk) {
  return krow * ld * 2 + ((chunk ^ (4 * (krow & 3))) * 16);
}

template <int ROWS>
__device__ __forceinline__ int gh_block_off(int ld, int q, int lane) {
  constexpr int cpr = ROWS / 8;
  const int idx = 64 * q + lane;
  return gh_off(ld, idx / cpr, idx % cpr);
}

// Passes a fragment set through an empty statement, so that whatever uses the
// fragments stays after the statement before it.
template <int FM>
__device__ __forceinline__ void gh_tie(u32x4 (&fa)[FM], u32x4 (&fb)[4]) {
#pragma unroll
  for (int i = 0; i < FM; ++i) asm volatile("" : "+v"(fa[i]));
  asm volatile("" : "+v"(fb[0]), "+v"(fb[1]), "+v"(fb[2]), "+v"(fb[3]));
}

// s_waitcnt vmcnt(N), lgkmcnt(0), then s_barrier; fragments pass through so
// that the MFMAs after it stay after it
template <int N, int FM>
__device__ __forceinline__ void gh_wait_barrier(u32x4 (&fa)[2][FM], u32x4 (&fb)[2][4]) {
  static_assert(N >= 0 && N < 64, "vmcnt immediate");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" : : "n"(N) : "memory");
  gh_tie<FM>(fa[1], fb[1]);
}

template <int FM>
__device__ __forceinline__ void gh_pin_acc(f32x16 (&acc)[FM][4]) {
#pragma unroll
  for (int i = 0; i < FM; ++i) asm volatile("" : "+a"(acc[i][0]), "+a"(acc[i][1]), "+a"(acc[i][2]), "+a"(acc[i][3]));
}

// Waits for this wave's LDS reads (the fragments of the next MFMAs) and ties
// the fragments to that point, so the MFMAs that use them stay after it.
template <int FM>
__device__ __forceinline__ void gh_wait_frags(u32x4 (&fa)[2][FM], u32x4 (&fb)[2][4]) {
  asm volatile("s_waitcnt lgkmcnt(0)" : : : "memory");
  gh_tie<FM>(fa[0], fb[0]);
}

// ds_read_b64_tr_b16 as inline assembly.  The compiler cannot tell these LDS
// reads from reads of the stages the buffer-to-LDS copies are still filling,
// and with the builtin it waits for every outstanding copy (vmcnt(0)) before
// each one.  Here the pipeline's own waits apply instead: fragments read in
// step 0 are used after the step-1 barrier (which waits lgkmcnt(0)), fragments
// read in step 1 after gh_wait_frags.
__device__ __forceinline__ u32x2 gh_tr_read(uint32_t addr) {
  u32x2 v;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}

// One MFMA fragment from a [K][ROWS] stage at LDS byte address `stage`: rows
// n0 .. n0 + 31, k = kk * 16 + 8 (lane / 32) .. + 7.  In a 16-lane group the
// transposing read hands output lane t, element j, the element t mod 4 of
// source lane 4 j + t / 4; with source lane 4 j + q pointing at K row k0 + j,
// columns n0 + 4 q .. + 3, lane t receives column n0 + t of K rows k0 .. k0 + 3.
// Two such reads (h = 0, 1) give the 8 K values of the fragment.
template <int ROWS>
__device__ __forceinline__ u32x4 gh_frag(uint32_t stage, int n0, int kk, int lane) {
  const int g = lane >> 4, s = lane & 15;
  const int j = s >> 2, q = s & 3;
  const int col = n0 + (g & 1) * 16 + q * 4;
  u32x4 out;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int k = kk * 16 + (g >> 1) * 8 + 4 * h + j;
    const int chunk = (col >> 3) ^ (4 * (k & 3));
    const uint32_t off = static_cast<uint32_t>(k * ROWS + chunk * 8 + (col & 7));
    const u32x2 v = gh_tr_read(stage + 2u * off);
    out[2 * h] = v.x;
    out[2 * h + 1] = v.y;
  }
  return out;
}

// Fragments of 16-deep step kk of the stage at LDS byte offsets (sa, sb):
// rows r0 .. r0 + 32 FM - 1 of z^T, columns c0 .. c0 + 127 of dL/do.
template <int SHAPE>
__device__ __forceinline__ void gh_read(uint32_t lbase, uint32_t sa, uint32_t sb, int r0, int c0, int lane, int kk,
                                        u32x4 (&fa)[GhShape<SHAPE>::kFm], u32x4 (&fb)[4]) {
  using S = GhShape<SHAPE>;
#pragma unroll
  for (int i = 0; i < S::kFm; ++i) fa[i] = gh_frag<S::kTm>(lbase + sa, r0 + i * 32, kk, lane);
#pragma unroll
  for (int j = 0; j < 4; ++j) fb[j] = gh_frag<S::kTn>(lbase + sb, c0 + j * 32, kk, lane);
}

// The G^ partial tile of workgroup (split, layer, column tile, row tile).
template <int SHAPE>
__device__ __forceinline__ void ghat_w4(const GhatW4Params& prm) {
  using S = GhShape<SHAPE>;
  constexpr int FM = S::kFm, NM = S::kFm * S::kFn;  // fragments (rows), MFMAs per step
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // this wave's rows and columns inside the tile: 2 x 2 waves for the
  // 256-wide tiles, 4 x 1 for the tall one
  const int wr0 = S::kTn == 256 ? (wave >> 1) * S::kWaveRows : wave * S::kWaveRows;
  const int wc0 = S::kTn == 256 ? (wave & 1) * 128 : 0;
  const uint32_t logical = xcd_remap(blockIdx.x, gridDim.x);
  // order (split, layer, column tile, row tile): the row tiles that share dL/do
  // columns, and the column tiles of one layer that share z, are adjacent,
  // hence on the same XCD at the same time
  const int tiles = prm.tile_begin[prm.count];
  const int split = static_cast<int>(logical / tiles), tile_all = static_cast<int>(logical % tiles);
  const int li = batch_layer_of(prm.tile_begin, prm.count, tile_all);
  const GhatW4Layer& p = prm.layer[li];
  const int tile = tile_all - prm.tile_begin[li];
  const int ct = tile / p.tiles_r, rt = tile % p.tiles_r;
  const int row0 = rt * S::kTm, col0 = ct * S::kTn;
  const int t_begin = split * prm.split_len;
  const int t_end = min(t_begin + prm.split_len, prm.T);
  const int kt = (t_end - t_begin + kGhK - 1) / kGhK;

  // buffer ranges: from the split's first token to the last element of the
  // matrix (z and dL/do may be column slices of wider matrices)
  const int64_t zbytes = view_bytes(prm.T, p.r, p.ldz, t_begin, row0, 2);
  const int64_t ybytes = view_bytes(prm.T, p.m, p.lddy, t_begin, col0, 2);
  const __amdgpu_buffer_rsrc_t rz = w4_rsrc(p.z + static_cast<int64_t>(t_begin) * p.ldz + row0, zbytes);
  const __amdgpu_buffer_rsrc_t ry = w4_rsrc(p.dy + static_cast<int64_t>(t_begin) * p.lddy + col0, ybytes);
  // this wave's copy blocks: z^T blocks kACopies wave + q, dL/do blocks
  // kBCopies wave + q
  int voz[S::kACopies], voy[S::kBCopies];
#pragma unroll
  for (int q = 0; q < S::kACopies; ++q) voz[q] = gh_block_off<S::kTm>(p.ldz, wave * S::kACopies + q, lane);
#pragma unroll
  for (int q = 0; q < S::kBCopies; ++q) voy[q] = gh_block_off<S::kTn>(p.lddy, wave * S::kBCopies + q, lane);
  const uint32_t lbase = __builtin_amdgcn_groupstaticsize();
  // copy c (0 .. kCopies - 1) of this wave for K tile u into stage u % 4;
  // tokens past this split's K tiles or past T land out of range (the last
  // split is the only one whose K tiles run past T)
  auto copy = [&](int u, int c) {
    const int st = u % kGhStages;
    const uint32_t krow_bytes_z = static_cast<uint32_t>(u) * kGhK * p.ldz * 2;
    const uint32_t krow_bytes_y = static_cast<uint32_t>(u) * kGhK * p.lddy * 2;
    const uint32_t oob = u < kt ? 0u : kW4Oob;
    if (c < S::kACopies) {
      const uint32_t dst = lbase + st * S::kAStage + static_cast<uint32_t>(wave * S::kACopies + c) * 1024u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rz, reinterpret_cast<w4_lds_void*>(static_cast<uintptr_t>(dst)), 16,
                                               static_cast<int>((voz[c] + krow_bytes_z) | oob), 0, 0, 0);
    } else {
      const int q = c - S::kACopies;
      const uint32_t dst = lbase + S::kBBase + st * S::kBStage + static_cast<uint32_t>(wave * S::kBCopies + q) * 1024u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ry, reinterpret_cast<w4_lds_void*>(static_cast<uintptr_t>(dst)), 16,
                                               static_cast<int>((voy[q] + krow_bytes_y) | oob), 0, 0, 0);
    }
  };
  f32x16 acc[FM][4];
  const f32x16 zero = {};
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = zero;
  u32x4 fa[2][FM], fb[2][4];  // [kk parity][fragment]
  // copies in step 0 (MFMAs 0, kEvery, 2 kEvery, ...) and step 1 of a K tile
  constexpr int kStep0 = (NM + S::kEvery - 1) / S::kEvery;
  static_assert(kStep0 * 2 == S::kCopies, "the copies split evenly over the two steps");
  if (kt > 0) {
#pragma unroll
    for (int u = 0; u < kGhAhead; ++u)
#pragma unroll
      for (int c = 0; c < S::kCopies; ++c) copy(u, c);
    w4_wait_vm<0>();
    asm volatile("s_barrier" ::: "memory");
    gh_read<SHAPE>(lbase, 0, S::kBBase, wr0, wc0, lane, 0, fa[0], fb[0]);
    gh_wait_frags<FM>(fa, fb);
    for (int t = 0; t < kt; ++t) {
      const uint32_t st0 = static_cast<uint32_t>(t % kGhStages), st1 = static_cast<uint32_t>((t + 1) % kGhStages);
      const uint32_t sa = st0 * S::kAStage, sb = S::kBBase + st0 * S::kBStage;
      const uint32_t sa1 = st1 * S::kAStage, sb1 = S::kBBase + st1 * S::kBStage;
      // step 0
      gh_read<SHAPE>(lbase, sa, sb, wr0, wc0, lane, 1, fa[1], fb[1]);
#pragma unroll
      for (int i = 0; i < NM; ++i) {
        const int fi = i >> 2, fj = i & 3;
        acc[fi][fj] = mfma32x32x16(fa[0][fi], fb[0][fj], acc[fi][fj]);
        if (i % S::kEvery == 0) copy(t + kGhAhead, i / S::kEvery);
      }
      gh_pin_acc<FM>(acc);
      // step 1: this wave's copies of K tile t + 1 have landed when at most the
      // copies of the next kGhAhead - 2 K tiles and the step-0 copies of the
      // one after are in flight
      gh_wait_barrier<S::kCopies * (kGhAhead - 2) + kStep0, FM>(fa, fb);
      gh_read<SHAPE>(lbase, sa1, sb1, wr0, wc0, lane, 0, fa[0], fb[0]);
#pragma unroll
      for (int i = 0; i < NM; ++i) {
        const int fi = i >> 2, fj = i & 3;
        acc[fi][fj] = mfma32x32x16(fa[1][fi], fb[1][fj], acc[fi][fj]);
        if (i % S::kEvery == 0) copy(t + kGhAhead, kStep0 + i / S::kEvery);
      }
      gh_wait_frags<FM>(fa, fb);
    }
    w4_wait_vm<0>();  // no copy may still be writing LDS when the workgroup ends
  }
  // fp32 partial tile: lane (l % 32) owns a column, 16 rows per fragment
  const int64_t ldp = static_cast<int64_t>(p.tiles_m) * S::kTn;
  float* out = p.part + static_cast<int64_t>(split) * (p.tiles_r * S::kTm) * ldp;
  const int64_t r0 = row0 + wr0, c0 = col0 + wc0;
  for_each_acc(acc, lane, [&](int row, int col, float v) { out[(r0 + row) * ldp + c0 + col] = v; });
}

}  // namespace compact
