// G^ = z^T dL/do (the compressed weight gradient) as a split-K bf16 GEMM for
// gfx950: M = r, N = m, K = tokens.  Both operands are token-major in memory
// (z [T][r], dL/do [T][m]), i.e. M- and N-contiguous; they are copied to LDS as
// K rows and read back as MFMA fragments with the transposing LDS read
// ds_read_b64_tr_b16.
//
// Workgroup: 4 waves, output tile 128 (rows of G^) x 256 (columns), each
// wave 64 x 128 (2 x 4 MFMA 32x32x16 fragments), over one range of tokens
// (a split); the fp32 partial tile goes to part[split] and a separate kernel
// sums the splits in a fixed order (deterministic G^).  One launch covers up
// to 8 projections of the same tokens (a layer table): the projections of an
// input group then share one grid of about one workgroup per CU, with fewer
// and longer splits than a launch per projection would have.
//
// Pipeline as in gemm_w4.hpp: 32-token K tiles, four LDS stages, copies by
// buffer_load_dwordx4 ... lds issued 3 K tiles ahead (six stages, 5 ahead, time
// the same) and spread over the MFMAs, one barrier per K tile:
//   step 0: read fragments (t, 1); copies 0 .. 2 of this wave for K tile
//           t + 3; 8 MFMAs on fragments (t, 0)
//   step 1: wait for this wave's copies of K tile t + 1 (9 later copies may
//           still be in flight); barrier; read fragments (t + 1, 0); copies
//           3 .. 5; 8 MFMAs on fragments (t, 1)
//
// LDS (bytes from the dynamic base): stage s of z^T at 8192 s ([32][128]
// bf16, 256-byte K rows), stage s of dL/do at 32768 + 16384 s ([32][256] bf16,
// 512-byte K rows).  16-byte chunk c of K row k sits at c ^ (4 (k mod 4)).
// The transposing 64-bit read is served 32 lanes at a time; those lanes touch
// 4 K rows x 64 bytes (4 aligned chunks per row), which this swizzle puts on
// the 64 distinct banks.
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

constexpr int kGhTm = 128, kGhTn = 256;  // tile: rows of G^ (r), columns (m)
constexpr int kGhK = 32;                 // K tile (tokens)
constexpr int kGhStages = 4;
constexpr int kGhAhead = kGhStages - 1;  // K tiles copied ahead
constexpr int kGhCopies = 6;             // copies per wave per K tile (2 of z^T, 4 of dL/do)
constexpr int kGhAStage = kGhK * kGhTm * 2;  // 8 KB
constexpr int kGhBStage = kGhK * kGhTn * 2;  // 16 KB
constexpr int kGhBBase = kGhStages * kGhAStage;
constexpr size_t kGhLds = size_t(kGhStages) * (kGhAStage + kGhBStage);  // 96 KB

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
};

// Per-lane copy offsets.  z^T copy block q (1 KB = 4 K rows of 256 bytes):
// lane L lands at K row 4 q + L / 16, physical chunk L % 16; dL/do block q
// (2 K rows of 512 bytes): K row 2 q + L / 32, physical chunk L % 32.  Each
// lane fetches the logical chunk phys ^ (4 (k mod 4)).  Offsets are bytes from
// the operand's first token of the split and first column of the tile.
__device__ __forceinline__ int gh_off(int ld, int krow, int chunk) {
  return krow * ld * 2 + ((chunk ^ (4 * (krow & 3))) * 16);
}

// s_waitcnt vmcnt(N), lgkmcnt(0), then s_barrier; fragments pass through so
// that the MFMAs after it stay after it
template <int N>
__device__ __forceinline__ void gh_wait_barrier(u32x4 (&fa)[2][2], u32x4 (&fb)[2][4]) {
  static_assert(N >= 0 && N < 64, "vmcnt immediate");
  asm volatile("s_waitcnt vmcnt(%6) lgkmcnt(0)\n\ts_barrier"
               : "+v"(fa[1][0]), "+v"(fa[1][1]), "+v"(fb[1][0]), "+v"(fb[1][1]), "+v"(fb[1][2]), "+v"(fb[1][3])
               : "n"(N)
               : "memory");
}

__device__ __forceinline__ void gh_pin_acc(f32x16 (&acc)[2][4]) {
  asm volatile(""
               : "+a"(acc[0][0]), "+a"(acc[0][1]), "+a"(acc[0][2]), "+a"(acc[0][3]), "+a"(acc[1][0]),
                 "+a"(acc[1][1]), "+a"(acc[1][2]), "+a"(acc[1][3]));
}

// Waits for this wave's LDS reads (the fragments of the next MFMAs) and ties
// the fragments to that point, so the MFMAs that use them stay after it.
__device__ __forceinline__ void gh_wait_frags(u32x4 (&fa)[2][2], u32x4 (&fb)[2][4]) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(fa[0][0]), "+v"(fa[0][1]), "+v"(fb[0][0]), "+v"(fb[0][1]), "+v"(fb[0][2]), "+v"(fb[0][3]));
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

// Fragments of 16-deep step kk of the stage at LDS byte offsets (sa, sb).
__device__ __forceinline__ void gh_read(uint32_t lbase, uint32_t sa, uint32_t sb, int wm, int wn, int lane, int kk,
                                        u32x4 (&fa)[2], u32x4 (&fb)[4]) {
#pragma unroll
  for (int i = 0; i < 2; ++i) fa[i] = gh_frag<kGhTm>(lbase + sa, wm * 64 + i * 32, kk, lane);
#pragma unroll
  for (int j = 0; j < 4; ++j) fb[j] = gh_frag<kGhTn>(lbase + sb, wn * 128 + j * 32, kk, lane);
}

// The G^ partial tile of workgroup (split, layer, column tile, row tile).
__device__ __forceinline__ void ghat_w4(const GhatW4Params& prm) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
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
  const int row0 = rt * kGhTm, col0 = ct * kGhTn;
  const int t_begin = split * prm.split_len;
  const int t_end = min(t_begin + prm.split_len, prm.T);
  const int kt = (t_end - t_begin + kGhK - 1) / kGhK;

  // buffer ranges: from the split's first token to the last element of the
  // matrix (z and dL/do may be column slices of wider matrices)
  const int64_t zbytes = view_bytes(prm.T, p.r, p.ldz, t_begin, row0, 2);
  const int64_t ybytes = view_bytes(prm.T, p.m, p.lddy, t_begin, col0, 2);
  const __amdgpu_buffer_rsrc_t rz = w4_rsrc(p.z + static_cast<int64_t>(t_begin) * p.ldz + row0, zbytes);
  const __amdgpu_buffer_rsrc_t ry = w4_rsrc(p.dy + static_cast<int64_t>(t_begin) * p.lddy + col0, ybytes);
  // this wave's copy blocks: z^T blocks 2 wave + {0, 1}, dL/do blocks 4 wave + {0 .. 3}
  int voz[2], voy[4];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int b = wave * 2 + q;
    voz[q] = gh_off(p.ldz, 4 * b + (lane >> 4), lane & 15);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int b = wave * 4 + q;
    voy[q] = gh_off(p.lddy, 2 * b + (lane >> 5), lane & 31);
  }
  const uint32_t lbase = __builtin_amdgcn_groupstaticsize();
  // copy c (0 .. 5) of this wave for K tile u into stage u % 4; tokens past
  // this split's K tiles or past T land out of range (the last split is the only
  // one whose K tiles run past T)
  auto copy = [&](int u, int c) {
    const int st = u % kGhStages;
    const uint32_t krow_bytes_z = static_cast<uint32_t>(u) * kGhK * p.ldz * 2;
    const uint32_t krow_bytes_y = static_cast<uint32_t>(u) * kGhK * p.lddy * 2;
    const uint32_t oob = u < kt ? 0u : kW4Oob;
    if (c < 2) {
      const uint32_t dst = lbase + st * kGhAStage + static_cast<uint32_t>(wave * 2 + c) * 1024u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rz, reinterpret_cast<w4_lds_void*>(static_cast<uintptr_t>(dst)), 16,
                                               static_cast<int>((voz[c] + krow_bytes_z) | oob), 0, 0, 0);
    } else {
      const int q = c - 2;
      const uint32_t dst = lbase + kGhBBase + st * kGhBStage + static_cast<uint32_t>(wave * 4 + q) * 1024u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ry, reinterpret_cast<w4_lds_void*>(static_cast<uintptr_t>(dst)), 16,
                                               static_cast<int>((voy[q] + krow_bytes_y) | oob), 0, 0, 0);
    }
  };
  f32x16 acc[2][4];
  const f32x16 zero = {};
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = zero;
  u32x4 fa[2][2], fb[2][4];  // [kk parity][fragment]
  if (kt > 0) {
#pragma unroll
    for (int u = 0; u < kGhAhead; ++u)
#pragma unroll
      for (int c = 0; c < kGhCopies; ++c) copy(u, c);
    w4_wait_vm<0>();
    asm volatile("s_barrier" ::: "memory");
    gh_read(lbase, 0, kGhBBase, wm, wn, lane, 0, fa[0], fb[0]);
    gh_wait_frags(fa, fb);
    for (int t = 0; t < kt; ++t) {
      const uint32_t st0 = static_cast<uint32_t>(t % kGhStages), st1 = static_cast<uint32_t>((t + 1) % kGhStages);
      const uint32_t sa = st0 * kGhAStage, sb = kGhBBase + st0 * kGhBStage;
      const uint32_t sa1 = st1 * kGhAStage, sb1 = kGhBBase + st1 * kGhBStage;
      // step 0
      gh_read(lbase, sa, sb, wm, wn, lane, 1, fa[1], fb[1]);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int fi = i >> 2, fj = i & 3;
        acc[fi][fj] = mfma32x32x16(fa[0][fi], fb[0][fj], acc[fi][fj]);
        if (i % 3 == 0) copy(t + kGhAhead, i / 3);
      }
      gh_pin_acc(acc);
      // step 1: this wave's copies of K tile t + 1 have landed when at most the
      // copies of the next kGhAhead - 2 K tiles and 3 of the one after are in flight
      gh_wait_barrier<kGhCopies * (kGhAhead - 2) + 3>(fa, fb);
      gh_read(lbase, sa1, sb1, wm, wn, lane, 0, fa[0], fb[0]);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int fi = i >> 2, fj = i & 3;
        acc[fi][fj] = mfma32x32x16(fa[1][fi], fb[1][fj], acc[fi][fj]);
        if (i % 3 == 0) copy(t + kGhAhead, 3 + i / 3);
      }
      gh_wait_frags(fa, fb);
    }
    w4_wait_vm<0>();  // no copy may still be writing LDS when the workgroup ends
  }
  // fp32 partial tile: lane (l % 32) owns a column, 16 rows per fragment
  const int64_t ldp = static_cast<int64_t>(p.tiles_m) * kGhTn;
  float* out = p.part + static_cast<int64_t>(split) * (p.tiles_r * kGhTm) * ldp;
  const int64_t r0 = row0 + wm * 64, c0 = col0 + wn * 128;
  for_each_acc(acc, lane, [&](int row, int col, float v) { out[(r0 + row) * ldp + c0 + col] = v; });
}

}  // namespace compact
