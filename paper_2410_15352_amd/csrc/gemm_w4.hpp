// Persistent four-wave bf16 GEMM for gfx950: C = A B^T, A [M][K] and B [N][K]
// both K-contiguous, C bf16.  One workgroup per CU walks a list of 256 x 256
// output tiles; each of its four waves owns a 128 x 128 accumulator tile
// (4 x 4 MFMA 32x32x16 fragments, 256 accumulator registers).
//
// Why four waves of 128 x 128.  On MI355X an LDS fragment read (ds_read_b128)
// moves about 170 B/clk per CU.  Eight 64 x 128 wave tiles read 192 KB of
// fragments per 64-deep K step, which keeps LDS busy as long as the MFMA pipes
// take for the step; four 128 x 128 tiles read 128 KB.  One wave per SIMD
// cannot hide LDS latency by switching waves, so the loop software-pipelines
// it: the fragments of the next 16-deep step are read while the current
// step's 16 MFMAs issue.
//
// Global -> LDS copies use buffer_load_dwordx4 ... lds: one wave instruction
// moves 64 x 16 bytes straight into LDS (lane L's chunk lands at M0 + 16 L),
// with no staging registers and no ds_write.  K tiles are 32 deep and LDS
// holds four of them; the copy stream runs 3 K tiles ahead of the MFMAs over
// the workgroup's whole list of (tile, K tile) steps, across tile boundaries,
// so a new tile starts with its operands already in LDS.
//
// Why persistent.  With one workgroup per output tile, all 256 workgroups
// finish their tiles together and write 32 MB at once while no MFMA work is
// left to overlap it.  Here a finished tile is converted to bf16 pairs in
// registers and written out 16 stores a K tile during the first 8 K tiles of
// the next tile (8 a K tile over 16 K tiles with A in 64-deep slots).
//
// Step h of the flat sequence (K tile t of tile q, LDS stage h % 4):
//   step 0: 16 MFMAs on fragments (h, 0) (t = 0: accumulators start from
//           zero); between them, read fragments (h, 1) and issue half of the
//           copies of step h + 3 into stage (h + 3) % 4 (last read during step
//           h - 1, before its barrier)
//   step 1: wait until this wave's copies of step h + 1 have landed; barrier
//           (every wave's copies landed, every read of stage h % 4 done);
//           16 MFMAs on fragments (h, 1); between them, read fragments
//           (h + 1, 0) and issue the other half of the copies of step h + 3
//   t < 8: 16 stores of the previous tile, spread over both steps
// Copies and stores share the in-order vmcnt counter; the wait of step 1
// allows exactly the operations issued after the copies of step h + 1
// (see w4_vm_allow).
// Copies past the end of the list still issue, against an empty buffer range,
// so that the count is the same on every step; they land in stages no later
// step reads.
//
// LDS layout (bytes from the dynamic LDS base): A stage s at 16384 s, B stage
// s at 65536 + 16384 s, each [256 rows][32] bf16.  Row R is 64 bytes = four
// 16-byte chunks; logical chunk c of row R sits at c ^ ((R >> 2) & 3).  A
// ds_read_b128 is served 16 lanes at a time over 64 four-byte banks (256
// bytes): the 16 consecutive rows those lanes read then fill 16 distinct
// 16-byte bank groups (4 rows per 256 bytes, 4 chunk positions).
//
// With A in 64-deep slots (w4p_ktile below) the K tiles of an output tile are
// taken in pairs: 3 slots of 32 KB + the 4 B stages = 160 KB, and each A copy
// instruction fetches 8 rows x 128 bytes.
//
// Edges: operand rows past the matrix and chunks at k >= K read as zero (buffer
// range check), so the K sum is exact; stores past the last row are dropped by
// the same check, column pairs past the last column are steered out of range
// (an odd width writes its last column alone, w4_store_tail).  With K % 8 != 0
// the chunk that holds element K - 1 is read whole and its elements past K are
// cleared in registers (w4_mask_k); B must then be K-tiled (staged by this
// library, zero past K).  Requirements (checked by the host): K >= 320,
// 256 * ld * 2 + 2 K < 2^31 for every matrix, lda and ldb multiples of 8
// (16-byte chunks); for a K-tiled B (below) the whole operand below 2^31
// bytes.
#pragma once
#include "common.hpp"

namespace compact {

constexpr int kW4Tile = 256;     // workgroup tile, M and N
constexpr int kW4Threads = 256;  // four waves
constexpr int kW4K = 32;         // K tile
constexpr int kW4Stages = 4;
constexpr int kW4StageBytes = kW4Tile * kW4K * 2;          // one operand, one stage
constexpr int kW4BBase = kW4Stages * kW4StageBytes;        // B stages follow A stages
constexpr size_t kW4Lds = 2u * kW4Stages * kW4StageBytes;  // 128 KB
constexpr int kW4MinKTiles = 10;                           // the store schedule spans K tiles 0 .. 9

// A in 64-deep slots (an even number of K tiles, see gemm_w4_persistent):
// three slots of [256 rows][64] bf16, then the four B stages.
constexpr int kW4PairBytes = kW4Tile * 2 * kW4K * 2;                      // 32 KB
constexpr int kW4PairSlots = 3;
constexpr int kW4PBBase = kW4PairSlots * kW4PairBytes;                    // 96 KB
constexpr size_t kW4PLds = size_t(kW4PBBase) + kW4Stages * kW4StageBytes;  // 160 KB
constexpr int kW4PDrip = 16;                                              // K tiles the stores drip over
constexpr int kW4PMinKTiles = kW4PDrip + 2;                               // 18: K >= 545

// Output columns come in up to two segments (the forward pass writes y and z
// in one launch): column tile ct < seg[0].tiles writes columns 256 ct .. of
// seg[0].C, the others columns 256 (ct - seg[0].tiles) .. of seg[1].C.  B row
// 256 ct + c feeds column c of column tile ct in either case, so B stacks the
// two segments' rows with segment 1 starting at row 256 seg[0].tiles.
// Sizes are 32-bit (the host checks that they fit).
struct W4Seg {
  uint16_t* C;  // [M][ldc]
  int ldc, cols;
  int tiles;    // ceil(cols / 256)
};

// B layouts.  Row-major: row R, element k at B[R * ldb + k].  K-tiled
// (b_tiled != 0): the 32-element K tiles of all rows_b rows follow each other,
// element (R, k) at B[((k / 32) * rows_b + R) * 32 + k % 32], so that the 16
// rows one copy instruction fetches are 1 KB of contiguous memory (whole cache
// lines) instead of 16 separate 64-byte row pieces; rows_b is then a multiple
// of 256 and ceil(K / 32) * rows_b * 64 < 2^31.  Operands that this library
// stages itself use it.
struct W4Gemm {
  const uint16_t* A;  // [M][lda]
  int lda, M, K;
  const uint16_t* B;  // [rows_b][ldb], or K-tiled
  int ldb, rows_b;
  int b_tiled;
  W4Seg seg[2];       // seg[1].tiles == 0 when unused
  int tiles_n;        // seg[0].tiles + seg[1].tiles
  int tiles;          // ceil(M / 256) * tiles_n
  int band_rows;      // rows of tiles per band of the walk order (>= 1)
};

typedef __attribute__((address_space(3))) void w4_lds_void;
typedef __attribute__((address_space(3))) u32x4 w4_lds_u32x4;

constexpr uint32_t kW4Oob = 0x80000000u;  // a buffer offset past every range

__device__ __forceinline__ __amdgpu_buffer_rsrc_t w4_rsrc(const void* base, int64_t bytes) {
  const int nrec = bytes <= 0 ? 0 : (bytes > 0x7FFFFFFF ? 0x7FFFFFFF : static_cast<int>(bytes));
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0), nrec, 0x00020000);
}

// Bytes of a row-major view [rows x cols] (ld elements per row) from element
// (r0, c0) through its last element, rounded up to 16: a buffer range that ends
// inside the view's own allocation also when the view is a column slice of a
// wider matrix.  (rows - r0) * ld * esz would run past the allocation's end by
// the slice's column offset on the last row.  The rounding stays inside the
// row because the view starts 16-byte aligned and ld * esz is a multiple of 16;
// rows from `rows` on are out of range.
__host__ __device__ inline int64_t view_bytes(int64_t rows, int64_t cols, int64_t ld, int64_t r0, int64_t c0,
                                              int esz) {
  const int64_t elems = (rows - 1 - r0) * ld + cols - c0;
  return elems <= 0 ? 0 : (elems * esz + 15) & ~int64_t(15);
}

// s_waitcnt lgkmcnt(0) + s_barrier with the fragments of the following MFMAs
// passed through it: MFMAs have no memory side effects, so without this data
// dependence the compiler may issue them ahead of the barrier.  Global
// operations stay in flight (a workgroup fence would wait for them).
struct W4Frags {
  u32x4 a[4], b[4];
};

__device__ __forceinline__ void w4_lds_barrier(W4Frags& f) {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier"
               : "+v"(f.a[0]), "+v"(f.a[1]), "+v"(f.a[2]), "+v"(f.a[3]), "+v"(f.b[0]), "+v"(f.b[1]), "+v"(f.b[2]),
                 "+v"(f.b[3])
               :
               : "memory");
}

// Keeps the fragment reads of the next step in this basic block: without a
// use here the compiler sinks them past the branch that follows, next to the
// MFMAs that consume them.
__device__ __forceinline__ void w4_pin(W4Frags& f) {
  asm volatile(""
               : "+v"(f.a[0]), "+v"(f.a[1]), "+v"(f.a[2]), "+v"(f.a[3]), "+v"(f.b[0]), "+v"(f.b[1]), "+v"(f.b[2]),
                 "+v"(f.b[3]));
}

// Orders the MFMAs issued so far before whatever follows (a barrier): without
// a use of their results the compiler may move them past it.
__device__ __forceinline__ void w4_pin_acc(f32x16 (&acc)[4][4]) {
  asm volatile(""
               : "+a"(acc[0][0]), "+a"(acc[0][1]), "+a"(acc[0][2]), "+a"(acc[0][3]), "+a"(acc[1][0]), "+a"(acc[1][1]),
                 "+a"(acc[1][2]), "+a"(acc[1][3]), "+a"(acc[2][0]), "+a"(acc[2][1]), "+a"(acc[2][2]), "+a"(acc[2][3]),
                 "+a"(acc[3][0]), "+a"(acc[3][1]), "+a"(acc[3][2]), "+a"(acc[3][3]));
}

// s_waitcnt vmcnt(N), other counters untouched (gfx9 encoding).
template <int N>
__device__ __forceinline__ void w4_wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// VMEM operations issued after the last copy of step h + 1 by the time step
// (h, 1) waits, for K tile T of a tile (T past the drip span stands for every
// later T).  Copies of step h + 3 go out at MFMAs 0, 4, 8, 12 of step (h, 0)
// and 2, 6, 10, 14 of step (h, 1).  The 128 stores of the previous tile drip
// out over its first S K tiles: S = 8, at the odd MFMAs of both steps (16 per
// K tile); S = 16, at MFMAs 3, 7, 11, 15 of both steps (8 per K tile).  After
// copy 7 of step h + 1 (issued in step (h - 2, 1)) come the store at MFMA 15
// of that step, all of K tile h - 1 and step (h, 0).
template <int S>
constexpr bool w4_drip(int T) {
  return T >= 0 && T < S;
}
template <int T, int S>
constexpr int w4_vm_allow() {
  return (w4_drip<S>(T - 2) ? 1 : 0) + 8 + (w4_drip<S>(T - 1) ? 128 / S : 0) + 4 + (w4_drip<S>(T) ? 64 / S : 0);
}
static_assert(w4_vm_allow<0, 8>() == 20 && w4_vm_allow<2, 8>() == 37 && w4_vm_allow<2, 16>() == 25 &&
                  w4_vm_allow<17, 16>() == 13 && w4_vm_allow<18, 16>() == 12,
              "vmcnt allowances");

// The lane id, computed where it is used (volatile: not merged with another
// computation of it, so no register holds it across the tile loop).
__device__ __forceinline__ int w4_lane_id() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// ------------------------------ per-lane state ------------------------------
struct W4Lane {
  int lane, wave, wm, wn;
  uint32_t a0, a1, b0, b1;  // fragment byte addresses, stage 0, steps 0 and 1
  uint32_t lds;             // dynamic LDS base
  int va, vb;               // A and B copy offsets (k = 0) of block 4 wave (q = 0)
  int qa, qb;               // what the offsets add per block q (16 rows; wave-uniform)
  int kchunk;               // 8 * logical chunk this lane copies
  int ksb;                  // bytes the B offsets advance per element of k0
  // A in 64-deep slots only: the copy offset of the odd copy blocks (the even
  // ones use va) and the element offset of this lane's chunk in an even block
  int va2, kca;
};

// Fragment chunk of lane `lane` for step kk (0, 1), fragment 0, stage 0, in a
// wave tile starting at row `wrow`; fragment i adds 2048 i, stage s 16384 s.
__device__ __forceinline__ uint32_t w4_frag_off(int wrow, int lane, int kk) {
  const int lr = lane & 31, lh = lane >> 5;
  const int phys = (2 * kk + lh) ^ ((lr >> 2) & 3);
  return static_cast<uint32_t>(wrow * 64 + lr * 64 + phys * 16);
}

// Lane L of copy block j lands at row 16 j + L / 4, physical chunk L % 4, so
// it fetches logical chunk (L % 4) ^ ((L / 16) % 4).
__device__ __forceinline__ int w4_copy_off(int64_t ld, int lane, int j, int& kchunk) {
  const int c = (lane & 3) ^ ((lane >> 4) & 3);
  kchunk = 8 * c;
  return static_cast<int>((16 * j + (lane >> 2)) * ld * 2) + 16 * c;
}

// A in 64-deep slots.  Row R of a slot is 128 bytes, 8 chunks: chunks 0 .. 3
// hold the first K tile of the pair, 4 .. 7 the second; logical chunk c of
// row R sits at c ^ ((R >> 1) & 7).  The 16 rows that 16 lanes of a
// ds_read_b128 read fill 16 distinct 16-byte bank groups (2 rows per 256
// bytes, 8 chunk positions).  Fragment chunk of lane `lane` for step kk of
// the pair's first K tile, fragment 0, in a wave tile starting at row `wrow`
// (a multiple of 16); the second K tile flips bit 6 of the offset (chunk
// c + 4 = c ^ 4), fragment i adds 4096 i.
__device__ __forceinline__ uint32_t w4p_frag_off(int wrow, int lane, int kk) {
  const int lr = lane & 31, lh = lane >> 5;
  const int phys = (2 * kk + lh) ^ ((lr >> 1) & 7);
  return static_cast<uint32_t>((wrow + lr) * 128 + phys * 16);
}

// A copy block j (0 .. 7) of wave w fetches rows 64 w + 8 j .. + 7 of a pair,
// 128 bytes each: lane L lands at row 64 w + 8 j + L / 8, physical chunk
// L % 8, so it fetches logical chunk (L % 8) ^ (L / 16) ^ 4 (j % 2).
__device__ __forceinline__ int w4p_copy_off(int64_t ld, int lane, int w, int jodd, int& kchunk) {
  const int c = (lane & 7) ^ (lane >> 4) ^ (4 * jodd);
  kchunk = 8 * c;
  return static_cast<int>((64 * w + (lane >> 3)) * ld * 2) + 16 * c;
}

template <bool PAIRS>
__device__ __forceinline__ W4Lane w4_lane(const W4Gemm& g) {
  W4Lane L;
  const int tid = threadIdx.x;
  L.lane = tid & 63;
  L.wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  L.wm = L.wave >> 1;
  L.wn = L.wave & 1;
  L.lds = __builtin_amdgcn_groupstaticsize();
  const int bbase = PAIRS ? kW4PBBase : kW4BBase;
  if constexpr (PAIRS) {
    // lane-relative offsets (the slot and the LDS base are added where they
    // are read, after the bit-6 flip of a pair's second K tile)
    L.a0 = w4p_frag_off(L.wm * 128, L.lane, 0);
    L.a1 = w4p_frag_off(L.wm * 128, L.lane, 1);
  } else {
    L.a0 = L.lds + w4_frag_off(L.wm * 128, L.lane, 0);
    L.a1 = L.lds + w4_frag_off(L.wm * 128, L.lane, 1);
  }
  L.b0 = L.lds + bbase + w4_frag_off(L.wn * 128, L.lane, 0);
  L.b1 = L.lds + bbase + w4_frag_off(L.wn * 128, L.lane, 1);
  // block q = 0 of this wave; block q adds 16 q rows (a wave-uniform step),
  // so only one offset per operand stays in a vector register
  const int ldb_rows = g.b_tiled ? 32 : g.ldb;
  L.vb = w4_copy_off(ldb_rows, L.lane, L.wave * 4, L.kchunk);
  L.qb = 32 * ldb_rows;
  L.ksb = g.b_tiled ? 2 * g.rows_b : 2;
  if constexpr (PAIRS) {
    int unused;
    L.va = w4p_copy_off(g.lda, L.lane, L.wave, 0, L.kca);
    L.va2 = w4p_copy_off(g.lda, L.lane, L.wave, 1, unused);
    L.qa = 16 * g.lda;  // block j adds 8 j rows
  } else {
    int kca;
    L.va = w4_copy_off(g.lda, L.lane, L.wave * 4, kca);  // the same chunk as B
    L.va2 = 0;
    L.kca = kca;
    L.qa = 32 * g.lda;
  }
  return L;
}

// ------------------------------ tile cursor --------------------------------
// Walk order.  Tiles are listed band by band (band_rows rows of tiles each),
// column by column inside a band, row by row inside a column.  The workgroups
// of one XCD (consecutive logical ids, see xcd_remap) take one contiguous
// stretch of that list, dealt round-robin: in every round the workgroups of an
// XCD work on a block of about band_rows x (workgroups / band_rows) tiles,
// whose operand row and column blocks they share through that XCD's L2.
// A workgroup's q-th tile is list entry off + q * gx + w (gx: workgroups on
// its XCD, w: its place among them, off: tiles of the XCDs before it).
struct W4Walk {
  int gx, w, off;
};

__device__ __forceinline__ W4Walk w4_walk(const W4Gemm& g, int p, int G) {
  // xcd_remap gives XCD x the logical ids start .. start + gx - 1
  const int q = G / kNumXcd, rem = G % kNumXcd;
  const int x = p < (q + 1) * rem ? p / (q + 1) : rem + (p - (q + 1) * rem) / (q > 0 ? q : 1);
  const int start = x * q + (x < rem ? x : rem);
  const int full = g.tiles / G, rem_t = g.tiles % G;
  W4Walk k;
  k.gx = q + (x < rem ? 1 : 0);
  k.w = p - start;
  k.off = start * full + (rem_t < start ? rem_t : start);
  return k;
}

struct W4Cursor {
  int q, rt, ct;
};

// Row and column tile of the workgroup's q-th tile (clamped to the last tile
// past the end of its list; such positions are never live).
__device__ __forceinline__ void w4_tile_at(const W4Gemm& g, const W4Walk& k, W4Cursor& c) {
  int i = k.off + c.q * k.gx + k.w;
  i = i < g.tiles ? i : g.tiles - 1;
  const int rows_total = g.tiles / g.tiles_n;
  const int per_band = g.band_rows * g.tiles_n;
  const int b = i / per_band;
  const int r0 = b * g.band_rows;
  const int rows_b = rows_total - r0 < g.band_rows ? rows_total - r0 : g.band_rows;
  const int within = i - b * per_band;
  c.ct = within / rows_b;
  c.rt = r0 + within - c.ct * rows_b;
}

__device__ __forceinline__ void w4_next_tile(const W4Gemm& g, const W4Walk& k, W4Cursor& c) {
  c.q += 1;
  w4_tile_at(g, k, c);
}

struct W4CopyDesc {
  __amdgpu_buffer_rsrc_t ra, rb;
};

__device__ __forceinline__ W4CopyDesc w4_copy_desc(const W4Gemm& g, const W4Cursor& c, int n_my) {
  W4CopyDesc d;
  const bool live = c.q < n_my;
  const int64_t row0 = static_cast<int64_t>(c.rt) * kW4Tile;
  const int64_t brow0 = static_cast<int64_t>(c.ct) * kW4Tile;
  d.ra = w4_rsrc(g.A + row0 * g.lda, live ? (g.M - row0) * int64_t(g.lda) * 2 : 0);
  if (g.b_tiled)
    d.rb = w4_rsrc(g.B + brow0 * 32, live ? (ceil_div(g.K, kW4K) * g.rows_b - brow0) * 64 : 0);
  else
    d.rb = w4_rsrc(g.B + brow0 * g.ldb, live ? (g.rows_b - brow0) * int64_t(g.ldb) * 2 : 0);
  return d;
}

// Copy the K tile starting at k0 of the tile `d` into stage byte offsets
// (sa, sb) of A and B.  Chunks at k >= K get an offset past every range (set
// with a shift, not a select, so the compiler keeps the copies branch-free).
__device__ __forceinline__ void w4_copy(const W4Gemm& g, const W4Lane& L, const W4CopyDesc& d, int k0,
                                        uint32_t sa, uint32_t sb) {
  // bit 31 set iff k0 + kchunk >= K
  const uint32_t oob = ~static_cast<uint32_t>(k0 + L.kchunk - g.K) & kW4Oob;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t vo = static_cast<uint32_t>(L.va + q * L.qa + 2 * k0) | oob;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        d.ra, reinterpret_cast<w4_lds_void*>(static_cast<uintptr_t>(sa + (L.wave * 4 + q) * 1024u)), 16,
        static_cast<int>(vo), 0, 0, 0);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t vo = static_cast<uint32_t>(L.vb + q * L.qb + L.ksb * k0) | oob;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        d.rb, reinterpret_cast<w4_lds_void*>(static_cast<uintptr_t>(sb + (L.wave * 4 + q) * 1024u)), 16,
        static_cast<int>(vo), 0, 0, 0);
  }
}

// The copy stream: the next (tile, K tile) to copy.
struct W4CopyCursor {
  W4Cursor c;
  int k;  // K tile
  W4CopyDesc d;
};

__device__ __forceinline__ void w4_copy_advance(const W4Gemm& g, W4CopyCursor& cc, int kt, int n_my,
                                                const W4Walk& wk) {
  cc.k += 1;
  if (cc.k == kt) {
    cc.k = 0;
    w4_next_tile(g, wk, cc.c);
    cc.d = w4_copy_desc(g, cc.c, n_my);
  }
}

// ------------------------------ output side --------------------------------
// The bf16 result of a wave tile, as packed column pairs: for accumulator
// block (i, j) and row group gr, the even lane of a pair holds rows R, R + 1
// of columns C, C + 1 and the odd lane rows R + 2, R + 3 (one DPP swap).
struct W4Out {
  __amdgpu_buffer_rsrc_t rc;  // base at the wave tile's first element
  uint32_t vj[4];             // lane byte offset for column block j, or out of range
  uint32_t rstride;           // ldc * 2
  int room;                   // columns of the wave tile inside the matrix (cols - first column)
};

__device__ __forceinline__ W4Out w4_out_desc(const W4Gemm& g, const W4Lane& L, const W4Cursor& c, bool live) {
  W4Out o;
  const int seg = c.ct >= g.seg[0].tiles ? 1 : 0;
  uint16_t* C = seg ? g.seg[1].C : g.seg[0].C;
  const int64_t ldc = seg ? g.seg[1].ldc : g.seg[0].ldc;
  const int64_t cols = seg ? g.seg[1].cols : g.seg[0].cols;
  const int64_t wrow0 = static_cast<int64_t>(c.rt) * kW4Tile + L.wm * 128;
  const int64_t wcol0 = static_cast<int64_t>(seg ? c.ct - g.seg[0].tiles : c.ct) * kW4Tile + L.wn * 128;
  o.rc = w4_rsrc(C + wrow0 * ldc + wcol0, live ? ((g.M - wrow0) * ldc - wcol0) * 2 : 0);
  o.rstride = static_cast<uint32_t>(ldc * 2);
  // 32-bit lane arithmetic (every size fits; the host checks), from a lane
  // id recomputed here: lane values kept alive across the tile loop would be
  // spilled, and each reload waits for every copy in flight
  const int lane = w4_lane_id();
  const int lr = lane & 31, lh = lane >> 5, odd = lane & 1;
  const uint32_t rl = static_cast<uint32_t>(4 * lh + 2 * odd) * o.rstride;
  o.room = static_cast<int>(cols) - static_cast<int>(wcol0);
  const int room = o.room - 1 - (lr & ~1);  // cl + 1 < cols - wcol0
#pragma unroll
  for (int j = 0; j < 4; ++j)
    o.vj[j] = j * 32 < room ? rl + 2u * static_cast<uint32_t>(j * 32 + (lr & ~1)) : kW4Oob;
  return o;
}

// Accumulator block b (row group gr: rows 8 gr + 4 (lane / 32) + 0 .. 3 of
// column lane % 32) converted to bf16 pairs: raw[(b * 4 + gr) * 2] holds rows
// + 0, + 1 and raw[... + 1] rows + 2, + 3.
__device__ __forceinline__ void w4_convert_block(const f32x16& a, int b, uint32_t (&raw)[128]) {
  // The accumulators are read out one block at a time, each block after the
  // previous one is converted (the first read takes that block's last value
  // as an input).  Left to itself the compiler reads 13 of the 16 blocks out
  // of the accumulator registers before converting any: 208 VGPRs at once,
  // the peak that made the K % 8 != 0 variants spill.
  float v[16];
  const uint32_t dep = b > 0 ? raw[b * 8 - 1] : 0u;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    if (e == 0)
      asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v[e]) : "a"(a[e]), "v"(dep));
    else
      asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v[e]) : "a"(a[e]));
  }
#pragma unroll
  for (int gr = 0; gr < 4; ++gr) {
    raw[(b * 4 + gr) * 2] = pack_bf16x2(v[4 * gr + 0], v[4 * gr + 1]);
    raw[(b * 4 + gr) * 2 + 1] = pack_bf16x2(v[4 * gr + 2], v[4 * gr + 3]);
  }
}

// The two stores of (block, row group) from its raw pair p01, p23, one DPP
// swap between the lanes of a column pair: the even lane gets rows R, R + 1 of
// columns C, C + 1 (o0, o1), the odd lane rows R + 2, R + 3 of C - 1, C.
__device__ __forceinline__ void w4_shuffle(uint32_t p01, uint32_t p23, bool odd, uint32_t& o0, uint32_t& o1) {
  const uint32_t snd = odd ? p01 : p23;
  const uint32_t rcv =
      static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(snd), 0xB1, 0xF, 0xF, false));  // 1,0,3,2
  const uint32_t hi = odd ? p23 : rcv, lo = odd ? rcv : p01;
  o0 = __builtin_amdgcn_perm(hi, lo, 0x05040100u);
  o1 = __builtin_amdgcn_perm(hi, lo, 0x07060302u);
}

__device__ __forceinline__ uint32_t w4_store_off(const W4Out& od, int b, int gr, int w) {
  return od.vj[b & 3] + static_cast<uint32_t>((b >> 2) * 32 + gr * 8 + w) * od.rstride;
}

// An odd output width: the column pair that straddles the last column is
// steered out of range by w4_store_off; its first column (the low halves)
// goes out here with 2-byte stores, all 32 of a wave tile at once, right
// after the tile is converted (only wave tiles that hold the last column).
template <int J>
__device__ __forceinline__ void w4_store_tails_j(const W4Out& od, const uint32_t (&raw)[128]) {
  const int lane = w4_lane_id();
  const int lr = lane & 31, lh = lane >> 5, odd = lane & 1;
  const int cl = J * 32 + (lr & ~1);
  const uint32_t base = cl + 1 == od.room ? static_cast<uint32_t>(4 * lh + 2 * odd) * od.rstride +
                                                2u * static_cast<uint32_t>(cl)
                                          : kW4Oob;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int gr = 0; gr < 4; ++gr) {
      const int b = i * 4 + J;
      uint32_t o0, o1;
      w4_shuffle(raw[(b * 4 + gr) * 2], raw[(b * 4 + gr) * 2 + 1], odd != 0, o0, o1);
      const uint32_t r = static_cast<uint32_t>(i * 32 + gr * 8) * od.rstride;
      __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(o0), od.rc, static_cast<int>(base + r), 0, 0);
      __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(o1), od.rc,
                                            static_cast<int>(base + r + od.rstride), 0, 0);
    }
}

// The column block of the last column is wave-uniform; a branch per block
// keeps every index into raw a constant (an index computed at run time would
// put raw in scratch memory).
__device__ __forceinline__ void w4_store_tails(const W4Out& od, const uint32_t (&raw)[128]) {
  if ((od.room & 1) == 0 || od.room <= 0 || od.room >= 128) return;  // wave-uniform
  switch ((od.room - 1) >> 5) {  // column block of the last column
    case 0: w4_store_tails_j<0>(od, raw); break;
    case 1: w4_store_tails_j<1>(od, raw); break;
    case 2: w4_store_tails_j<2>(od, raw); break;
    default: w4_store_tails_j<3>(od, raw); break;
  }
}

// Every store of a converted tile at once (the last tile of the workgroup).
template <bool ODD>
__device__ __forceinline__ void w4_flush(const W4Out& od, const uint32_t (&raw)[128]) {
  const bool odd = (w4_lane_id() & 1) != 0;
#pragma unroll
  for (int b = 0; b < 16; ++b)
#pragma unroll
    for (int gr = 0; gr < 4; ++gr) {
      uint32_t o0, o1;
      w4_shuffle(raw[(b * 4 + gr) * 2], raw[(b * 4 + gr) * 2 + 1], odd, o0, o1);
      __builtin_amdgcn_raw_buffer_store_b32(o0, od.rc, static_cast<int>(w4_store_off(od, b, gr, 0)), 0, 0);
      __builtin_amdgcn_raw_buffer_store_b32(o1, od.rc, static_cast<int>(w4_store_off(od, b, gr, 1)), 0, 0);
    }
  if constexpr (ODD) w4_store_tails(od, raw);
}

// ------------------------------ MFMA steps ---------------------------------
__device__ __forceinline__ void w4_read(uint32_t a, uint32_t b, W4Frags& f) {
#pragma unroll
  for (int i = 0; i < 4; ++i) f.a[i] = *reinterpret_cast<const w4_lds_u32x4*>(static_cast<uintptr_t>(a + i * 2048));
#pragma unroll
  for (int i = 0; i < 4; ++i) f.b[i] = *reinterpret_cast<const w4_lds_u32x4*>(static_cast<uintptr_t>(b + i * 2048));
}

// One K tile, T = its index in the tile (10: any T >= 10); h = flat step.
// The source order below is the issue order: this header is compiled with
// the machine scheduler off, so MFMAs, LDS reads, copies and stores stay
// interleaved as written.  Copies and stores are spread out because the
// vector memory unit takes about 16 clocks per 64-lane 16-byte copy: issued
// in bursts they stall the in-order issue of the MFMAs behind them.
template <int T>
__device__ __forceinline__ void w4_copy_one(const W4Lane& L, const W4CopyCursor& cc, int c, uint32_t oob,
                                            int k3, uint32_t s3) {
  const int q = c & 3;
  const bool is_a = c < 4;
  const uint32_t vo = static_cast<uint32_t>(is_a ? L.va + q * L.qa + 2 * k3 : L.vb + q * L.qb + L.ksb * k3) | oob;
  const uint32_t dst = L.lds + (is_a ? 0u : static_cast<uint32_t>(kW4BBase)) + s3 + (L.wave * 4 + q) * 1024u;
  __builtin_amdgcn_raw_ptr_buffer_load_lds(is_a ? cc.d.ra : cc.d.rb,
                                           reinterpret_cast<w4_lds_void*>(static_cast<uintptr_t>(dst)), 16,
                                           static_cast<int>(vo), 0, 0, 0);
}

// Store n (0 .. 128 / S - 1) of K tile T in a drip span of S K tiles: store
// i = 128 T / S + n of the tile, block i / 8, row group (i / 2) % 4, row i % 2.
// An even n shuffles the pair of its (block, row group) and keeps the second
// value in `hold` for store n + 1.
template <int T, int S>
__device__ __forceinline__ void w4_store_one(const W4Out& od, const uint32_t (&raw)[128], bool odd, uint32_t& hold,
                                             int n) {
  const int idx = T * (128 / S) + n;
  const int b = idx >> 3, gr = (idx >> 1) & 3, w = idx & 1;
  uint32_t v;
  if (w == 0) {
    w4_shuffle(raw[(b * 4 + gr) * 2], raw[(b * 4 + gr) * 2 + 1], odd, v, hold);
  } else {
    v = hold;
  }
  __builtin_amdgcn_raw_buffer_store_b32(v, od.rc, static_cast<int>(w4_store_off(od, b, gr, w)), 0, 0);
}

// K % 8 != 0: the last 16-byte chunk of every A row holds K % 8 elements of
// the row and then whatever the caller's row padding holds (possibly NaN);
// the copies bring it into LDS whole.  In the tile's last K tile the A
// fragments that hold that chunk (k step kk, the lanes of half h) have the
// elements past K cleared before their MFMAs.  (B past K is zero: this
// library stages it.)
__device__ __forceinline__ void w4_mask_k(const W4Gemm& g, W4Frags& f, int kk, bool last) {
  const int c = ((g.K - 1) & 31) >> 3;  // chunk of element K - 1 in its K tile
  if ((c >> 1) != kk) return;           // (wave-uniform, fixed for the launch)
  // per dword of the chunk (two elements): the bits kept in the last K tile
  // (wave-uniform values, so only the lane-half test is per lane)
  const bool hit = (w4_lane_id() >> 5) == (c & 1);  // this lane's fragments hold the chunk
  const int keep = g.K & 7;
  uint32_t pm[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const uint32_t part = 2 * d + 1 < keep ? 0xFFFFFFFFu : (2 * d < keep ? 0x0000FFFFu : 0u);
    pm[d] = last ? part : 0xFFFFFFFFu;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int d = 0; d < 4; ++d) f.a[i][d] = hit ? (f.a[i][d] & pm[d]) : f.a[i][d];
}

template <int T, bool KMASK, bool ODD>
__device__ __forceinline__ void w4_ktile(const W4Gemm& g, const W4Lane& L, int h, W4CopyCursor& cc, int kt,
                                         int n_my, const W4Walk& wk, const W4Out& od,
                                         uint32_t (&raw)[128], W4Frags (&f)[2], f32x16 (&acc)[4][4],
                                         bool last = false) {
  const bool odd = w4_drip<8>(T) ? (w4_lane_id() & 1) != 0 : false;
  uint32_t hold = 0;
  const uint32_t s0 = static_cast<uint32_t>(h & 3) * kW4StageBytes;
  const uint32_t s1 = static_cast<uint32_t>((h + 1) & 3) * kW4StageBytes;
  const uint32_t s3 = static_cast<uint32_t>((h + 3) & 3) * kW4StageBytes;
  const f32x16 zero = {};
  const int k3 = cc.k * kW4K;
  const uint32_t oob = ~static_cast<uint32_t>(k3 + L.kchunk - g.K) & kW4Oob;
  if constexpr (KMASK) w4_mask_k(g, f[0], 0, last);
  // step 0: MFMAs on f[0]; reads of f[1]; copies 0 .. 3 of step h + 3
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int fa = i >> 2, fb = i & 3;
    acc[fa][fb] = mfma32x32x16(f[0].a[fa], f[0].b[fb], T == 0 ? zero : acc[fa][fb]);
    if (i < 4) {
      f[1].a[i] = *reinterpret_cast<const w4_lds_u32x4*>(static_cast<uintptr_t>(L.a1 + s0 + i * 2048));
    } else if (i < 8) {
      f[1].b[i - 4] = *reinterpret_cast<const w4_lds_u32x4*>(static_cast<uintptr_t>(L.b1 + s0 + (i - 4) * 2048));
    }
    if (i % 4 == 0) w4_copy_one<T>(L, cc, i / 4, oob, k3, s3);
    if constexpr (w4_drip<8>(T)) {
      if (i % 2 == 1) w4_store_one<T, 8>(od, raw, odd, hold, i / 2);
    }
  }
  w4_pin_acc(acc);
  // step 1: MFMAs on f[1]; reads of f[0] for step h + 1; copies 4 .. 7
  w4_wait_vm<w4_vm_allow<T, 8>()>();
  w4_lds_barrier(f[1]);
  if constexpr (KMASK) w4_mask_k(g, f[1], 1, last);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int fa = i >> 2, fb = i & 3;
    acc[fa][fb] = mfma32x32x16(f[1].a[fa], f[1].b[fb], acc[fa][fb]);
    if (i < 4) {
      f[0].a[i] = *reinterpret_cast<const w4_lds_u32x4*>(static_cast<uintptr_t>(L.a0 + s1 + i * 2048));
    } else if (i < 8) {
      f[0].b[i - 4] = *reinterpret_cast<const w4_lds_u32x4*>(static_cast<uintptr_t>(L.b0 + s1 + (i - 4) * 2048));
    }
    if (i % 4 == 2) w4_copy_one<T>(L, cc, 4 + i / 4, oob, k3, s3);
    if constexpr (w4_drip<8>(T)) {
      if (i % 2 == 1) w4_store_one<T, 8>(od, raw, odd, hold, 8 + i / 2);
    }
  }
  w4_pin(f[0]);
  w4_copy_advance(g, cc, kt, n_my, wk);
}

// ------------------------- A in 64-deep slots ------------------------------
// With an even number kt of K tiles per tile (an odd count is rounded up: the
// last K tile then lies wholly past K and reads zeros), K tiles 2P and 2P + 1
// of the flat sequence (pair P, never split across two tiles) read A from slot
// P % 3, and A is copied a pair at a time: each group of 8 lanes fetches one
// 128-byte row piece (a whole cache line) instead of two 64-byte halves in
// two K tiles.  The row-major A is the operand whose copies cost the
// vector-memory path most (B is K-tiled: 1 KB of contiguous memory per copy
// instruction already).  Pair P + 2 is copied during K tiles 2P (blocks
// 0 .. 3 of each wave) and 2P + 1 (blocks 4 .. 7), at the MFMAs where the
// 32-deep layout issues its A copies, so the copies per K tile and the vmcnt
// accounting (w4_vm_allow) stay the same: the last copies that K tile h + 1
// needs are still the B copies issued during K tile h - 2 (the second half of
// pair (h + 1) / 2 went out in the step before them, or earlier).  Slot
// (P + 2) % 3 last held pair P - 1, whose last fragments were read before the
// barrier of K tile 2P - 1.
struct W4PairCursor {
  W4Cursor c;   // tile of the pair being copied
  int kp;       // its pair index in that tile
  __amdgpu_buffer_rsrc_t ra;
  uint32_t sa;  // slot byte offset of the pair the MFMAs are on
};

__device__ __forceinline__ void w4p_advance(const W4Gemm& g, W4PairCursor& ap, int kt, int n_my, const W4Walk& wk) {
  ap.kp += 1;
  if (2 * ap.kp == kt) {
    ap.kp = 0;
    w4_next_tile(g, wk, ap.c);
    ap.ra = w4_copy_desc(g, ap.c, n_my).ra;
  }
}

// Out-of-range bits of the even (oe) and odd (oo) A blocks of the pair that
// starts at element k0.
__device__ __forceinline__ void w4p_oob(const W4Gemm& g, const W4Lane& L, int k0, uint32_t& oe, uint32_t& oo) {
  oe = ~static_cast<uint32_t>(k0 + L.kca - g.K) & kW4Oob;
  oo = ~static_cast<uint32_t>(k0 + (L.kca ^ 32) - g.K) & kW4Oob;
}

// A copy block j (0 .. 7) of the pair at element k0 into slot byte offset `slot`.
__device__ __forceinline__ void w4p_copy_a(const W4Lane& L, __amdgpu_buffer_rsrc_t ra, int k0, uint32_t oob,
                                           uint32_t slot, int j) {
  const uint32_t vo = static_cast<uint32_t>(((j & 1) ? L.va2 : L.va) + j * L.qa + 2 * k0) | oob;
  const uint32_t dst = L.lds + slot + static_cast<uint32_t>(L.wave * 8 + j) * 1024u;
  __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, reinterpret_cast<w4_lds_void*>(static_cast<uintptr_t>(dst)), 16,
                                           static_cast<int>(vo), 0, 0, 0);
}

// B copy block q (0 .. 3) of the K tile at element k3 into the B stage at byte
// offset `stage` (from the B base).
__device__ __forceinline__ void w4p_copy_b(const W4Lane& L, __amdgpu_buffer_rsrc_t rb, int k3, uint32_t oob,
                                           uint32_t stage, int q) {
  const uint32_t vo = static_cast<uint32_t>(L.vb + q * L.qb + L.ksb * k3) | oob;
  const uint32_t dst = L.lds + kW4PBBase + stage + static_cast<uint32_t>(L.wave * 4 + q) * 1024u;
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, reinterpret_cast<w4_lds_void*>(static_cast<uintptr_t>(dst)), 16,
                                           static_cast<int>(vo), 0, 0, 0);
}

// w4_ktile with A in 64-deep slots (T = 18 and 19: any even and odd T >= 18);
// the previous tile's stores drip out over K tiles 0 .. 15, 8 per K tile.
template <int T, bool KMASK, bool ODD>
__device__ __forceinline__ void w4p_ktile(const W4Gemm& g, const W4Lane& L, int h, W4CopyCursor& cc,
                                          W4PairCursor& ap, int kt, int n_my, const W4Walk& wk, const W4Out& od,
                                          uint32_t (&raw)[128], W4Frags (&f)[2], f32x16 (&acc)[4][4],
                                          bool last = false) {
  constexpr uint32_t e = T & 1;  // K tile h is the first (0) or second (1) of its pair
  const bool odd = w4_drip<kW4PDrip>(T) ? (w4_lane_id() & 1) != 0 : false;
  uint32_t hold = 0;
  const uint32_t s0 = static_cast<uint32_t>(h & 3) * kW4StageBytes;
  const uint32_t s1 = static_cast<uint32_t>((h + 1) & 3) * kW4StageBytes;
  const uint32_t s3 = static_cast<uint32_t>((h + 3) & 3) * kW4StageBytes;
  const uint32_t sa_next = ap.sa == 2u * kW4PairBytes ? 0u : ap.sa + kW4PairBytes;
  const uint32_t sa_copy = ap.sa == 0u ? 2u * kW4PairBytes : ap.sa - kW4PairBytes;  // slot of pair + 2
  const uint32_t ar1 = (L.a1 ^ (64u * e)) + L.lds + ap.sa;                         // A fragments (h, 1)
  const uint32_t ar0 = (L.a0 ^ (64u * (1u - e))) + L.lds + (e ? sa_next : ap.sa);  // A fragments (h + 1, 0)
  const f32x16 zero = {};
  const int k3 = cc.k * kW4K;  // B copies: step h + 3
  const uint32_t oobb = ~static_cast<uint32_t>(k3 + L.kchunk - g.K) & kW4Oob;
  const int k0 = ap.kp * (2 * kW4K);  // A copies: pair h / 2 + 2
  uint32_t oe, oo;
  w4p_oob(g, L, k0, oe, oo);
  if constexpr (KMASK) w4_mask_k(g, f[0], 0, last);
  // step 0: MFMAs on f[0]; reads of f[1]; A copy blocks 4 e .. 4 e + 3 of pair h / 2 + 2
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int fa = i >> 2, fb = i & 3;
    acc[fa][fb] = mfma32x32x16(f[0].a[fa], f[0].b[fb], T == 0 ? zero : acc[fa][fb]);
    if (i < 4) {
      f[1].a[i] = *reinterpret_cast<const w4_lds_u32x4*>(static_cast<uintptr_t>(ar1 + i * 4096));
    } else if (i < 8) {
      f[1].b[i - 4] = *reinterpret_cast<const w4_lds_u32x4*>(static_cast<uintptr_t>(L.b1 + s0 + (i - 4) * 2048));
    }
    if (i % 4 == 0) {
      const int j = 4 * static_cast<int>(e) + i / 4;
      w4p_copy_a(L, ap.ra, k0, (j & 1) ? oo : oe, sa_copy, j);
    }
    if constexpr (w4_drip<kW4PDrip>(T)) {
      if (i % 4 == 3) w4_store_one<T, kW4PDrip>(od, raw, odd, hold, i / 4);
    }
  }
  w4_pin_acc(acc);
  // step 1: MFMAs on f[1]; reads of f[0] for step h + 1; B copies of step h + 3
  w4_wait_vm<w4_vm_allow<T, kW4PDrip>()>();
  w4_lds_barrier(f[1]);
  if constexpr (KMASK) w4_mask_k(g, f[1], 1, last);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int fa = i >> 2, fb = i & 3;
    acc[fa][fb] = mfma32x32x16(f[1].a[fa], f[1].b[fb], acc[fa][fb]);
    if (i < 4) {
      f[0].a[i] = *reinterpret_cast<const w4_lds_u32x4*>(static_cast<uintptr_t>(ar0 + i * 4096));
    } else if (i < 8) {
      f[0].b[i - 4] = *reinterpret_cast<const w4_lds_u32x4*>(static_cast<uintptr_t>(L.b0 + s1 + (i - 4) * 2048));
    }
    if (i % 4 == 2) w4p_copy_b(L, cc.d.rb, k3, oobb, s3, i / 4);
    if constexpr (w4_drip<kW4PDrip>(T)) {
      if (i % 4 == 3) w4_store_one<T, kW4PDrip>(od, raw, odd, hold, 4 + i / 4);
    }
  }
  w4_pin(f[0]);
  w4_copy_advance(g, cc, kt, n_my, wk);
  if constexpr (e == 1) {
    w4p_advance(g, ap, kt, n_my, wk);
    ap.sa = sa_next;
  }
}

// The whole persistent GEMM for this workgroup.  Launch with kW4Threads
// threads, kW4Lds bytes of dynamic LDS and at most one workgroup per CU.
// KMASK: K % 8 != 0 (B K-tiled); ODD: an output width is odd; PAIRS: A in
// 64-deep slots (kW4PLds bytes of LDS).
template <bool KMASK, bool ODD, bool PAIRS>
__device__ __forceinline__ void gemm_w4_persistent(const W4Gemm& g) {
  const int G = static_cast<int>(gridDim.x);
  const int p = static_cast<int>(xcd_remap(blockIdx.x, gridDim.x));
  if (p >= g.tiles) return;
  const int n_my = (g.tiles - p + G - 1) / G;
  // K tiles per output tile; with PAIRS an odd count gets one more, all past
  // K (its copies read zero), so that pairs never straddle two output tiles
  const int kt_k = static_cast<int>(ceil_div(g.K, kW4K));
  const int kt = PAIRS ? (kt_k + 1) & ~1 : kt_k;
  const int kl = kt_k - 1;  // the K tile that holds element K - 1
  const W4Walk wk = w4_walk(g, p, G);
  const W4Lane L = w4_lane<PAIRS>(g);

  W4CopyCursor cc;
  cc.c = W4Cursor{0, 0, 0};
  w4_tile_at(g, wk, cc.c);
  cc.k = 0;
  cc.d = w4_copy_desc(g, cc.c, n_my);
  W4PairCursor ap;
  if constexpr (PAIRS) {
    ap.c = cc.c;
    ap.kp = 0;
    ap.ra = cc.d.ra;
    ap.sa = 0;
    // A pairs 0 and 1 (steps 0 .. 3) into slots 0 and 1, B of steps 0 .. 2
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      uint32_t oe, oo;
      w4p_oob(g, L, ap.kp * (2 * kW4K), oe, oo);
#pragma unroll
      for (int j = 0; j < 8; ++j) w4p_copy_a(L, ap.ra, ap.kp * (2 * kW4K), (j & 1) ? oo : oe, pp * kW4PairBytes, j);
      w4p_advance(g, ap, kt, n_my, wk);
    }
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      const int k3 = cc.k * kW4K;
      const uint32_t oob = ~static_cast<uint32_t>(k3 + L.kchunk - g.K) & kW4Oob;
#pragma unroll
      for (int q = 0; q < 4; ++q) w4p_copy_b(L, cc.d.rb, k3, oob, s * kW4StageBytes, q);
      w4_copy_advance(g, cc, kt, n_my, wk);
    }
  } else {
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      w4_copy(g, L, cc.d, cc.k * kW4K, L.lds + s * kW4StageBytes, L.lds + kW4BBase + s * kW4StageBytes);
      w4_copy_advance(g, cc, kt, n_my, wk);
    }
  }
  W4Frags f[2];
  f32x16 acc[4][4];
  uint32_t raw[128];
#pragma unroll
  for (int e = 0; e < 128; ++e) raw[e] = 0u;  // stored against an empty range by the first tile
  W4Cursor oc{0, 0, 0};
  w4_tile_at(g, wk, oc);
  W4Out od = w4_out_desc(g, L, oc, false);  // nothing to store before the first tile
  w4_wait_vm<0>();
  w4_lds_barrier(f[1]);
  if constexpr (PAIRS) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      f[0].a[i] = *reinterpret_cast<const w4_lds_u32x4*>(static_cast<uintptr_t>(L.a0 + L.lds + i * 4096));
#pragma unroll
    for (int i = 0; i < 4; ++i)
      f[0].b[i] = *reinterpret_cast<const w4_lds_u32x4*>(static_cast<uintptr_t>(L.b0 + i * 2048));
  } else {
    w4_read(L.a0, L.b0, f[0]);
  }
  int h = 0;
  for (int q = 0; q < n_my; ++q) {
    if constexpr (PAIRS) {
      w4p_ktile<0, KMASK, ODD>(g, L, h + 0, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<1, KMASK, ODD>(g, L, h + 1, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<2, KMASK, ODD>(g, L, h + 2, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<3, KMASK, ODD>(g, L, h + 3, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<4, KMASK, ODD>(g, L, h + 4, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<5, KMASK, ODD>(g, L, h + 5, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<6, KMASK, ODD>(g, L, h + 6, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<7, KMASK, ODD>(g, L, h + 7, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<8, KMASK, ODD>(g, L, h + 8, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<9, KMASK, ODD>(g, L, h + 9, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<10, KMASK, ODD>(g, L, h + 10, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<11, KMASK, ODD>(g, L, h + 11, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<12, KMASK, ODD>(g, L, h + 12, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<13, KMASK, ODD>(g, L, h + 13, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<14, KMASK, ODD>(g, L, h + 14, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<15, KMASK, ODD>(g, L, h + 15, cc, ap, kt, n_my, wk, od, raw, f, acc);
      w4p_ktile<16, KMASK, ODD>(g, L, h + 16, cc, ap, kt, n_my, wk, od, raw, f, acc, kl == 16);
      w4p_ktile<17, KMASK, ODD>(g, L, h + 17, cc, ap, kt, n_my, wk, od, raw, f, acc, kl == 17);
      for (int t = kW4PMinKTiles; t < kt; t += 2) {
        w4p_ktile<18, KMASK, ODD>(g, L, h + t, cc, ap, kt, n_my, wk, od, raw, f, acc, kl == t);
        w4p_ktile<19, KMASK, ODD>(g, L, h + t + 1, cc, ap, kt, n_my, wk, od, raw, f, acc, kl == t + 1);
      }
    } else {
      w4_ktile<0, KMASK, ODD>(g, L, h + 0, cc, kt, n_my, wk, od, raw, f, acc);
      w4_ktile<1, KMASK, ODD>(g, L, h + 1, cc, kt, n_my, wk, od, raw, f, acc);
      w4_ktile<2, KMASK, ODD>(g, L, h + 2, cc, kt, n_my, wk, od, raw, f, acc);
      w4_ktile<3, KMASK, ODD>(g, L, h + 3, cc, kt, n_my, wk, od, raw, f, acc);
      w4_ktile<4, KMASK, ODD>(g, L, h + 4, cc, kt, n_my, wk, od, raw, f, acc);
      w4_ktile<5, KMASK, ODD>(g, L, h + 5, cc, kt, n_my, wk, od, raw, f, acc);
      w4_ktile<6, KMASK, ODD>(g, L, h + 6, cc, kt, n_my, wk, od, raw, f, acc);
      w4_ktile<7, KMASK, ODD>(g, L, h + 7, cc, kt, n_my, wk, od, raw, f, acc);
      w4_ktile<8, KMASK, ODD>(g, L, h + 8, cc, kt, n_my, wk, od, raw, f, acc);
      w4_ktile<9, KMASK, ODD>(g, L, h + 9, cc, kt, n_my, wk, od, raw, f, acc, kl == 9);
      for (int t = 10; t < kt; ++t)
        w4_ktile<10, KMASK, ODD>(g, L, h + t, cc, kt, n_my, wk, od, raw, f, acc, kl == t);
    }
    // bf16 pairs only here (the stores of the next tile's first K tiles do
    // the lane shuffles, in the shadow of its MFMAs)
#pragma unroll
    for (int b = 0; b < 16; ++b) w4_convert_block(acc[b >> 2][b & 3], b, raw);
    h += kt;
    od = w4_out_desc(g, L, oc, true);
    if constexpr (ODD) {
      if (q + 1 < n_my) w4_store_tails(od, raw);  // the last tile's go out with w4_flush
    }
    w4_next_tile(g, wk, oc);
  }
  w4_flush<ODD>(od, raw);
  w4_wait_vm<0>();  // no copy may still be writing LDS when the workgroup ends
}

}  // namespace compact
