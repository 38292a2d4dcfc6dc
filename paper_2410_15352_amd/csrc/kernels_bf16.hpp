// bf16 kernels of the CompAct layer (gfx950, MFMA 32x32x16, fp32 accumulate).
//
//   k_fwd_bf16          [y | z] = x [W | P]     (CompAct Alg. 1)
//   k_pstream_t_bf16    P^T panel (r x n, bf16, unscaled) for the forward
//   k_dx_bf16           dx = dL/do W^T          (Alg. 2, second line)
//   k_ghat_bf16         split-K partials of G^ = z^T dL/do (Alg. 2, first line)
//   k_splitk_reduce     fixed-order sum of the split-K partials
#pragma once
#include "gemm_bf16.hpp"
#include "kernels_common.hpp"

namespace compact {

// Workgroups per CU the register budget is tuned for: wave tiles of 128x128 or
// more keep 256 accumulators per lane and need the whole 512-register file.
__host__ __device__ constexpr int occupancy_for(int bm, int bn, int wgm, int wgn) {
  return (bm / wgm) * (bn / wgn) >= 128 * 128 ? 1 : 2;
}

// ------------------------------- forward -----------------------------------
struct FwdParams {
  const uint16_t* x;
  int64_t ldx;
  const uint16_t* W;
  int64_t ldw;
  uint16_t* y;
  int64_t ldy;
  uint16_t* z;
  int64_t ldz;
  const uint16_t* pt;  // materialised P^T = bf16(pscale G^T) (r rows, K = n contiguous), or null
  int64_t ldpt;
  int64_t T, n, m, r;
  PhiloxKey key;
  ProjDesc proj;
  float pscale;      // 1/sqrt(r) (Gaussian) or 1/sqrt(s) (sparse) applied before rounding; 1 for the identity
  int tiles_y;       // column tiles covering y (m columns)
  int tiles_z;       // column tiles covering z (r columns)
};

template <int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(WGM* WGN* kWave, occupancy_for(BM, BN, WGM, WGN)) void k_fwd_bf16(FwdParams p) {
  constexpr int NT = WGM * WGN * kWave;
  constexpr int FM = BM / WGM / 32, FN = BN / WGN / 32;
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  const uint32_t logical = xcd_remap(blockIdx.x, gridDim.x);
  const int ncols = p.tiles_y + p.tiles_z;
  const int rt = static_cast<int>(logical / ncols), ct = static_cast<int>(logical % ncols);
  const int64_t row0 = static_cast<int64_t>(rt) * BM;
  KMajorLoader<BM, NT> la{p.x, p.ldx, p.T, p.n, row0};
  f32x16 acc[FM][FN];
  if (ct < p.tiles_y) {
    const int64_t col0 = static_cast<int64_t>(ct) * BN;
    MNMajorLoader<BN, NT> lb{p.W, p.ldw, p.m, p.n, col0};
    gemm_mainloop<BM, BN, WGM, WGN>(la, lb, 0, p.n, lds, acc);
    store_tile_bf16_lds<BM, BN, WGM, WGN>(acc, lds, p.y, p.ldy, p.T, p.m, row0, col0, 1.0f);
  } else {
    const int64_t col0 = static_cast<int64_t>(ct - p.tiles_y) * BN;
    if (p.pt != nullptr) {
      KMajorLoader<BN, NT> lb{p.pt, p.ldpt, p.r, p.n, col0};
      gemm_mainloop<BM, BN, WGM, WGN>(la, lb, 0, p.n, lds, acc);
    } else {
      PGenLoader<BN, NT> lb{p.key, p.n, p.r, col0, p.proj, p.pscale};
      gemm_mainloop<BM, BN, WGM, WGN>(la, lb, 0, p.n, lds, acc);
    }
    store_tile_bf16_lds<BM, BN, WGM, WGN>(acc, lds, p.z, p.ldz, p.T, p.r, row0, col0, 1.0f);
  }
}

// P^T panel for the forward: out[j * ld + i] = bf16(scale x stream element
// (i, j)), or the identity (scale 1).  One thread per quad (4 rows of one
// column); columns i >= n of the padded rows are written as zero.
__global__ void k_pstream_t_bf16(ProjDesc d, PhiloxKey key, int64_t n, float scale, uint16_t* out, int64_t ld) {
  const int64_t u = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (u >= proj_t_units(d.kind, d.r, ld)) return;
  proj_t_unit(d, key, n, scale, PanelOut{out, ld, 0}, 0, ld, u);
}

// Element (c, i) of `out` = in[i * ldi + c] for i < rows, c < cols (bf16),
// through a 64 x 64 LDS tile.  256 threads; each moves two 16-byte chunks:
// loads 8 consecutive columns of one row, scatters them down the transposed
// tile, and stores 8 consecutive rows of one output row (one 16-byte store:
// 8-aligned runs of k stay inside a 32-wide K tile of a K-tiled panel).  ldi
// and the panel's ld are multiples of 8 and both pointers 16-byte aligned;
// partial chunks at the edges go element by element.
__device__ __forceinline__ void transpose_tile_bf16(const uint16_t* in, int64_t ldi, int64_t rows, int64_t cols,
                                                    const PanelOut& out, int tiles_c, int block) {
  __shared__ __attribute__((aligned(16))) uint16_t tile[64][72];  // tile[c][i]; rows padded to 144 bytes
  const int t = threadIdx.x;
  const int64_t r0 = static_cast<int64_t>(block / tiles_c) * 64;
  const int64_t c0 = static_cast<int64_t>(block % tiles_c) * 64;
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const int id = t + 256 * p, i = id >> 3, cc = (id & 7) * 8;
    const int64_t gi = r0 + i, gc = c0 + cc;
    uint16_t v[8];
    if (gi < rows && gc + 8 <= cols) {
      const u32x4 w = *reinterpret_cast<const u32x4*>(in + gi * ldi + gc);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] = static_cast<uint16_t>(w[e]);
        v[2 * e + 1] = static_cast<uint16_t>(w[e] >> 16);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = (gi < rows && gc + e < cols) ? in[gi * ldi + gc + e] : uint16_t(0);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) tile[cc + e][i] = v[e];
  }
  __syncthreads();
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const int id = t + 256 * p, c = id >> 3, ii = (id & 7) * 8;
    const int64_t gc = c0 + c, gi = r0 + ii;
    if (gc >= cols || gi >= rows) continue;
    // the tile holds zeros past `rows`: a chunk that straddles the end is
    // written whole, so that the operand is zero up to the next multiple of 8
    // (the panel's K extent is a multiple of 32)
    *reinterpret_cast<u32x4*>(panel_at(out, gc, gi)) = *reinterpret_cast<const u32x4*>(&tile[c][ii]);
  }
}

// Staging of the persistent forward GEMM's B operand in one launch: the first
// workgroups write the P^T panels of the projections (one quad per thread, as
// k_pstream_t_bf16), the rest transpose W into W^T (64 x 64 tiles).  The P
// stream is arithmetic latency bound and the transpose memory bound, so they
// overlap.  Projection j's panel P_j^T [r_j][ldb] starts at row row_off[j] of
// the staged operand.
constexpr int kMaxGroup = 8;  // projections sharing one input

// ---------------------------------------------------------------------------
// Gather-add z of a sparse projection (COMPACT_PROJ_GATHER).  Row i of S has
// s <= kGatherMaxS draws (pstream.hpp); its table row holds s entries
//   column | bf16(S[i][column] * scale) << 16
// at the first draw of each column (the signs of the row's draws on that
// column summed), and kGatherSkip where a draw repeats an earlier column or
// the signs cancel.  The value half, read as fp32 bits, is that bf16 value
// exactly: the same P = bf16(S / sqrt(s)) element the P^T panel holds.
constexpr int kGatherMaxS = 16;
constexpr uint32_t kGatherSkip = 0xFFFFu;  // column of a skipped entry

__device__ __forceinline__ void gather_table_row(const ProjDesc& d, PhiloxKey key, float scale, uint32_t i,
                                                 uint32_t* row) {
  uint32_t h[kGatherMaxS];
  float v[kGatherMaxS];
#pragma unroll
  for (int p = 0; p < kGatherMaxS / 2; ++p) {
    h[2 * p] = h[2 * p + 1] = kGatherSkip;
    v[2 * p] = v[2 * p + 1] = 0.0f;
    if (2 * p < d.s) {
      sjlt_pair(key, i, static_cast<uint32_t>(p), static_cast<uint32_t>(d.r), h[2 * p], v[2 * p], h[2 * p + 1],
                v[2 * p + 1]);
      if (2 * p + 1 >= d.s) {  // odd s: the pair's second draw is not taken
        h[2 * p + 1] = kGatherSkip;
        v[2 * p + 1] = 0.0f;
      }
    }
  }
  // a later draw on a column adds its sign to the first draw on it
#pragma unroll
  for (int q = 1; q < kGatherMaxS; ++q)
#pragma unroll
    for (int p = 0; p < q; ++p)
      if (h[q] != kGatherSkip && h[p] == h[q]) {
        v[p] += v[q];
        h[q] = kGatherSkip;
      }
#pragma unroll
  for (int q = 0; q < kGatherMaxS; ++q)
    if (q < d.s)
      row[q] = (h[q] == kGatherSkip || v[q] == 0.0f)
                   ? kGatherSkip
                   : (h[q] | (static_cast<uint32_t>(f32_to_bf16(v[q] * scale)) << 16));
}

struct FwdStage {
  const uint16_t* W;
  int64_t ldw, n, m;      // W [n x m]; m = the sum of the projections' widths
  PanelOut b;             // staged operand (K-tiled): W^T in rows 0 .. m-1
  int64_t ldb;            // its K extent (a multiple of 32)
  int count;
  int kind, sparse_s;     // projection kind and draws per row (sparse)
  int tiles_c;            // ceil(m / 64)
  int pt_begin[kMaxGroup + 1];  // first P^T workgroup of each projection
  int64_t row_off[kMaxGroup];
  int64_t r[kMaxGroup];
  PhiloxKey key[kMaxGroup];
  float pscale[kMaxGroup];
  uint32_t* table[kMaxGroup];   // gather-add tables ([n][s]) instead of P^T rows, or NULL
};

__global__ __launch_bounds__(256) void k_fwd_stage_bf16(FwdStage a) {
  const int b = static_cast<int>(blockIdx.x);
  if (b < a.pt_begin[a.count]) {
    int j = 0;
    while (j + 1 < a.count && a.pt_begin[j + 1] <= b) ++j;
    const int64_t u = static_cast<int64_t>(b - a.pt_begin[j]) * 256 + threadIdx.x;
    const ProjDesc d{a.kind, static_cast<int>(a.r[j]), a.sparse_s};
    if (a.table[j] != nullptr) {  // one table row per thread
      if (u < a.n) gather_table_row(d, a.key[j], a.pscale[j], static_cast<uint32_t>(u), a.table[j] + u * a.sparse_s);
      return;
    }
    if (u >= proj_t_units(a.kind, a.r[j], a.ldb)) return;
    proj_t_unit(d, a.key[j], a.n, a.pscale[j], a.b, a.row_off[j], a.ldb, u);
  } else {
    transpose_tile_bf16(a.W, a.ldw, a.n, a.m, a.b, a.tiles_c, b - a.pt_begin[a.count]);
  }
}

// z_j = x P_j for sparse projections by gather-add (COMPACT_PROJ_GATHER).
// One workgroup is one wave: lane L owns token t = 64 b + L and an fp32 row of
// kGatherChunk columns of z_j in LDS (plus one dummy column that takes the
// skipped entries).  For each input feature i in order and each of the s
// table entries of row i in order, the lane adds x[t][i] * P[i][c] (exact in
// fp32: two bf16 factors) into column c of its row; the entry is the same for
// every lane, so the work per entry is one multiply, one address add and one
// LDS add, with the table read through the scalar cache.  Rows of 129 floats
// put the 64 lanes of an LDS access on distinct banks.  The sum is rounded
// once to bf16 and stored row by row (16-byte stores).
// Workgroup b: token block b / chunks, column chunk b % chunks (the chunks of
// a token block are adjacent in the grid, so x is read from memory once).
constexpr int kGatherChunk = 128;
constexpr int kGatherTok = 64;
constexpr int kGatherRow = kGatherChunk + 1;

struct GatherLayer {
  const uint32_t* table;  // [n][s]
  uint16_t* z;            // first column of z_j
  int r;
};

struct GatherParams {
  const uint16_t* x;
  int64_t ldx, T, ldz;
  int n, s;
  int count;
  GatherLayer layer[kMaxGroup];
  int chunk_begin[kMaxGroup + 1];  // first column chunk of each projection
};

__global__ __launch_bounds__(kGatherTok) void k_sjl_gather(GatherParams g) {
  __shared__ float acc[kGatherTok * kGatherRow];
  const int chunks = g.chunk_begin[g.count];
  const int b = static_cast<int>(blockIdx.x);
  const int tb = b / chunks, ch = b - tb * chunks;
  const int l = batch_layer_of(g.chunk_begin, g.count, ch);
  const GatherLayer& L = g.layer[l];
  const uint32_t c0 = static_cast<uint32_t>(ch - g.chunk_begin[l]) * kGatherChunk;
  const int lane = static_cast<int>(threadIdx.x);
  const int64_t t = static_cast<int64_t>(tb) * kGatherTok + lane;
  const bool live = t < g.T;
  float* my = acc + lane * kGatherRow;
  for (int c = 0; c < kGatherRow; ++c) my[c] = 0.0f;
  // lanes past T read the last token's row and store nothing; the 16-byte
  // chunk holding x[t][i0 .. i0 + 7] lies inside the row's leading dimension
  // (a multiple of 8), and features past n are not used
  const uint16_t* xr = g.x + (live ? t : g.T - 1) * g.ldx;
  // the table is read-only in this kernel: read through the constant address
  // space, so that wave-uniform reads become scalar loads
  typedef __attribute__((address_space(4))) const uint32_t const_u32;
  const_u32* tab = (const_u32*)(L.table);
  const int s = g.s;
  u32x4 xn = *reinterpret_cast<const u32x4*>(xr);
  for (int i0 = 0; i0 < g.n; i0 += 8) {
    const u32x4 xv = xn;
    if (i0 + 8 < g.n) xn = *reinterpret_cast<const u32x4*>(xr + i0 + 8);  // the next chunk, one step ahead
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (i0 + e >= g.n) break;
      const uint32_t w = xv[e >> 1];
      const float xf = __uint_as_float((e & 1) ? (w & 0xFFFF0000u) : (w << 16));
      // the table row is the same for every lane: a wave-uniform index, so
      // its entries come through the scalar cache
      const int row = __builtin_amdgcn_readfirstlane(i0 + e);
      const_u32* ent = tab + static_cast<int64_t>(row) * s;
      for (int q = 0; q < s; ++q) {
        const uint32_t en = ent[q];
        const uint32_t d = min((en & 0xFFFFu) - c0, static_cast<uint32_t>(kGatherChunk));
        __hip_atomic_fetch_add(my + d, xf * __uint_as_float(en & 0xFFFF0000u), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    }
  }
  if (!live) return;
  const int cnt = min(kGatherChunk, L.r - static_cast<int>(c0));
  uint16_t* zr = L.z + t * g.ldz + c0;
  int c = 0;
  for (; c + 8 <= cnt; c += 8) {
    u32x4 o;
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] = pack_bf16x2(my[c + 2 * k], my[c + 2 * k + 1]);
    *reinterpret_cast<u32x4*>(zr + c) = o;
  }
  for (; c < cnt; ++c) zr[c] = f32_to_bf16(my[c]);
}

// The dx GEMM's B operand, W [n x m] (row R = input feature, K = m), copied
// into the K-tiled layout: element (R, k) of `out` = W[R * ldw + k] for R < n,
// k < m, and zero for m <= k < round_up(m, 8).  One thread per 8 consecutive
// k of one row: a 16-byte load and a 16-byte store (the last chunk of a row
// element by element when m % 8 != 0: the row's padding is not read).
__global__ __launch_bounds__(256) void k_stage_rows_bf16(const uint16_t* W, int64_t ldw, int64_t n, int64_t m,
                                                         PanelOut out) {
  const int64_t kq = ceil_div(m, 8);
  const int64_t u = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (u >= n * kq) return;
  const int64_t row = u / kq, k = (u - row * kq) * 8;
  u32x4 v;
  if (k + 8 <= m) {
    v = *reinterpret_cast<const u32x4*>(W + row * ldw + k);
  } else {
    uint16_t e[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) e[i] = k + i < m ? W[row * ldw + k + i] : uint16_t(0);
#pragma unroll
    for (int d = 0; d < 4; ++d) v[d] = static_cast<uint32_t>(e[2 * d]) | (static_cast<uint32_t>(e[2 * d + 1]) << 16);
  }
  *reinterpret_cast<u32x4*>(panel_at(out, row, k)) = v;
}

// Unscaled fp32 stream of any projection (n x r, leading dimension ld), one
// thread per quad of rows of one column: the exported test generator.
__global__ void k_projection_f32(ProjDesc d, PhiloxKey key, int64_t n, float* out, int64_t ld) {
  const int64_t nq = (n + 3) / 4;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (q >= nq * d.r) return;
  const int64_t p = q % nq, j = q / nq;
  float g[4];
  proj_quad(d, key, 4 * p, j, g);
  for (int e = 0; e < 4; ++e) {
    const int64_t i = 4 * p + e;
    if (i < n) out[i * ld + j] = g[e];
  }
}

// Unscaled fp32 stream G (n x r, leading dimension ld): the standalone P tile
// generator, exported for bitwise tests.
__global__ void k_pstream_f32(PhiloxKey key, int64_t n, int64_t r, float* out, int64_t ld) {
  const int64_t nq = (n + 3) / 4;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (q >= nq * r) return;
  const int64_t p = q % nq, j = q / nq;
  float g[4];
  pstream_quad(key, static_cast<uint32_t>(p), static_cast<uint32_t>(j), g);
  for (int e = 0; e < 4; ++e) {
    const int64_t i = 4 * p + e;
    if (i < n) out[i * ld + j] = g[e];
  }
}

__global__ void k_boxmuller(const uint32_t* a, const uint32_t* b, float* ge, float* go,
                            int64_t count) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= count) return;
  float g0, g1;
  pstream_pair(a[e], b[e], g0, g1);
  ge[e] = g0;
  go[e] = g1;
}

// ------------------------------- backward ----------------------------------
struct DxParams {
  const uint16_t* dy;
  int64_t lddy;
  const uint16_t* W;
  int64_t ldw;
  uint16_t* dx;
  int64_t lddx;
  int64_t T, n, m;
  int tiles_n;
};

template <int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(WGM* WGN* kWave, occupancy_for(BM, BN, WGM, WGN)) void k_dx_bf16(DxParams p) {
  constexpr int NT = WGM * WGN * kWave;
  constexpr int FM = BM / WGM / 32, FN = BN / WGN / 32;
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  const uint32_t logical = xcd_remap(blockIdx.x, gridDim.x);
  const int rt = static_cast<int>(logical / p.tiles_n), ct = static_cast<int>(logical % p.tiles_n);
  const int64_t row0 = static_cast<int64_t>(rt) * BM, col0 = static_cast<int64_t>(ct) * BN;
  KMajorLoader<BM, NT> la{p.dy, p.lddy, p.T, p.m, row0};
  KMajorLoader<BN, NT> lb{p.W, p.ldw, p.n, p.m, col0};
  f32x16 acc[FM][FN];
  gemm_mainloop<BM, BN, WGM, WGN>(la, lb, 0, p.m, lds, acc);
  store_tile_bf16_lds<BM, BN, WGM, WGN>(acc, lds, p.dx, p.lddx, p.T, p.n, row0, col0, 1.0f);
}

struct GhatParams {
  const uint16_t* z;
  int64_t ldz;
  const uint16_t* dy;
  int64_t lddy;
  float* part;        // [splits][tiles_r * BM][tiles_m * BN]
  int64_t T, r, m;
  int tiles_r, tiles_m, splits;
  int64_t split_len;  // tokens per split, a multiple of 64
};

template <int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(WGM* WGN* kWave, occupancy_for(BM, BN, WGM, WGN)) void k_ghat_bf16(GhatParams p) {
  constexpr int NT = WGM * WGN * kWave;
  constexpr int FM = BM / WGM / 32, FN = BN / WGN / 32;
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  const uint32_t logical = xcd_remap(blockIdx.x, gridDim.x);
  const int tiles = p.tiles_r * p.tiles_m;
  // order (split, column tile, row tile): the row tiles that read the same
  // dL/do columns are adjacent, hence on the same XCD at the same time
  const int split = static_cast<int>(logical / tiles), tile = static_cast<int>(logical % tiles);
  const int ct = tile / p.tiles_r, rt = tile % p.tiles_r;
  const int64_t row0 = static_cast<int64_t>(rt) * BM, col0 = static_cast<int64_t>(ct) * BN;
  const int64_t k_begin = split * p.split_len;
  const int64_t k_end = k_begin + p.split_len < p.T ? k_begin + p.split_len : p.T;
  MNMajorLoader<BM, NT> la[2] = {{p.z, p.ldz, p.r, p.T, row0}, {p.z, p.ldz, p.r, p.T, row0}};
  MNMajorLoader<BN, NT> lb[2] = {{p.dy, p.lddy, p.m, p.T, col0}, {p.dy, p.lddy, p.m, p.T, col0}};
  f32x16 acc[FM][FN];
  gemm_mainloop_deep<BM, BN, WGM, WGN>(la, lb, k_begin, k_end, lds, acc);
  const int64_t ldp = static_cast<int64_t>(p.tiles_m) * BN;
  float* out = p.part + static_cast<int64_t>(split) * (p.tiles_r * BM) * ldp;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int64_t r0 = row0 + wm * (BM / WGM), c0 = col0 + wn * (BN / WGN);
  for_each_acc(acc, lane, [&](int row, int col, float v) { out[(r0 + row) * ldp + c0 + col] = v; });
}

// G[j][c] = sum over s = 0 .. splits-1 (in this order) of part[s][j][c]
// (accumulate: G[j][c] + that sum, one addition at the end); four consecutive
// columns per thread (m % 4 == 0), else one.
__global__ void k_splitk_reduce4(const float* part, int splits, int64_t ldp, int64_t plane,
                                 int64_t r, int64_t m, float* G, int accumulate) {
  const int64_t q = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t mq = m / 4;
  if (q >= r * mq) return;
  const int64_t j = q / mq, c = (q % mq) * 4;
  const float* src = part + j * ldp + c;
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
  // sixteen loads in flight (the grid is small: r m / 1024 workgroups), then
  // added in split order
  int k = 0;
  for (; k + 16 <= splits; k += 16) {
    f32x4 v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = *reinterpret_cast<const f32x4*>(src + (k + u) * plane);
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      s.x = s.x + v[u].x;
      s.y = s.y + v[u].y;
      s.z = s.z + v[u].z;
      s.w = s.w + v[u].w;
    }
  }
  for (; k < splits; ++k) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(src + k * plane);
    s.x = s.x + v.x;
    s.y = s.y + v.y;
    s.z = s.z + v.z;
    s.w = s.w + v.w;
  }
  f32x4* dst = reinterpret_cast<f32x4*>(G + j * m + c);
  if (accumulate) {
    const f32x4 g = *dst;
    s.x = g.x + s.x;
    s.y = g.y + s.y;
    s.z = g.z + s.z;
    s.w = g.w + s.w;
  }
  *dst = s;
}

// The reduction for several projections in one launch (one G^ split-K launch
// over a layer table): thread q of layer l sums columns 4 (q mod (m/4 rounded
// up)) .. + 3 of one row over the splits in order; the partial rows are
// 256-column padded, so the 16-byte loads stay inside them.
struct ReduceLayer {
  const float* part;  // [splits][rows][ldp]
  float* G;           // [r][m] dense
  int64_t ldp, plane;
  int r, m, mq;       // mq = ceil(m / 4)
  int vec;            // m % 4 == 0 and G 16-byte aligned: 16-byte stores
};

struct ReduceBatch {
  int count, splits;
  int accumulate;  // G + the sum instead of the sum
  int begin[9];  // first workgroup of each layer; begin[count] = grid
  ReduceLayer layer[8];
};

__global__ void k_splitk_reduce_batched(ReduceBatch b) {
  const int l = batch_layer_of(b.begin, b.count, static_cast<int>(blockIdx.x));
  const ReduceLayer& p = b.layer[l];
  const int64_t q = static_cast<int64_t>(blockIdx.x - b.begin[l]) * blockDim.x + threadIdx.x;
  if (q >= static_cast<int64_t>(p.r) * p.mq) return;
  const int64_t j = q / p.mq, c = (q % p.mq) * 4;
  const float* src = p.part + j * p.ldp + c;
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
  int k = 0;
  for (; k + 16 <= b.splits; k += 16) {
    f32x4 v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = *reinterpret_cast<const f32x4*>(src + (k + u) * p.plane);
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      s.x = s.x + v[u].x;
      s.y = s.y + v[u].y;
      s.z = s.z + v[u].z;
      s.w = s.w + v[u].w;
    }
  }
  for (; k < b.splits; ++k) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(src + k * p.plane);
    s.x = s.x + v.x;
    s.y = s.y + v.y;
    s.z = s.z + v.z;
    s.w = s.w + v.w;
  }
  float* dst = p.G + j * p.m + c;
  if (p.vec) {
    if (b.accumulate) {
      const f32x4 g = *reinterpret_cast<const f32x4*>(dst);
      s.x = g.x + s.x;
      s.y = g.y + s.y;
      s.z = g.z + s.z;
      s.w = g.w + s.w;
    }
    *reinterpret_cast<f32x4*>(dst) = s;
  } else {
    const float e[4] = {s.x, s.y, s.z, s.w};
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (c + u < p.m) dst[u] = b.accumulate ? dst[u] + e[u] : e[u];
  }
}

// G[j][c] = sum over s = 0 .. splits-1 (in this order) of part[s][j][c]
// (accumulate: G[j][c] + that sum).
__global__ void k_splitk_reduce(const float* part, int splits, int64_t ldp, int64_t plane,
                                int64_t r, int64_t m, float* G, int accumulate) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= r * m) return;
  const int64_t j = e / m, c = e % m;
  const float* src = part + j * ldp + c;
  float s = 0.0f;
  for (int k = 0; k < splits; ++k) s += src[k * plane];
  G[e] = accumulate ? G[e] + s : s;
}

}  // namespace compact
