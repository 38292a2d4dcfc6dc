// bf16 kernels of the CompAct layer (gfx950, MFMA 32x32x16, fp32 accumulate).
//
//   k_fwd_bf16          [y | z] = x [W | P]     (CompAct Alg. 1)
//   k_pstream_t_bf16    P^T panel (r x n, bf16, unscaled) for the forward
//   k_dx_bf16           dx = dL/do W^T          (Alg. 2, second line)
//   k_ghat_bf16         split-K partials of G^ = z^T dL/do (Alg. 2, first line)
//   k_splitk_reduce     fixed-order sum of the split-K partials
//   k_decompress_bf16   W <- W - lr alpha P N, P regenerated per row panel in
//                       LDS (Alg. 3, decompression and update)
#pragma once
#include "gemm_bf16.hpp"

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
  int identity;
  float pscale;      // fp32(1/sqrt(r)) applied to G before rounding; 1 for the identity
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
      PGenLoader<BN, NT> lb{p.key, p.n, p.r, col0, p.identity, p.pscale};
      gemm_mainloop<BM, BN, WGM, WGN>(la, lb, 0, p.n, lds, acc);
    }
    store_tile_bf16_lds<BM, BN, WGM, WGN>(acc, lds, p.z, p.ldz, p.T, p.r, row0, col0, 1.0f);
  }
}

// P^T panel for the forward: out[j * ld + i] = bf16(scale * G[i][j]), or the
// identity (scale 1).  One thread per quad (4 rows of one column); columns
// i >= n of the padded rows are written as zero.
__global__ void k_pstream_t_bf16(PhiloxKey key, int64_t n, int64_t r, int identity, float scale,
                                 uint16_t* out, int64_t ld) {
  const int64_t quads_per_row = ld / 4;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (q >= quads_per_row * r) return;
  const int64_t j = q / quads_per_row, i0 = (q % quads_per_row) * 4;
  float g[4] = {0.f, 0.f, 0.f, 0.f};
  if (i0 < n) {
    if (identity) {
      for (int e = 0; e < 4; ++e) g[e] = (i0 + e == j) ? 1.0f : 0.0f;
    } else {
      pstream_quad(key, static_cast<uint32_t>(i0 >> 2), static_cast<uint32_t>(j), g);
      for (int e = 0; e < 4; ++e) g[e] = g[e] * scale;
    }
    for (int e = 0; e < 4; ++e)
      if (i0 + e >= n) g[e] = 0.0f;
  }
  u32x2 v;
  v.x = pack_bf16x2(g[0], g[1]);
  v.y = pack_bf16x2(g[2], g[3]);
  *reinterpret_cast<u32x2*>(out + j * ld + i0) = v;
}

// out[c * ldo + i] = in[i * ldi + c] for i < rows, c < cols (bf16), through a
// 64 x 64 LDS tile.  256 threads; each moves two 16-byte chunks: loads 8
// consecutive columns of one row, scatters them down the transposed tile, and
// stores 8 consecutive rows of one output row.  ldi and ldo are multiples of 8
// and both pointers 16-byte aligned; partial chunks at the edges go element
// by element.
__global__ __launch_bounds__(256) void k_transpose_bf16(const uint16_t* in, int64_t ldi, int64_t rows, int64_t cols,
                                                        uint16_t* out, int64_t ldo, int tiles_c) {
  __shared__ __attribute__((aligned(16))) uint16_t tile[64][72];  // tile[c][i]; rows padded to 144 bytes
  const int t = threadIdx.x;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x / tiles_c) * 64;
  const int64_t c0 = static_cast<int64_t>(blockIdx.x % tiles_c) * 64;
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
    if (gc >= cols) continue;
    const u32x4 w = *reinterpret_cast<const u32x4*>(&tile[c][ii]);
    if (gi + 8 <= rows) {
      *reinterpret_cast<u32x4*>(out + gc * ldo + gi) = w;
    } else {
      for (int e = 0; e < 8 && gi + e < rows; ++e) out[gc * ldo + gi + e] = static_cast<uint16_t>(w[e >> 1] >> (16 * (e & 1)));
    }
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

// G[j][c] = sum over s = 0 .. splits-1 (in this order) of part[s][j][c];
// four consecutive columns per thread (m % 4 == 0), else one.
__global__ void k_splitk_reduce4(const float* part, int splits, int64_t ldp, int64_t plane,
                                 int64_t r, int64_t m, float* G) {
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
  *reinterpret_cast<f32x4*>(G + j * m + c) = s;
}

// G[j][c] = sum over s = 0 .. splits-1 (in this order) of part[s][j][c].
__global__ void k_splitk_reduce(const float* part, int splits, int64_t ldp, int64_t plane,
                                int64_t r, int64_t m, float* G) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= r * m) return;
  const int64_t j = e / m, c = e % m;
  const float* src = part + j * ldp + c;
  float s = 0.0f;
  for (int k = 0; k < splits; ++k) s += src[k * plane];
  G[e] = s;
}

// ------------------------------- update ------------------------------------
struct DecParams {
  void* W;              // bf16 or fp32, n x m
  int64_t ldw;
  int w_f32;
  const uint16_t* N;    // r x m, bf16, leading dimension ldn (multiple of 8)
  int64_t ldn;
  int64_t n, m, r;
  int64_t r_pad;        // round_up(r, 64): panel columns
  PhiloxKey key;
  int identity;
  float coef;           // fp32(lr * alpha / sqrt(r))
  int panels;           // ceil(n / BM)
  int col_groups;       // column groups per panel
  int tiles_m;          // ceil(m / BN)
};

// Panel layout: [BM][r_pad + 8] bf16; the +8 pad puts the rows of one MFMA
// fragment read on distinct LDS banks (r_pad / 8 is even).
template <int BM, int BN, int WGM, int WGN>
__device__ __forceinline__ void decompress_block(const DecParams& p, uint32_t logical) {
  constexpr int NT = WGM * WGN * kWave;
  constexpr int FM = BM / WGM / 32, FN = BN / WGN / 32;
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  const int64_t ldp = p.r_pad + 8;
  uint16_t* Ap = lds;
  const int64_t bs0 = BM * ldp;  // N tile stages at lds + bs0 and lds + bs0 + BN * 64
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int panel = static_cast<int>(logical % p.panels), group = static_cast<int>(logical / p.panels);
  const int64_t row0 = static_cast<int64_t>(panel) * BM;

  // 1. P panel rows row0 .. row0+BM-1, all r_pad columns, generated once.
  {
    const int jgroups = static_cast<int>(p.r_pad / 8);
    const int items = (BM / 4) * jgroups;
    for (int it = tid; it < items; it += NT) {
      const int jg = it % jgroups, qr = it / jgroups;
      const int64_t i0 = row0 + qr * 4, j0 = static_cast<int64_t>(jg) * 8;
      float g[8][4];
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        const int64_t j = j0 + jj;
#pragma unroll
        for (int e = 0; e < 4; ++e) g[jj][e] = 0.0f;
        if (j < p.r && i0 < p.n) {
          if (p.identity) {
#pragma unroll
            for (int e = 0; e < 4; ++e) g[jj][e] = (i0 + e == j) ? 1.0f : 0.0f;
          } else {
            pstream_quad(p.key, static_cast<uint32_t>(i0 >> 2), static_cast<uint32_t>(j), g[jj]);
          }
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        u32x4 v;
        v.x = pack_bf16x2(g[0][e], g[1][e]);
        v.y = pack_bf16x2(g[2][e], g[3][e]);
        v.z = pack_bf16x2(g[4][e], g[5][e]);
        v.w = pack_bf16x2(g[6][e], g[7][e]);
        if (i0 + e >= p.n) v = u32x4{0u, 0u, 0u, 0u};
        *reinterpret_cast<u32x4*>(Ap + (qr * 4 + e) * ldp + j0) = v;
      }
    }
  }
  __syncthreads();

  // 2. Column tiles of this group: acc = P_panel N_tile, then W -= coef acc.
  //    The W tile (BM x BN) is read with 16-byte loads issued before the N tile
  //    and the MFMAs, so its latency overlaps them; coef * acc is staged in LDS
  //    (the N stages are free after the K loop) and W is written back in 16-byte
  //    chunks.
  const int per = (p.tiles_m + p.col_groups - 1) / p.col_groups;
  const int ct_begin = group * per;
  const int ct_end = ct_begin + per < p.tiles_m ? ct_begin + per : p.tiles_m;
  const int lr = lane & 31, lh = lane >> 5;
  const int kt_count = static_cast<int>(p.r_pad / kBK);
  constexpr int kWElems = 8;                                   // elements per 16-byte bf16 chunk
  constexpr int kWChunks = BM * BN / kWElems / NT;             // bf16 chunks per thread
  static_assert(BM * BN % (kWElems * NT) == 0, "W tile split");
  constexpr int kCpr = BN / kWElems;                           // chunks per W-tile row
  float* stage = reinterpret_cast<float*>(lds + bs0);          // BM x (BN + 4) fp32 after the K loop
  constexpr int kSld = BN;
  static_assert(BM * kSld * 4 <= 2 * BN * kBK * 2, "staging fits in the N stages");
  for (int ct = ct_begin; ct < ct_end; ++ct) {
    const int64_t col0 = static_cast<int64_t>(ct) * BN;
    // (a) W tile loads (bf16: one 16-byte chunk = 8 columns; fp32: two)
    u32x4 wreg[kWChunks][2];
#pragma unroll
    for (int i = 0; i < kWChunks; ++i) {
      const int c = tid + i * NT;
      const int row = c / kCpr, cc = c % kCpr;
      int64_t gr = row0 + row;
      gr = gr < p.n ? gr : p.n - 1;
      int64_t gc = col0 + cc * kWElems;
      const int64_t c_last = (p.m - 1) & ~int64_t(kWElems - 1);
      gc = gc < p.m ? gc : c_last;
      if (p.w_f32) {
        const float* src = static_cast<const float*>(p.W) + gr * p.ldw + gc;
        wreg[i][0] = *reinterpret_cast<const u32x4*>(src);
        wreg[i][1] = *reinterpret_cast<const u32x4*>(src + 4);
      } else {
        wreg[i][0] = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(p.W) + gr * p.ldw + gc);
      }
    }
    // (b) acc = P_panel[:, k] N[k, col0 ..] over the rank
    MNMajorLoader<BN, NT> lb{p.N, p.ldn, p.m, p.r, col0};
    f32x16 acc[FM][FN];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[fm][fn][v] = 0.0f;
    lb.fetch(0, tid);
    lb.commit(lds + bs0, tid);
    __syncthreads();
    for (int kt = 0; kt < kt_count; ++kt) {
      const int64_t cur = bs0 + (kt & 1) * (BN * kBK);
      const int64_t nxt = bs0 + ((kt + 1) & 1) * (BN * kBK);
      const bool more = kt + 1 < kt_count;
      if (more) lb.fetch(static_cast<int64_t>(kt + 1) * kBK, tid);
#pragma unroll
      for (int kk = 0; kk < kBK / 16; ++kk) {
        u32x4 a[FM], b[FN];
        const int k = kk * 16 + lh * 8;
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
          a[fm] = *reinterpret_cast<const u32x4*>(Ap + (wm * FM * 32 + fm * 32 + lr) * ldp +
                                                  kt * kBK + k);
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
          b[fn] = *reinterpret_cast<const u32x4*>(lds + cur + tile_off(wn * FN * 32 + fn * 32 + lr, k));
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
          for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma32x32x16(a[fm], b[fn], acc[fm][fn]);
      }
      if (more) lb.commit(lds + nxt, tid);
      __syncthreads();
    }
    // (c) d = coef * acc into the LDS staging tile (row-major, fp32)
    const float coef = p.coef;
    {
      const int r0 = wm * (BM / WGM), c0 = wn * (BN / WGN);
      for_each_acc(acc, lane, [&](int row, int col, float v) {
        const float d = coef * v;
        stage[(r0 + row) * kSld + c0 + col] = d;
      });
    }
    __syncthreads();
    // (d) W = W - d, 16-byte chunks
#pragma unroll
    for (int i = 0; i < kWChunks; ++i) {
      const int c = tid + i * NT;
      const int row = c / kCpr, cc = c % kCpr;
      const int64_t gr = row0 + row, gc = col0 + cc * kWElems;
      if (gr >= p.n || gc >= p.m) continue;
      const float* dsrc = stage + row * kSld + cc * kWElems;
      const f32x4 d0 = *reinterpret_cast<const f32x4*>(dsrc);
      const f32x4 d1 = *reinterpret_cast<const f32x4*>(dsrc + 4);
      const float dv[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
      const int cnt = gc + kWElems <= p.m ? kWElems : static_cast<int>(p.m - gc);
      if (p.w_f32) {
        float* dst = static_cast<float*>(p.W) + gr * p.ldw + gc;
        const uint32_t wbits[8] = {wreg[i][0].x, wreg[i][0].y, wreg[i][0].z, wreg[i][0].w,
                                   wreg[i][1].x, wreg[i][1].y, wreg[i][1].z, wreg[i][1].w};
        float out[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) out[e] = __uint_as_float(wbits[e]) - dv[e];
        if (cnt == kWElems) {
          *reinterpret_cast<f32x4*>(dst) = f32x4{out[0], out[1], out[2], out[3]};
          *reinterpret_cast<f32x4*>(dst + 4) = f32x4{out[4], out[5], out[6], out[7]};
        } else {
          for (int e = 0; e < cnt; ++e) dst[e] = out[e];
        }
      } else {
        uint16_t* dst = static_cast<uint16_t*>(p.W) + gr * p.ldw + gc;
        const uint32_t wp[4] = {wreg[i][0].x, wreg[i][0].y, wreg[i][0].z, wreg[i][0].w};
        uint32_t outp[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = __uint_as_float(wp[e] << 16) - dv[2 * e];
          const float hi = __uint_as_float(wp[e] & 0xFFFF0000u) - dv[2 * e + 1];
          outp[e] = pack_bf16x2(lo, hi);
        }
        if (cnt == kWElems) {
          *reinterpret_cast<u32x4*>(dst) = u32x4{outp[0], outp[1], outp[2], outp[3]};
        } else {
          for (int e = 0; e < cnt; ++e) dst[e] = static_cast<uint16_t>(outp[e >> 1] >> (16 * (e & 1)));
        }
      }
    }
    __syncthreads();  // the staging tile is the next column tile's N stage
  }
}

template <int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(WGM* WGN* kWave, 1) void k_decompress_bf16(DecParams p) {
  decompress_block<BM, BN, WGM, WGN>(p, xcd_remap(blockIdx.x, gridDim.x));
}

struct DecBatch {
  int count;
  int begin[kBatchLayers + 1];
  DecParams layer[kBatchLayers];
};

template <int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(WGM* WGN* kWave, 1) void k_decompress_batched(DecBatch d) {
  const int b = static_cast<int>(xcd_remap(blockIdx.x, gridDim.x));
  const int l = batch_layer_of(d.begin, d.count, b);
  decompress_block<BM, BN, WGM, WGN>(d.layer[l], static_cast<uint32_t>(b - d.begin[l]));
}

}  // namespace compact
