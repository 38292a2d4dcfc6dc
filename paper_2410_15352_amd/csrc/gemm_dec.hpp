// Decompression and update of Alg. 3 for gfx950:  W <- W - coef (P N), with
// P = bf16(G) [n x r] (the raw normals of the P stream, staged once per step as
// P^T [r][ldpt] by the Adam launch), N [r x m] bf16 from Adam, coef =
// fp32(lr alpha / sqrt(r)).  The product is HBM bound (4 bytes of W read and
// written per n x m element against 2 r flops), so the kernel is built to keep
// W loads in flight, not to run the MFMA pipes hard.
//
// Each workgroup computes one 128 x 128 tile of W.  The read-modify-write of W
// is done on the accumulators in registers (no LDS).  bf16 W: an 8 x 8
// transpose across lanes (DPP) turns the MFMA output layout into rows, so that
// each lane reads and writes 8 consecutive columns (one 16-byte access; 8 loads
// and 8 stores per lane and tile instead of 32 + 32).  fp32 W: one DPP swap
// between adjacent lanes gives pairs of two columns.
//
// Workgroup: 4 waves, each 64 (columns of W) x 64 (rows of W) = 2 x 2 MFMA
// 32x32x16 fragments.  Both operands are K-row major (N [r][m], P^T [r][n]); they
// are copied to LDS as 16-deep K steps by buffer_load_dwordx4 ... lds (4 stages,
// copies 3 K steps ahead) and read as fragments with the transposing LDS read,
// as in the G^ kernel (same 256-byte K rows and swizzle).  32 KB of LDS and at
// most 128 registers per lane let four workgroups share a CU.  The tile of W
// (32 KB bf16) is loaded into registers after the K loop: held through the
// loop it would cost 32 registers per lane and one workgroup per CU (measured:
// 81.4 us per launch with three workgroups and W loaded early, 77.6 us with
// four and W loaded late), and the other workgroups of the CU cover its
// latency.
//
// Edges: K rows past r read as zero (buffer range ends at row r of N and P^T),
// rows of W past n are out of range (loads zero, stores dropped), columns of W
// past m are never stored.
#pragma once
#include "gemm_ghat.hpp"

namespace compact {

constexpr int kDecT = 128;                            // tile rows and columns
constexpr int kDecK = 16;                             // K step (rank): one MFMA deep
constexpr int kDecStages = 4;
constexpr int kDecAhead = kDecStages - 1;             // K steps copied ahead
constexpr uint32_t kDecStage = kDecK * kDecT * 2;     // 4 KB, one operand
constexpr uint32_t kDecBBase = kDecStages * kDecStage;
constexpr size_t kDecLds = 2u * kDecStages * kDecStage;  // 32 KB
constexpr int kDecBatch = 40;                         // layers per launch

struct DecW4Layer {
  void* W;              // [n x m], ld ldw; bf16 or fp32 (the launch's w_f32)
  const uint16_t* N;    // [r x m] bf16, ld ldn (multiple of 8)
  const uint16_t* pt;   // [r x ldpt] bf16 P^T (unscaled), ldpt a multiple of 8
  int ldw, ldn, ldpt;
  int n, m, r;
  int tiles_c;          // ceil(m / 128)
  float coef;
};

struct DecW4Batch {
  int count;
  int begin[kDecBatch + 1];  // first workgroup of each layer; begin[count] = grid
  DecW4Layer layer[kDecBatch];
};
static_assert(sizeof(DecW4Batch) <= 4096, "kernel argument size");

// s_waitcnt vmcnt(N) lgkmcnt(0), then s_barrier.
template <int N>
__device__ __forceinline__ void dec_wait_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt immediate");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// Waits for this wave's transposing reads and ties the fragments to that point.
__device__ __forceinline__ void dec_wait_frags(u32x4 (&fa)[2], u32x4 (&fb)[2]) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(fa[0]), "+v"(fa[1]), "+v"(fb[0]), "+v"(fb[1]));
}

// 8 x 8 transpose of fp32 values across the 8 lanes of each lane group: on
// exit lane t of a group holds in x[u] what lane u held in x[t] on entry.
// Three exchanges of a lane bit with an element bit: xor 1 and xor 2 lanes by
// quad permutes, xor 4 by row shifts of 4 with bank masks (4-lane banks).
// one exchange of lane bit log2(D) with element bit log2(D) (D = 1, 2) by a
// quad permute (QP: quad_perm 1,0,3,2 or 2,3,0,1)
template <int D, int QP>
__device__ __forceinline__ void dec_xchg(float (&x)[8], int lane) {
  const bool hi = (lane & D) != 0;
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    if (p & D) continue;
    const float snd = hi ? x[p] : x[p | D];
    const float rcv = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(snd), QP, 0xF, 0xF, false));
    x[p] = hi ? rcv : x[p];
    x[p | D] = hi ? x[p | D] : rcv;
  }
}

__device__ __forceinline__ void dec_transpose8(float (&x)[8], int lane) {
  dec_xchg<1, 0xB1>(x, lane);
  dec_xchg<2, 0x4E>(x, lane);
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const float keep = x[p];
    // lanes 4-7 of each 8 take the partner's x[p + 4] into x[p] (row_shr:4),
    // lanes 0-3 the partner's x[p] into x[p + 4] (row_shl:4)
    x[p] = __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(x[p]), __float_as_int(x[p + 4]), 0x114, 0xF, 0xA,
                                                      false));
    x[p + 4] = __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(x[p + 4]), __float_as_int(keep), 0x104, 0xF,
                                                          0x5, false));
  }
}

template <bool WF32>
__device__ __forceinline__ void dec_w4_tile(const DecW4Layer& p, int tile) {
  typedef typename std::conditional<WF32, u32x2, uint32_t>::type WVec;
  constexpr int kEsz = WF32 ? 4 : 2;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wc = wave >> 1, wi = wave & 1;
  const int ti = tile / p.tiles_c, tc = tile - ti * p.tiles_c;
  const int i0 = ti * kDecT, c0 = tc * kDecT;
  const int kt = (p.r + kDecK - 1) / kDecK;

  // copies: block `wave` of each operand (1 KB = 4 K rows of 256 B)
  const __amdgpu_buffer_rsrc_t rn = w4_rsrc(p.N + c0, view_bytes(p.r, p.m, p.ldn, 0, c0, 2));
  const __amdgpu_buffer_rsrc_t rp = w4_rsrc(p.pt + i0, view_bytes(p.r, p.n, p.ldpt, 0, i0, 2));
  const int von = gh_off(p.ldn, 4 * wave + (lane >> 4), lane & 15);
  const int vop = gh_off(p.ldpt, 4 * wave + (lane >> 4), lane & 15);
  const uint32_t lbase = __builtin_amdgcn_groupstaticsize();
  const uint32_t kstep_n = static_cast<uint32_t>(kDecK * p.ldn * 2), kstep_p = static_cast<uint32_t>(kDecK * p.ldpt * 2);
  // copy K step u into stage u % 6 (2 copies per wave); past the last K step
  // the offsets are out of range and the stage is filled with zeros
  auto copy = [&](int u) {
    const uint32_t st = static_cast<uint32_t>(u % kDecStages) * kDecStage + static_cast<uint32_t>(wave) * 1024u;
    const uint32_t oob = u < kt ? 0u : kW4Oob;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rn, reinterpret_cast<w4_lds_void*>(static_cast<uintptr_t>(lbase + st)),
                                             16, static_cast<int>((von + u * kstep_n) | oob), 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rp, reinterpret_cast<w4_lds_void*>(static_cast<uintptr_t>(lbase + kDecBBase + st)), 16,
        static_cast<int>((vop + u * kstep_p) | oob), 0, 0, 0);
  };
#pragma unroll
  for (int u = 0; u < kDecAhead; ++u) copy(u);

  // The W tile.  Accumulator block (b, a) of a wave covers rows
  // wi 64 + b 32 .. + 31 and columns wc 64 + a 32 .. + 31 of the tile; lane l
  // holds column l mod 32 of it and, in register group g, rows 8 g + 4 (l / 32)
  // .. + 3.  After one swap of values between the lanes of a column pair, the
  // even lane owns rows 8 g + 4 (l / 32) + {0, 1} and the odd lane rows
  // + {2, 3}, both for the two columns of the pair: 4 bytes of bf16 W (8 of
  // fp32) per row, and an access instruction covers 4 row segments of 64
  // bytes.  item (b, a, g, q) of this lane is row wrow(b, g) + q, columns
  // wcol(a), wcol(a) + 1.
  // W may be a column slice of a wider matrix: the range ends at its last element
  const __amdgpu_buffer_rsrc_t rw = w4_rsrc(static_cast<char*>(p.W) + (static_cast<int64_t>(i0) * p.ldw + c0) * kEsz,
                                            view_bytes(p.n, p.m, p.ldw, i0, c0, kEsz));
  const int odd = lane & 1;
  const int row_l = wi * 64 + 4 * (lane >> 5) + 2 * odd, col_l = wc * 64 + (lane & 30);
  // bf16 W in rows: lane (l / 32, c = (l % 32) / 8, t = l % 8) holds, for block
  // (b, a) and half s, row wi 64 + 32 b + 16 s + 8 (t / 4) + 4 (l / 32) + t % 4
  // and the 8 columns wc 64 + 32 a + 8 c .. + 7 (one 16-byte access); the
  // accumulators reach that layout through an 8 x 8 transpose across lanes
  const int tr = lane & 7, row_r = wi * 64 + 8 * (tr >> 2) + 4 * (lane >> 5) + (tr & 3);
  const int col_r = wc * 64 + 8 * ((lane & 31) >> 3);
  f32x16 acc[2][2];  // [b][a]
  const f32x16 zero = {};
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int a = 0; a < 2; ++a) acc[b][a] = zero;
  for (int t = 0; t < kt; ++t) {
    // this wave's copies of K step t have landed (later VMEM operations: the
    // copies of the next kDecAhead - 1 K steps); the barrier makes the whole
    // stage visible and ends every wave's reads of stage
    // (t + kDecAhead) % kDecStages = (t - 1) % kDecStages, which the next
    // copies overwrite
    dec_wait_barrier<2 * (kDecAhead - 1)>();
    copy(t + kDecAhead);
    const uint32_t st = static_cast<uint32_t>(t % kDecStages) * kDecStage;
    u32x4 fa[2], fb[2];  // fragments of N (columns of W) and of P^T (rows of W)
#pragma unroll
    for (int a = 0; a < 2; ++a) fa[a] = gh_frag<kDecT>(lbase + st, wc * 64 + a * 32, 0, lane);
#pragma unroll
    for (int b = 0; b < 2; ++b) fb[b] = gh_frag<kDecT>(lbase + kDecBBase + st, wi * 64 + b * 32, 0, lane);
    dec_wait_frags(fa, fb);
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int a = 0; a < 2; ++a) acc[b][a] = mfma32x32x16(fb[b], fa[a], acc[b][a]);
  }
  WVec wv[2][2][4][2];
  u32x4 wr[2][2][2];
  if constexpr (WF32) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            const int off = ((row_l + b * 32 + 8 * g + q) * p.ldw + col_l + a * 32) * kEsz;
            wv[b][a][g][q] = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rw, off, 0, 0));
          }
  } else {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int sh = 0; sh < 2; ++sh) {
          const int off = ((row_r + b * 32 + 16 * sh) * p.ldw + col_r + a * 32) * 2;
          wr[b][a][sh] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rw, off, 0, 0));
        }
  }

  w4_wait_vm<0>();  // the W tile, and every copy (past-the-end ones too) has landed in LDS

  // W <- W - coef acc, one rounding (RNE for bf16); columns past m not stored
  const float coef = p.coef;
  const int m_left = p.m - c0;
  if constexpr (!WF32) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int sh = 0; sh < 2; ++sh) {
          float x[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) x[e] = coef * acc[b][a][8 * sh + e];
          dec_transpose8(x, lane);  // x[u] = column col_r + 32 a + u of this lane's row
          const u32x4 w = wr[b][a][sh];
          u32x4 o;
#pragma unroll
          for (int k = 0; k < 4; ++k)
            o[k] = pack_bf16x2(__uint_as_float(w[k] << 16) - x[2 * k], __uint_as_float(w[k] & 0xFFFF0000u) - x[2 * k + 1]);
          const int col = col_r + a * 32;
          const int off = ((row_r + b * 32 + 16 * sh) * p.ldw + col) * 2;
          if (col + 8 <= m_left) {
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(f32x4, o), rw, off, 0, 0);
          } else if (col < m_left) {
            // the tile's last columns: whole pairs, then a last single column
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              if (col + 2 * k + 2 <= m_left)
                __builtin_amdgcn_raw_buffer_store_b32(o[k], rw, off + 4 * k, 0, 0);
              else if (col + 2 * k < m_left)
                __builtin_amdgcn_raw_buffer_store_b16(static_cast<unsigned short>(o[k]), rw, off + 4 * k, 0, 0);
            }
          }
        }
    return;
  }
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int col = col_l + a * 32;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float d[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) d[e] = coef * acc[b][a][4 * g + e];
        // the even lane sends rows +2, +3 and keeps rows +0, +1; the odd lane
        // the other way round
        const float s0 = odd ? d[0] : d[2], s1 = odd ? d[1] : d[3];
        const float r0 = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(s0), 0xB1, 0xF, 0xF, false));
        const float r1 = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(s1), 0xB1, 0xF, 0xF, false));
        // (column col, column col + 1) of this lane's two rows
        const float lo[2] = {odd ? r0 : d[0], odd ? r1 : d[1]};
        const float hi[2] = {odd ? d[2] : r0, odd ? d[3] : r1};
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int off = ((row_l + b * 32 + 8 * g + q) * p.ldw + col) * kEsz;
          if constexpr (WF32) {
            const u32x2 w = wv[b][a][g][q];
            u32x2 o;
            o.x = __float_as_uint(__uint_as_float(w.x) - lo[q]);
            o.y = __float_as_uint(__uint_as_float(w.y) - hi[q]);
            if (col + 2 <= m_left)
              __builtin_amdgcn_raw_buffer_store_b64(o, rw, off, 0, 0);
            else if (col < m_left)
              __builtin_amdgcn_raw_buffer_store_b32(o.x, rw, off, 0, 0);
          } else {
            const uint32_t w = wv[b][a][g][q];
            const uint32_t o = pack_bf16x2(__uint_as_float(w << 16) - lo[q], __uint_as_float(w & 0xFFFF0000u) - hi[q]);
            if (col + 2 <= m_left)
              __builtin_amdgcn_raw_buffer_store_b32(o, rw, off, 0, 0);
            else if (col < m_left)
              __builtin_amdgcn_raw_buffer_store_b16(static_cast<unsigned short>(o), rw, off, 0, 0);
          }
        }
      }
    }
}

}  // namespace compact
