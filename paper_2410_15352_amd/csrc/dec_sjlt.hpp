// Decompression and update of Alg. 3 for the sparse JL projection, as a row
// gather:  W[i, :] <- W[i, :] - coef sum_q sign_q N[h_q, :],  P = S / sqrt(s)
// (1/sqrt(s) is inside coef = lr alpha / sqrt(s)).  Row i of S holds the s
// signed draws (h_q, sign_q) of the sparse stream (pstream.hpp, sjlt_pair),
// so row i of P N is a signed sum of s rows of N: s additions per element of
// W instead of a product over all r rows of N, and no S panel.  The kernel
// streams W once (read, update in fp32, one rounding, write) and reads the
// rows of N it needs, which stay in L2 (N is r x m).
//
// Work unit: kSjltRows rows of W and up to kSjltChunks chunks of 512
// columns, one wave; lane l owns columns 512 k + 8 l .. + 7 of chunk k.  The
// W chunks of all rows of the unit are loaded first, so that each wave keeps
// kSjltRows x 1 KB (bf16) of W in flight.  The draws of the
// row depend only on the row and the key, so each wave makes them once (they
// are wave-uniform).  The N rows of 8 draws are loaded at once (one L2 round
// trip per 8 draws, not one per draw), then summed in draw order in fp32
// (each term a bf16 value of N, exact in fp32); W - coef x sum rounds once
// (RNE for bf16 W), as the tiled kernel does with its accumulators.
#pragma once
#include "common.hpp"
#include "gemm_w4.hpp"
#include "pstream.hpp"

namespace compact {

constexpr int kSjltChunks = 2;    // chunks of 512 columns per wave
constexpr int kSjltDraws = 8;     // draws whose N rows are loaded together
constexpr int kSjltRows = 4;      // rows of W per wave (their W loads are in flight together)
constexpr int kSjltBatch = 40;    // layers per launch

struct DecSjltLayer {
  void* W;             // [n x m], ld ldw; bf16 or fp32 (the launch's w_f32)
  const uint16_t* N;   // [r x m] bf16, ld ldn (multiple of 8, 16-byte aligned)
  int ldw, ldn;
  int n, m, r, s;
  PhiloxKey key;
  float coef;
  int groups;          // ceil(m / (512 kSjltChunks)): work units per row group
  int vec;             // W rows 16-byte aligned (16-byte accesses inside the row; the
                       // entry points require it, the element path is a guard)
};

struct DecSjltBatch {
  int count;
  int begin[kSjltBatch + 1];  // first workgroup of each layer; begin[count] = grid
  DecSjltLayer layer[kSjltBatch];
};
static_assert(sizeof(DecSjltBatch) <= 4096, "kernel argument size");

// Raw W chunk: 8 columns (bf16: one 16-byte word; fp32: two).
template <bool WF32>
struct SjltW {
  u32x4 v[WF32 ? 2 : 1];
};

template <bool WF32>
__device__ __forceinline__ SjltW<WF32> sjlt_load_w(__amdgpu_buffer_rsrc_t rw, int c0, int m, bool vec) {
  SjltW<WF32> w;
  if (vec && c0 + 8 <= m) {
#pragma unroll
    for (int h = 0; h < (WF32 ? 2 : 1); ++h) w.v[h] = __builtin_amdgcn_raw_buffer_load_b128(rw, c0 * (WF32 ? 4 : 2) + 16 * h, 0, 0);
  } else {
    uint32_t e32[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int c = c0 + e;
      if constexpr (WF32)
        e32[e] = c < m ? __builtin_amdgcn_raw_buffer_load_b32(rw, c * 4, 0, 0) : 0u;
      else
        e32[e] = c < m ? static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(rw, c * 2, 0, 0)) : 0u;
    }
    if constexpr (WF32) {
      w.v[0] = u32x4{e32[0], e32[1], e32[2], e32[3]};
      w.v[1] = u32x4{e32[4], e32[5], e32[6], e32[7]};
    } else {
      w.v[0] = u32x4{e32[0] | (e32[1] << 16), e32[2] | (e32[3] << 16), e32[4] | (e32[5] << 16), e32[6] | (e32[7] << 16)};
    }
  }
  return w;
}

template <bool WF32>
__device__ __forceinline__ float sjlt_w_elem(const SjltW<WF32>& w, int e) {
  if constexpr (WF32) return __uint_as_float(w.v[e >> 2][e & 3]);
  const uint32_t word = w.v[0][e >> 1];
  return __uint_as_float((e & 1) ? (word & 0xFFFF0000u) : (word << 16));
}

template <bool WF32>
__device__ __forceinline__ void dec_sjlt_unit(const DecSjltLayer& p, int64_t unit) {
  constexpr int kEsz = WF32 ? 4 : 2;
  const int lane = static_cast<int>(threadIdx.x & 63);
  const int64_t i0 = (unit / p.groups) * kSjltRows;
  if (i0 >= p.n) return;  // wave-uniform
  const int cbase = static_cast<int>(unit % p.groups) * (512 * kSjltChunks);
  const int m = p.m;
  const __amdgpu_buffer_rsrc_t rn = w4_rsrc(p.N, static_cast<int64_t>(p.r) * p.ldn * 2);
  // the W chunks of all rows of the unit, loaded first: kSjltRows x
  // kSjltChunks 16-byte accesses per lane in flight while the draws are made
  // and the N rows are summed
  __amdgpu_buffer_rsrc_t rw[kSjltRows];
  SjltW<WF32> w[kSjltRows][kSjltChunks];
#pragma unroll
  for (int j = 0; j < kSjltRows; ++j) {
    const int64_t i = i0 + j;
    // row i (64-bit base: offsets inside the row stay small); rows past n
    // get an empty range
    rw[j] = w4_rsrc(static_cast<char*>(p.W) + i * static_cast<int64_t>(p.ldw) * kEsz,
                    i < p.n ? static_cast<int64_t>(m) * kEsz : 0);
#pragma unroll
    for (int k = 0; k < kSjltChunks; ++k) w[j][k] = sjlt_load_w<WF32>(rw[j], cbase + 512 * k + 8 * lane, m, p.vec != 0);
  }
  const float coef = p.coef;
#pragma unroll
  for (int j = 0; j < kSjltRows; ++j) {  // unrolled: w[j] and rw[j] stay in registers
    const int64_t i = i0 + j;
    if (i >= p.n) break;  // wave-uniform
    // sum_q sign_q N[h_q, columns]: N rows are ldn >= round_up(m, 8) wide, so
    // a chunk that starts before m lies inside its row
    float acc[kSjltChunks][8];
#pragma unroll
    for (int k = 0; k < kSjltChunks; ++k)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[k][e] = 0.0f;
    for (int q0 = 0; q0 < p.s; q0 += kSjltDraws) {
      uint32_t h[kSjltDraws];
      float sg[kSjltDraws];
#pragma unroll
      for (int u = 0; u < kSjltDraws; u += 2)
        sjlt_pair(p.key, static_cast<uint32_t>(i), static_cast<uint32_t>((q0 + u) >> 1), static_cast<uint32_t>(p.r),
                  h[u], sg[u], h[u + 1], sg[u + 1]);
      u32x4 v[kSjltDraws][kSjltChunks];
#pragma unroll
      for (int u = 0; u < kSjltDraws; ++u)
#pragma unroll
        for (int k = 0; k < kSjltChunks; ++k) {
          const int c0 = cbase + 512 * k + 8 * lane;
          const bool live = q0 + u < p.s && c0 < m;
          v[u][k] = __builtin_amdgcn_raw_buffer_load_b128(
              rn, live ? static_cast<int>(h[u]) * p.ldn * 2 + c0 * 2 : static_cast<int>(kW4Oob), 0, 0);
        }
#pragma unroll
      for (int u = 0; u < kSjltDraws; ++u) {
        const float g = q0 + u < p.s ? sg[u] : 0.0f;  // past s: loads of zeros, signs of zero
#pragma unroll
        for (int k = 0; k < kSjltChunks; ++k)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[k][2 * e] = acc[k][2 * e] + g * __uint_as_float(v[u][k][e] << 16);
            acc[k][2 * e + 1] = acc[k][2 * e + 1] + g * __uint_as_float(v[u][k][e] & 0xFFFF0000u);
          }
      }
    }
    // W - coef sum, one rounding; columns past m are not stored
#pragma unroll
    for (int k = 0; k < kSjltChunks; ++k) {
      const int c0 = cbase + 512 * k + 8 * lane;
      if (c0 >= m) continue;
      float o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = sjlt_w_elem<WF32>(w[j][k], e) - coef * acc[k][e];
      if (p.vec && c0 + 8 <= m) {
        if constexpr (WF32) {
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, f32x4{o[0], o[1], o[2], o[3]}), rw[j],
                                                 c0 * 4, 0, 0);
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, f32x4{o[4], o[5], o[6], o[7]}), rw[j],
                                                 c0 * 4 + 16, 0, 0);
        } else {
          u32x4 ov;
#pragma unroll
          for (int e = 0; e < 4; ++e) ov[e] = pack_bf16x2(o[2 * e], o[2 * e + 1]);
          __builtin_amdgcn_raw_buffer_store_b128(ov, rw[j], c0 * 2, 0, 0);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int c = c0 + e;
          if (c >= m) break;
          if constexpr (WF32)
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(o[e]), rw[j], c * 4, 0, 0);
          else
            __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(pack_bf16x2(o[e], 0.0f) & 0xFFFFu), rw[j],
                                                  c * 2, 0, 0);
        }
      }
    }
  }
}

// Four waves per workgroup, one work unit each.
template <bool WF32>
__global__ __launch_bounds__(256) void k_dec_sjlt(DecSjltBatch b) {
  const int l = batch_layer_of(b.begin, b.count, static_cast<int>(blockIdx.x));
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
  dec_sjlt_unit<WF32>(b.layer[l], (static_cast<int64_t>(blockIdx.x) - b.begin[l]) * 4 + wave);
}

}  // namespace compact
