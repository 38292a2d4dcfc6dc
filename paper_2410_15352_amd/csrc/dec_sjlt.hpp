// Decompression and update of Alg. 3 for the sparse JL projection, as a row
// gather:  W[i, :] <- W[i, :] - coef sum_q sign_q N[h_q, :],  P = S / sqrt(s)
// (1/sqrt(s) is inside coef = lr alpha / sqrt(s)).  Row i of S holds the s
// signed draws (h_q, sign_q) of the sparse stream (pstream.hpp, sjlt_pair),
// so row i of P N is a signed sum of s rows of N: s additions per element of
// W instead of a product over all r rows of N, and no S panel.  The kernel
// streams W once (read, update in fp32, one rounding, write) and reads the
// rows of N it needs, which stay in L2 (N is r x m).
//
// Work unit: one row of W and up to kSjltChunks chunks of 512 columns, one
// wave; lane l owns columns 512 k + 8 l .. + 7 of chunk k.  The draws of the
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
constexpr int kSjltBatch = 40;    // layers per launch

struct DecSjltLayer {
  void* W;             // [n x m], ld ldw; bf16 or fp32 (the launch's w_f32)
  const uint16_t* N;   // [r x m] bf16, ld ldn (multiple of 8, 16-byte aligned)
  int ldw, ldn;
  int n, m, r, s;
  PhiloxKey key;
  float coef;
  int groups;          // ceil(m / (512 kSjltChunks)): work units per row
  int vec;             // W rows 16-byte aligned (16-byte accesses inside the row; the
                       // entry points require it, the element path is a guard)
};

struct DecSjltBatch {
  int count;
  int begin[kSjltBatch + 1];  // first workgroup of each layer; begin[count] = grid
  DecSjltLayer layer[kSjltBatch];
};
static_assert(sizeof(DecSjltBatch) <= 4096, "kernel argument size");

template <bool WF32>
__device__ __forceinline__ void dec_sjlt_unit(const DecSjltLayer& p, int64_t unit) {
  constexpr int kEsz = WF32 ? 4 : 2;
  const int lane = static_cast<int>(threadIdx.x & 63);
  const int64_t i = unit / p.groups;
  if (i >= p.n) return;  // wave-uniform
  const int cbase = static_cast<int>(unit - i * p.groups) * (512 * kSjltChunks);
  const int m = p.m;
  // W row i (64-bit base: offsets inside the row stay small) and N
  const __amdgpu_buffer_rsrc_t rw =
      w4_rsrc(static_cast<char*>(p.W) + i * static_cast<int64_t>(p.ldw) * kEsz, static_cast<int64_t>(m) * kEsz);
  const __amdgpu_buffer_rsrc_t rn = w4_rsrc(p.N, static_cast<int64_t>(p.r) * p.ldn * 2);
  // the W chunks of this lane, loaded first (their latency overlaps the sum)
  float w[kSjltChunks][8];
#pragma unroll
  for (int k = 0; k < kSjltChunks; ++k) {
    const int c0 = cbase + 512 * k + 8 * lane;
    if (p.vec && c0 + 8 <= m) {
      if constexpr (WF32) {
        const f32x4 a = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rw, c0 * 4, 0, 0));
        const f32x4 b = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rw, c0 * 4 + 16, 0, 0));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          w[k][e] = a[e];
          w[k][4 + e] = b[e];
        }
      } else {
        const u32x4 a = __builtin_amdgcn_raw_buffer_load_b128(rw, c0 * 2, 0, 0);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          w[k][2 * e] = __uint_as_float(a[e] << 16);
          w[k][2 * e + 1] = __uint_as_float(a[e] & 0xFFFF0000u);
        }
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int c = c0 + e;
        if constexpr (WF32)
          w[k][e] = c < m ? __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rw, c * 4, 0, 0)) : 0.0f;
        else
          w[k][e] = c < m ? __uint_as_float(static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(rw, c * 2, 0, 0))
                                            << 16)
                          : 0.0f;
      }
    }
  }
  // sum_q sign_q N[h_q, columns]: N rows are ldn >= round_up(m, 8) wide, so a
  // chunk that starts before m lies inside its row
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
  const float coef = p.coef;
#pragma unroll
  for (int k = 0; k < kSjltChunks; ++k) {
    const int c0 = cbase + 512 * k + 8 * lane;
    if (c0 >= m) continue;
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = w[k][e] - coef * acc[k][e];
    if (p.vec && c0 + 8 <= m) {
      if constexpr (WF32) {
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, f32x4{o[0], o[1], o[2], o[3]}), rw, c0 * 4,
                                               0, 0);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, f32x4{o[4], o[5], o[6], o[7]}), rw,
                                               c0 * 4 + 16, 0, 0);
      } else {
        u32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = pack_bf16x2(o[2 * e], o[2 * e + 1]);
        __builtin_amdgcn_raw_buffer_store_b128(v, rw, c0 * 2, 0, 0);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int c = c0 + e;
        if (c >= m) break;
        if constexpr (WF32)
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(o[e]), rw, c * 4, 0, 0);
        else
          __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(pack_bf16x2(o[e], 0.0f) & 0xFFFFu), rw, c * 2,
                                                0, 0);
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
