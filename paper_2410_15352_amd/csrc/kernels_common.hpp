// Precision-independent kernels: the Adam moment update on the compressed
// r x m gradient (CompAct Alg. 3, first block) and a plain fp32 tiled GEMM used
// by the fp32 variant of every contraction.
#pragma once
#include "common.hpp"
#include "pstream.hpp"

namespace compact {

// ------------------------------- Adam --------------------------------------
// M <- b1 M + (1 - b1) G;  V <- b2 V + (1 - b2) G^2   (stored uncorrected)
// N  = (M / bc1) / (sqrt(V / bc2) + eps),  bc_k = 1 - b_k^t
// G, M, V dense r x m fp32; N written r x m with leading dimension ldn, as
// bf16 (n_f32 == 0) or fp32.
struct AdamParams {
  const float* G;
  float* M;
  float* V;
  void* N;
  int64_t ldn;
  int n_f32;
  int64_t r, m;
  float b1, b2, omb1, omb2, bc1, bc2, eps;
};

__global__ void k_adam(AdamParams p) {
  const int64_t total = p.r * p.m;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < total;
       e += stride) {
    const float g = p.G[e];
    const float m1 = p.b1 * p.M[e] + p.omb1 * g;
    const float v1 = p.b2 * p.V[e] + p.omb2 * (g * g);
    p.M[e] = m1;
    p.V[e] = v1;
    const float mhat = m1 / p.bc1;
    const float vhat = v1 / p.bc2;
    const float nv = mhat / (__builtin_sqrtf(vhat) + p.eps);
    const int64_t j = e / p.m, c = e - j * p.m;
    if (p.n_f32)
      static_cast<float*>(p.N)[j * p.ldn + c] = nv;
    else
      static_cast<uint16_t*>(p.N)[j * p.ldn + c] = f32_to_bf16(nv);
  }
}

// ------------------------------- fp32 GEMM ---------------------------------
// Operand element (u, v) = p[u * su + v * sv] for u < U, v < V (else 0), or,
// with pgen set, the projection stream G(u, v) (u = row i < n, v = column j < r)
// or the identity.
struct OperandF32 {
  const float* p;
  int64_t su, sv;
  int64_t U, V;
  int pgen;
  int identity;
  PhiloxKey key;
};

__device__ __forceinline__ float operand_elem(const OperandF32& o, int64_t u, int64_t v) {
  if (u >= o.U || v >= o.V) return 0.0f;
  if (o.pgen) {
    if (o.identity) return u == v ? 1.0f : 0.0f;
    return pstream_element(o.key, static_cast<uint32_t>(u), static_cast<uint32_t>(v));
  }
  return o.p[u * o.su + v * o.sv];
}

// C (M x N) = A (M x K) B (K x N).  mode 0: out = scale * C;  mode 1 (update):
// out = out - coef * C.
struct GemmF32Params {
  OperandF32 A, B;
  int64_t M, N, K;
  int mode;
  float* out;
  int64_t ldo;
  float scale, coef;
  int tiles_n;
};

__global__ __launch_bounds__(256) void k_gemm_f32(GemmF32Params p) {
  constexpr int TM = 64, TN = 64, TK = 16;
  __shared__ float As[TK][TM + 4];
  __shared__ float Bs[TK][TN + 4];
  const int tid = threadIdx.x, tx = tid % 16, ty = tid / 16;
  const int64_t row0 = static_cast<int64_t>(blockIdx.x / p.tiles_n) * TM;
  const int64_t col0 = static_cast<int64_t>(blockIdx.x % p.tiles_n) * TN;
  float acc[4][4] = {};
  for (int64_t k0 = 0; k0 < p.K; k0 += TK) {
    for (int l = 0; l < 4; ++l) {
      const int e = tid + l * 256;
      const int mm = e % TM, kk = e / TM;
      As[kk][mm] = (k0 + kk < p.K) ? operand_elem(p.A, row0 + mm, k0 + kk) : 0.0f;
      Bs[kk][mm] = (k0 + kk < p.K) ? operand_elem(p.B, k0 + kk, col0 + mm) : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk)
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
          acc[a][b] = __builtin_fmaf(As[kk][ty * 4 + a], Bs[kk][tx * 4 + b], acc[a][b]);
    __syncthreads();
  }
  for (int a = 0; a < 4; ++a)
    for (int b = 0; b < 4; ++b) {
      const int64_t gr = row0 + ty * 4 + a, gc = col0 + tx * 4 + b;
      if (gr >= p.M || gc >= p.N) continue;
      float* o = p.out + gr * p.ldo + gc;
      if (p.mode == 0) {
        *o = p.scale * acc[a][b];
      } else {
        const float d = p.coef * acc[a][b];
        *o = *o - d;
      }
    }
}

}  // namespace compact
