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

__device__ __forceinline__ void adam_one(const AdamParams& p, int64_t e, float g, float mo, float vo,
                                         float& m1, float& v1, float& nv) {
  m1 = p.b1 * mo + p.omb1 * g;
  v1 = p.b2 * vo + p.omb2 * (g * g);
  const float mhat = m1 / p.bc1;
  const float vhat = v1 / p.bc2;
  nv = mhat / (__builtin_sqrtf(vhat) + p.eps);
  (void)e;
}

// Elements [4 q, 4 q + 4) for q = first, first + stride, ... (m % 4 == 0, so a
// group of four never crosses a row), else one element per index.
__device__ __forceinline__ void adam_range(const AdamParams& p, int64_t first, int64_t stride) {
  const int64_t total = p.r * p.m;
  if (p.m % 4 == 0) {
    for (int64_t q = first; q * 4 < total; q += stride) {
      const int64_t e = q * 4;
      const f32x4 g = *reinterpret_cast<const f32x4*>(p.G + e);
      const f32x4 mo = *reinterpret_cast<const f32x4*>(p.M + e);
      const f32x4 vo = *reinterpret_cast<const f32x4*>(p.V + e);
      f32x4 m1, v1, nv;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float a, b, c;
        adam_one(p, e + i, g[i], mo[i], vo[i], a, b, c);
        m1[i] = a;
        v1[i] = b;
        nv[i] = c;
      }
      *reinterpret_cast<f32x4*>(p.M + e) = m1;
      *reinterpret_cast<f32x4*>(p.V + e) = v1;
      const int64_t j = e / p.m, c = e - j * p.m;
      if (p.n_f32) {
        *reinterpret_cast<f32x4*>(static_cast<float*>(p.N) + j * p.ldn + c) = nv;
      } else {
        u32x2 w;
        w.x = pack_bf16x2(nv[0], nv[1]);
        w.y = pack_bf16x2(nv[2], nv[3]);
        *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(p.N) + j * p.ldn + c) = w;
      }
    }
  } else {
    for (int64_t e = first; e < total; e += stride) {
      float m1, v1, nv;
      adam_one(p, e, p.G[e], p.M[e], p.V[e], m1, v1, nv);
      p.M[e] = m1;
      p.V[e] = v1;
      const int64_t j = e / p.m, c = e - j * p.m;
      if (p.n_f32)
        static_cast<float*>(p.N)[j * p.ldn + c] = nv;
      else
        static_cast<uint16_t*>(p.N)[j * p.ldn + c] = f32_to_bf16(nv);
    }
  }
}

__global__ void k_adam(AdamParams p) {
  adam_range(p, static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x,
             static_cast<int64_t>(gridDim.x) * blockDim.x);
}

struct AdamBatch {
  int count;
  int begin[kBatchLayers + 1];
  AdamParams layer[kBatchLayers];
};

__global__ void k_adam_batched(AdamBatch a) {
  const int b = static_cast<int>(blockIdx.x);
  const int l = batch_layer_of(a.begin, a.count, b);
  const int nb = a.begin[l + 1] - a.begin[l];
  adam_range(a.layer[l], static_cast<int64_t>(b - a.begin[l]) * blockDim.x + threadIdx.x,
             static_cast<int64_t>(nb) * blockDim.x);
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
