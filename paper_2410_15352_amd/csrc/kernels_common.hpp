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
//
// One launch serves a group of layers (same t and hyper-parameters) and also
// stages, for each layer that needs it, the P^T panel of the decompression:
// pt[j * ldpt + i] = bf16 of the unscaled stream element (i, j) (G, or S for
// the sparse projection; zero for i >= n).  The two
// jobs are independent; the Adam workgroups are spread evenly over the whole
// grid among the P^T workgroups (in proportion to their counts), so the
// HBM-bound moment update and the VALU-bound P stream run side by side from
// the first workgroup to the last.

// Values shared by every layer of a step.
struct AdamConsts {
  float b1, b2, omb1, omb2, bc1, bc2, eps;
  int n_f32;
  int kind;      // projection kind (kProjGaussian, kProjIdentity, kProjSparse)
  int sparse_s;  // draws per row of the sparse projection
};

struct AdamLayer {
  const float* G;
  float* M;
  float* V;
  void* N;
  uint16_t* pt;  // P^T panel [r][ldpt], or null
  PhiloxKey key;
  int ldn, r, m;
  int ldpt, n;
};

constexpr int kStepBatch = 40;  // layers per launch (kernel argument size)
constexpr int kAdamVec = 4;     // float4 groups per thread

struct StepBatch {
  AdamConsts c;
  int count;
  int adam_begin[kStepBatch + 1];  // first Adam workgroup of each layer
  int pt_begin[kStepBatch + 1];    // first P^T workgroup of each layer
  AdamLayer layer[kStepBatch];
};
static_assert(sizeof(StepBatch) <= 4096, "kernel argument size");

__device__ __forceinline__ void adam_one(const AdamConsts& c, float g, float mo, float vo, float& m1, float& v1,
                                         float& nv) {
  m1 = c.b1 * mo + c.omb1 * g;
  v1 = c.b2 * vo + c.omb2 * (g * g);
  const float mhat = m1 / c.bc1;
  const float vhat = v1 / c.bc2;
  nv = mhat / (__builtin_sqrtf(vhat) + c.eps);
}

// Elements [4 q, 4 q + 4) for q = first, first + stride, ... (m % 4 == 0, so a
// group of four never crosses a row), else one element per index.
__device__ __forceinline__ void adam_range(const AdamLayer& p, const AdamConsts& k, int64_t first, int64_t stride) {
  const int64_t total = int64_t(p.r) * p.m;
  if (p.m % 4 == 0) {
    for (int64_t q = first; q * 4 < total; q += stride) {
      const int64_t e = q * 4;
      // G, M and V are streamed once per step: non-temporal loads and stores (N,
      // which the decompression reads next, is stored normally)
      const f32x4 g = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p.G + e));
      const f32x4 mo = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p.M + e));
      const f32x4 vo = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p.V + e));
      f32x4 m1, v1, nv;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float a, b, c;
        adam_one(k, g[i], mo[i], vo[i], a, b, c);
        m1[i] = a;
        v1[i] = b;
        nv[i] = c;
      }
      __builtin_nontemporal_store(m1, reinterpret_cast<f32x4*>(p.M + e));
      __builtin_nontemporal_store(v1, reinterpret_cast<f32x4*>(p.V + e));
      const int64_t j = e / p.m, c = e - j * p.m;
      if (k.n_f32) {
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
      adam_one(k, p.G[e], p.M[e], p.V[e], m1, v1, nv);
      p.M[e] = m1;
      p.V[e] = v1;
      const int64_t j = e / p.m, c = e - j * p.m;
      if (k.n_f32)
        static_cast<float*>(p.N)[j * p.ldn + c] = nv;
      else
        static_cast<uint16_t*>(p.N)[j * p.ldn + c] = f32_to_bf16(nv);
    }
  }
}

// Adam workgroups of a layer: kAdamVec float4 groups (or elements) per thread.
__host__ __device__ inline int adam_blocks(int64_t r, int64_t m) {
  const int64_t work = (m % 4 == 0) ? ceil_div(r * m, 4) : r * m;
  const int64_t b = ceil_div(work, int64_t(256) * kAdamVec);
  return static_cast<int>(b < 1 ? 1 : b);
}

// Where a staged bf16 panel keeps element (row, k): row-major p[row * ld + k]
// (kblk == 0), or K-tiled p[((k / 32) * kblk + row) * 32 + k % 32], the layout
// of the persistent GEMM's K-tiled B operand (kblk = its row count).
struct PanelOut {
  uint16_t* p;
  int64_t ld, kblk;
};

__device__ __forceinline__ uint16_t* panel_at(const PanelOut& o, int64_t row, int64_t k) {
  return o.kblk ? o.p + (((k >> 5) * o.kblk + row) << 5) + (k & 31) : o.p + row * o.ld + k;
}

// One quad of a P^T panel: element (row0 + j, i0 .. i0 + 3) of `out` = bf16(scale
// x the unscaled stream elements (i0 .. i0 + 3, j)) (scale 1 for the identity);
// rows i >= n are written as zero.
__device__ __forceinline__ void pstream_t_quad(const ProjDesc& d, PhiloxKey key, int64_t n, float scale,
                                               const PanelOut& out, int64_t row0, int64_t j, int64_t i0) {
  float g[4] = {0.f, 0.f, 0.f, 0.f};
  if (i0 < n) {
    proj_quad(d, key, i0, j, g);
    if (d.kind != kProjIdentity)
      for (int e = 0; e < 4; ++e) g[e] = g[e] * scale;
    for (int e = 0; e < 4; ++e)
      if (i0 + e >= n) g[e] = 0.0f;
  }
  u32x2 v;
  v.x = pack_bf16x2(g[0], g[1]);
  v.y = pack_bf16x2(g[2], g[3]);
  *reinterpret_cast<u32x2*>(panel_at(out, row0 + j, i0)) = v;
}

// Work units of a P^T panel [r][ld]: a quad (four rows i of one column j)
// for the Gaussian and the identity; for the sparse projection one row i and
// kSjltChunk consecutive columns, so that the row's s draws are made once per
// unit rather than once per element.
constexpr int kSjltChunk = 32;

__host__ __device__ inline int64_t proj_t_units(int kind, int64_t r, int64_t ld) {
  return kind == kProjSparse ? ld * ceil_div(r, kSjltChunk) : (ld / 4) * r;
}

// Unit u of a P^T panel: element (row0 + j, i) of `out` = bf16(scale x stream
// element (i, j)) (scale 1 for the identity) for i < ld (the panel's K extent);
// rows i >= n are written as zero.
__device__ __forceinline__ void proj_t_unit(const ProjDesc& d, PhiloxKey key, int64_t n, float scale,
                                            const PanelOut& out, int64_t row0, int64_t ld, int64_t u) {
  if (d.kind != kProjSparse) {
    const int64_t qpr = ld / 4;
    pstream_t_quad(d, key, n, scale, out, row0, u / qpr, (u % qpr) * 4);
    return;
  }
  const int64_t i = u % ld, c0 = (u / ld) * kSjltChunk;
  float acc[kSjltChunk];
#pragma unroll
  for (int k = 0; k < kSjltChunk; ++k) acc[k] = 0.0f;
  if (i < n) {
#pragma unroll 1
    for (int q = 0; q < d.s; q += 2) {
      uint32_t h0, h1;
      float s0, s1;
      sjlt_pair(key, static_cast<uint32_t>(i), static_cast<uint32_t>(q >> 1), static_cast<uint32_t>(d.r), h0, s0,
                h1, s1);
      if (q + 1 >= d.s) s1 = 0.0f;  // odd s: the pair's second draw is not taken
#pragma unroll
      for (int k = 0; k < kSjltChunk; ++k) {
        const uint32_t c = static_cast<uint32_t>(c0 + k);
        acc[k] += (h0 == c ? s0 : 0.0f);
        acc[k] += (h1 == c ? s1 : 0.0f);
      }
    }
  }
#pragma unroll
  for (int k = 0; k < kSjltChunk; ++k)
    if (c0 + k < d.r) *panel_at(out, row0 + c0 + k, i) = f32_to_bf16(acc[k] * scale);
}

// P^T workgroups of a layer: one unit per thread.
__host__ __device__ inline int pt_blocks(int kind, int64_t r, int64_t ldpt) {
  return static_cast<int>(ceil_div(proj_t_units(kind, r, ldpt), 256));
}

__global__ void k_adam_pt_batched(StepBatch s) {
  const int na = s.adam_begin[s.count], np = s.pt_begin[s.count];
  const int64_t total = static_cast<int64_t>(na) + np;
  const int64_t b = blockIdx.x;
  // Adam workgroups before grid position b: floor(b na / total); position b is
  // an Adam workgroup where that count steps up
  const int before = static_cast<int>(b * na / total);
  const bool adam = static_cast<int>((b + 1) * na / total) > before;
  const int idx = adam ? before : static_cast<int>(b) - before;
  if (adam) {
    const int l = batch_layer_of(s.adam_begin, s.count, idx);
    const int nb = s.adam_begin[l + 1] - s.adam_begin[l];
    adam_range(s.layer[l], s.c, static_cast<int64_t>(idx - s.adam_begin[l]) * blockDim.x + threadIdx.x,
               static_cast<int64_t>(nb) * blockDim.x);
  } else {
    const int l = batch_layer_of(s.pt_begin, s.count, idx);
    const AdamLayer& p = s.layer[l];
    const int64_t u = static_cast<int64_t>(idx - s.pt_begin[l]) * blockDim.x + threadIdx.x;
    if (u >= proj_t_units(s.c.kind, p.r, p.ldpt)) return;
    proj_t_unit(ProjDesc{s.c.kind, p.r, s.c.sparse_s}, p.key, p.n, 1.0f, PanelOut{p.pt, p.ldpt, 0}, 0, p.ldpt, u);
  }
}

// ------------------------------- fp32 GEMM ---------------------------------
// Operand element (u, v) = p[u * su + v * sv] for u < U, v < V (else 0), or,
// with pgen set, the unscaled projection stream element (u = row i < n,
// v = column j < r): G, the identity or S.
struct OperandF32 {
  const float* p;
  int64_t su, sv;
  int64_t U, V;
  int pgen;
  ProjDesc proj;
  PhiloxKey key;
};

__device__ __forceinline__ float operand_elem(const OperandF32& o, int64_t u, int64_t v) {
  if (u >= o.U || v >= o.V) return 0.0f;
  if (o.pgen) return proj_element(o.proj, o.key, u, v);
  return o.p[u * o.su + v * o.sv];
}

// C (M x N) = A (M x K) B (K x N).  mode 0: out = scale * C;  mode 1 (update):
// out = out - coef * C;  mode 2 (accumulate): out = out + C.
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
      } else if (p.mode == 2) {
        *o = *o + acc[a][b];
      } else {
        const float d = p.coef * acc[a][b];
        *o = *o - d;
      }
    }
}

}  // namespace compact
