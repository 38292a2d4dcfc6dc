// P stream: the per-layer Gaussian projection of CompAct, generated on the fly.
//
// The method samples P ~ N(0, 1/r), P in R^{n x r}, from a per-layer seed in
// the forward pass and re-samples it with the same seed in the update step
// (CompAct Alg. 1 and Alg. 3; §3.3 "Random Projection Matrix").  P is never
// stored: any element is a pure function of (seed, i, j).
//
// Element (i, j) of the unscaled stream G (P = G / sqrt(r)):
//   key     = (seed mod 2^32, seed >> 32)
//   counter = (i >> 2, j, 0, 0)
//   (w0, w1, w2, w3) = Philox4x32-10(counter, key)       [Salmon et al., SC'11]
//   (a, b)  = (w0, w1) for rows 4p, 4p+1;  (w2, w3) for rows 4p+2, 4p+3
//   G = rho(a) * cos(theta(b)) on even rows, rho(a) * sin(theta(b)) on odd rows
// with the Box-Muller radius rho = sqrt(-2 ln u), u = (2 (a >> 9) + 1) 2^-24,
// and angle theta = 2 pi ((b >> 8) + 1/2) 2^-24.  One Philox call therefore
// yields four consecutive rows of one column.
//
// The transcendental parts are a fixed sequence of IEEE fp32 operations (one
// rounding each, no contraction into FMA): atanh series for ln, Taylor series
// for sin and cos on [0, pi/4] after an exact integer octant reduction.  Their
// coefficients are the fp32 roundings of 1/k and 1/k!.  The same definition is
// implemented separately by the CPU reference, so the stream matches bit for bit.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace compact {

struct PhiloxKey {
  uint32_t k0, k1;
};

__host__ __device__ inline PhiloxKey philox_key(uint64_t seed) {
  return PhiloxKey{static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32)};
}

// Philox4x32-10 with counter (c0, c1, c2, 0).
__device__ __forceinline__ void philox4x32_10(uint32_t c0, uint32_t c1, PhiloxKey key,
                                              uint32_t& o0, uint32_t& o1, uint32_t& o2,
                                              uint32_t& o3, uint32_t c2 = 0u) {
  constexpr uint32_t kM0 = 0xD2511F53u, kM1 = 0xCD9E8D57u;
  constexpr uint32_t kW0 = 0x9E3779B9u, kW1 = 0xBB67AE85u;
  uint32_t x0 = c0, x1 = c1, x2 = c2, x3 = 0u;
  uint32_t k0 = key.k0, k1 = key.k1;
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint32_t hi0 = __umulhi(kM0, x0), lo0 = kM0 * x0;
    const uint32_t hi1 = __umulhi(kM1, x2), lo1 = kM1 * x2;
    const uint32_t y0 = hi1 ^ x1 ^ k0;
    const uint32_t y2 = hi0 ^ x3 ^ k1;
    x0 = y0;
    x1 = lo1;
    x2 = y2;
    x3 = lo0;
    k0 += kW0;
    k1 += kW1;
  }
  o0 = x0;
  o1 = x1;
  o2 = x2;
  o3 = x3;
}

// ---------------------------------------------------------------------------
// fp32 Box-Muller.  Each statement is one rounded fp32 operation.
// ---------------------------------------------------------------------------

// ln(u) for fp32 u in (0, 1): u = 2^e f, f in (sqrt2/2, sqrt2], ln f = 2 atanh(s),
// s = (f - 1) / (f + 1), series 2s (1 + s^2/3 + s^4/5 + s^6/7 + s^8/9).
__device__ __forceinline__ float pstream_log(float u) {
#pragma clang fp contract(off)
  constexpr float c3 = 1.0f / 3.0f, c5 = 1.0f / 5.0f, c7 = 1.0f / 7.0f, c9 = 1.0f / 9.0f;
  constexpr float ln2 = 0.693147180559945309417232121458176568f;
  const uint32_t bits = __float_as_uint(u);
  int e = static_cast<int>(bits >> 23) - 127;
  const uint32_t mant = bits & 0x7FFFFFu;
  // fp32(sqrt 2) has mantissa bits 0x3504F3; above it, halve f.
  const bool big = mant > 0x3504F3u;
  const float f = __uint_as_float(mant | (big ? 0x3F000000u : 0x3F800000u));
  e += big ? 1 : 0;
  const float num = f - 1.0f;
  const float den = f + 1.0f;
  const float s = num / den;
  const float s2 = s + s;
  const float z = s * s;
  float p = c9;
  p = p * z;
  p = p + c7;
  p = p * z;
  p = p + c5;
  p = p * z;
  p = p + c3;
  float t = z * p;
  t = s2 * t;
  const float lnf = s2 + t;
  const float el = static_cast<float>(e) * ln2;
  return el + lnf;
}

// sin(x), cos(x) for x in [0, pi/4] (Taylor series to x^9 and x^10).
__device__ __forceinline__ void pstream_sincos(float x, float& sn, float& cs) {
#pragma clang fp contract(off)
  constexpr float s3 = -(1.0f / 6.0f), s5 = 1.0f / 120.0f, s7 = -(1.0f / 5040.0f),
                  s9 = 1.0f / 362880.0f;
  constexpr float k2 = -(1.0f / 2.0f), k4 = 1.0f / 24.0f, k6 = -(1.0f / 720.0f),
                  k8 = 1.0f / 40320.0f, k10 = -(1.0f / 3628800.0f);
  const float z = x * x;
  float p = s9;
  p = p * z;
  p = p + s7;
  p = p * z;
  p = p + s5;
  p = p * z;
  p = p + s3;
  const float xz = x * z;
  const float ts = xz * p;
  sn = x + ts;
  float q = k10;
  q = q * z;
  q = q + k8;
  q = q * z;
  q = q + k6;
  q = q * z;
  q = q + k4;
  q = q * z;
  q = q + k2;
  const float tc = z * q;
  cs = 1.0f + tc;
}

// Box-Muller radius from a 32-bit word: 23-bit code, u = (2k + 1) 2^-24.
__device__ __forceinline__ float pstream_radius(uint32_t a) {
#pragma clang fp contract(off)
  const uint32_t ka = a >> 9;
  const float u = static_cast<float>(2u * ka + 1u) * 0x1p-24f;  // exact
  const float lnu = pstream_log(u);
  const float t = lnu * -2.0f;                                  // exact
  return __builtin_sqrtf(t);                                    // IEEE sqrt
}

// (cos theta, sin theta) for the 24-bit angle code of word b.
__device__ __forceinline__ void pstream_angle(uint32_t b, float& ct, float& st) {
#pragma clang fp contract(off)
  constexpr float half_pi = 1.57079632679489661923132169163975144f;
  const uint32_t kb = b >> 8;
  const uint32_t q = kb >> 22;            // quadrant
  const uint32_t c = kb & 0x3FFFFFu;      // 22-bit position in the quadrant
  const bool h = (c >> 21) != 0u;         // upper half: reflect about pi/4
  const uint32_t cr = h ? (0x3FFFFFu - c) : c;
  const float phi = static_cast<float>(2u * cr + 1u) * 0x1p-23f;  // exact, (0, 1/2)
  const float x = phi * half_pi;
  float sx, cx;
  pstream_sincos(x, sx, cx);
  const float s_psi = h ? cx : sx;
  const float c_psi = h ? sx : cx;
  switch (q) {
    case 0: ct = c_psi;  st = s_psi;  break;
    case 1: ct = -s_psi; st = c_psi;  break;
    case 2: ct = -c_psi; st = -s_psi; break;
    default: ct = s_psi; st = -c_psi; break;
  }
}

__device__ __forceinline__ void pstream_pair(uint32_t a, uint32_t b, float& g_even,
                                             float& g_odd) {
#pragma clang fp contract(off)
  const float rho = pstream_radius(a);
  float ct, st;
  pstream_angle(b, ct, st);
  g_even = rho * ct;
  g_odd = rho * st;
}

// The four unscaled normals G[4p + 0..3][j].
__device__ __forceinline__ void pstream_quad(PhiloxKey key, uint32_t p, uint32_t j, float g[4]) {
  uint32_t w0, w1, w2, w3;
  philox4x32_10(p, j, key, w0, w1, w2, w3);
  pstream_pair(w0, w1, g[0], g[1]);
  pstream_pair(w2, w3, g[2], g[3]);
}

// One element G[i][j] (computes a whole quad; for cold paths only).
__device__ __forceinline__ float pstream_element(PhiloxKey key, uint32_t i, uint32_t j) {
  float g[4];
  pstream_quad(key, i >> 2, j, g);
  return g[i & 3];
}

// ---------------------------------------------------------------------------
// Sparse Johnson-Lindenstrauss projection (the sparse JL transform of
// Dasgupta, Kumar and Sarlos, 2010, named by the paper as an alternative to the
// Gaussian, §4 ablations and §6).  Row i of P (n x r) receives s signed unit
// draws; draws that land on the same column add up; P = S / sqrt(s):
//   draw q of row i, q = 0 .. s-1:
//     (w0, w1, w2, w3) = Philox4x32-10((i, q >> 1, kSjltTag, 0), key(seed))
//     (a, b) = (w0, w1) for even q, (w2, w3) for odd q
//     column h = floor(a r / 2^32),  sign = +1 if b < 2^31 else -1
//   S[i][c] = sum of the signs of the draws of row i with h = c.
// E[P P^T] = I, as for the Gaussian: the diagonal is 1 in expectation and the
// off-diagonal terms vanish with the independent signs.  S is small integers,
// exact in bf16 and fp32.
// ---------------------------------------------------------------------------
constexpr uint32_t kSjltTag = 0x4A4C5350u;  // counter word 2 of the sparse stream
constexpr int kSjltMaxS = 64;

// Projection kinds of the device generators (the ABI's compact_proj codes).
enum : int { kProjGaussian = 0, kProjIdentity = 1, kProjSparse = 2 };

// Draws 2p and 2p + 1 of row i: columns h0, h1 and signs (+1 / -1).
__device__ __forceinline__ void sjlt_pair(PhiloxKey key, uint32_t i, uint32_t p, uint32_t r, uint32_t& h0,
                                          float& s0, uint32_t& h1, float& s1) {
  uint32_t w0, w1, w2, w3;
  philox4x32_10(i, p, key, w0, w1, w2, w3, kSjltTag);
  h0 = __umulhi(w0, r);
  s0 = (w1 >> 31) ? -1.0f : 1.0f;
  h1 = __umulhi(w2, r);
  s1 = (w3 >> 31) ? -1.0f : 1.0f;
}

// S[i][j] (unscaled) for s draws per row.
__device__ __forceinline__ float sjlt_element(PhiloxKey key, uint32_t i, uint32_t j, uint32_t r, int s) {
  float v = 0.0f;
  for (int q = 0; q < s; q += 2) {
    uint32_t h0, h1;
    float s0, s1;
    sjlt_pair(key, i, static_cast<uint32_t>(q >> 1), r, h0, s0, h1, s1);
    if (h0 == j) v += s0;
    if (q + 1 < s && h1 == j) v += s1;
  }
  return v;
}

// The projection a generator draws from: its kind, the rank r (the column
// range of the sparse hash) and the draws per row s (sparse only).
struct ProjDesc {
  int kind;
  int r;
  int s;
};

// Unscaled stream elements of rows i0 .. i0 + 3 (i0 % 4 == 0) of column j:
// G for the Gaussian, I for the identity, S for the sparse projection.
__device__ __forceinline__ void proj_quad(const ProjDesc& d, PhiloxKey key, int64_t i0, int64_t j, float g[4]) {
  if (d.kind == kProjIdentity) {
#pragma unroll
    for (int e = 0; e < 4; ++e) g[e] = (i0 + e == j) ? 1.0f : 0.0f;
  } else if (d.kind == kProjSparse) {
#pragma unroll 1
    for (int e = 0; e < 4; ++e)
      g[e] = sjlt_element(key, static_cast<uint32_t>(i0 + e), static_cast<uint32_t>(j), static_cast<uint32_t>(d.r), d.s);
  } else {
    pstream_quad(key, static_cast<uint32_t>(i0 >> 2), static_cast<uint32_t>(j), g);
  }
}

__device__ __forceinline__ float proj_element(const ProjDesc& d, PhiloxKey key, int64_t i, int64_t j) {
  if (d.kind == kProjIdentity) return i == j ? 1.0f : 0.0f;
  if (d.kind == kProjSparse)
    return sjlt_element(key, static_cast<uint32_t>(i), static_cast<uint32_t>(j), static_cast<uint32_t>(d.r), d.s);
  return pstream_element(key, static_cast<uint32_t>(i), static_cast<uint32_t>(j));
}

}  // namespace compact
